// kernels_hidden_mfma.h -- the bf16 matrix-core column kernel for a block MLP whose hidden
// size HS differs from the block size BS (the AFNO layer's hidden-size factor; the paper's
// filter, "Model Innovations", has HS = BS and runs column_mfma).
//
// The same four products as column_mfma (forward DFT, the two layers, inverse DFT) in the same
// geometry, with the hidden layer taken in chunks of 2 BS entries: layer 1 writes one chunk
// H_c[k][entry] to LDS, layer 2 adds H_c W2x[chunk rows] to accumulators held in registers
// across the chunks.  The chunk tile occupies the table's LDS between the two transforms and
// the table is loaded again for the inverse, so the kernel needs no more LDS than column_mfma
// and two workgroups share a CU.  Weight fragments (prep_hidden_words): layer 1 as B fragments of W1x (K = 2 BS,
// N = 2 HS), word (s MH + t) 64 + lane; then layer 2 as B fragments of W2x (K = 2 HS, N = 2 BS),
// word L1 + (s MT + t) 64 + lane, with MH = 2 HS / 16, MT = 2 BS / 16, L1 = (2 BS / 32) MH 64.
#pragma once
#include "kernels_mfma.h"

namespace afno {

template <int HP, int BS, int HS>
struct MfmaHid {
  typedef MfmaCol<HP, BS> G;
  static constexpr int MH = 2 * HS / 16;            // 16-entry tiles over the hidden layer
  static constexpr int kChunks = MH / G::MT;        // hidden chunks of 2 BS entries
  static constexpr int64_t kL1Words = (int64_t)G::WKS * MH * 64;   // layer-1 fragment words
  static constexpr int64_t kBlockWords = 2 * kL1Words;            // both layers
  // the hidden chunk [k][entry] shares the row-major stride of the spectrum tile and, once
  // the forward transform is done, the table's LDS (the table is read again for the inverse)
  static constexpr int kChunkBytes = HP * G::kLdy * 2;
  static constexpr int kShared = ((G::kTabBytes > kChunkBytes ? G::kTabBytes : kChunkBytes) + 15) / 16 * 16;
  static constexpr int kBytes = kShared + G::kRegionBytes;
  static_assert(MH % G::MT == 0, "hidden tiles a multiple of the block's");
};

// grid B * KW * nb (block index fastest), 512 threads, dynamic LDS MfmaHid<HP, BS, HS>::kBytes.
// S: spectrum [B][H][KW][C] complex bf16, updated in place; wfrag, dtab from prep_operands
// (a job with hs set).
template <int HP, int BS, int HS>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4)))
column_mfma_hidden(bf16* __restrict__ S, const uint4* __restrict__ wfrag,
                   const uint4* __restrict__ dtab, const bf16* __restrict__ b1,
                   const bf16* __restrict__ b2, int H, int C, int KW, int nb, int kept_h,
                   float lam) {
  typedef MfmaCol<HP, BS> G;
  typedef MfmaHid<HP, BS, HS> Q;
  extern __shared__ uint4 smem_hid[];
  uint4* tab = smem_hid;
  bf16* Hc = reinterpret_cast<bf16*>(smem_hid);  // the hidden chunk, over the table
  bf16* R = reinterpret_cast<bf16*>(reinterpret_cast<char*>(smem_hid) + Q::kShared);
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int twm = wave / G::TWN, twn = wave % G::TWN;
  const int lwm = wave / G::LWN, lwn = wave % G::LWN;

  const int blk = blockIdx.x % nb;
  const int rest = blockIdx.x / nb;
  const int kw = rest % KW;
  const int64_t b = rest / KW;
  bf16* col = S + ((b * H) * KW + kw) * (int64_t)C * 2 + (int64_t)blk * BS * 2;
  const uint32_t rsb = (uint32_t)KW * (uint32_t)C * 4;
  const uint32_t cbytes = buf_bytes((uint64_t)H * rsb);
  const Buf wb(wfrag + blk * Q::kBlockWords, (uint32_t)(Q::kBlockWords * 16));
  constexpr uint32_t kL2Off = (uint32_t)(Q::kL1Words * 16);

  // ---- the table and the column (planar planes X[rho][c][h], rows >= H zero)
  for (int i = tid; i < G::kTabWords; i += G::kThreads) tab[i] = dtab[i];
  {
    const Buf cb(col, cbytes);
    constexpr int XT = BS * (HP / 8);
    constexpr int XR = (XT + G::kThreads - 1) / G::kThreads;
    uint32_t xv[XR][8];
#pragma unroll
    for (int u = 0; u < XR; ++u) {
      const int task = tid + u * G::kThreads;
      const int c = task % BS, r0 = 8 * (task / BS);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const bool ok = task < XT && r0 + e < H;
        const uint32_t wv = cb.ld32(ok ? c * 4u + (uint32_t)(r0 + e) * rsb : 0u, 0);
        xv[u][e] = ok ? wv : 0u;
      }
    }
#pragma unroll
    for (int u = 0; u < XR; ++u) {
      const int task = tid + u * G::kThreads;
      if (task < XT) {
        const int c = task % BS, r0 = 8 * (task / BS);
        uint4 re, im;
        re.x = __builtin_amdgcn_perm(xv[u][1], xv[u][0], 0x05040100u);
        re.y = __builtin_amdgcn_perm(xv[u][3], xv[u][2], 0x05040100u);
        re.z = __builtin_amdgcn_perm(xv[u][5], xv[u][4], 0x05040100u);
        re.w = __builtin_amdgcn_perm(xv[u][7], xv[u][6], 0x05040100u);
        im.x = __builtin_amdgcn_perm(xv[u][1], xv[u][0], 0x07060302u);
        im.y = __builtin_amdgcn_perm(xv[u][3], xv[u][2], 0x07060302u);
        im.z = __builtin_amdgcn_perm(xv[u][5], xv[u][4], 0x07060302u);
        im.w = __builtin_amdgcn_perm(xv[u][7], xv[u][6], 0x07060302u);
        *reinterpret_cast<uint4*>(R + c * G::kLdx + r0) = re;
        *reinterpret_cast<uint4*>(R + G::kPlane + c * G::kLdx + r0) = im;
      }
    }
  }
  __syncthreads();

  // ---- forward transform -> Y[k][entry]
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    dft_product<HP, BS>(R, tab, lane, twm, twn, 0, acc);
    __syncthreads();  // X and the table read
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) {
        const int k = 16 * (G::TNW * twn + n) + l16;
        const int e0 = 16 * (G::TMW * twm + m) + 4 * g;
        *reinterpret_cast<uint2*>(R + k * G::kLdy + e0) =
            make_uint2(cvt_pk(acc[m][n][0], acc[m][n][1]), cvt_pk(acc[m][n][2], acc[m][n][3]));
      }
  }
  __syncthreads();

  // ---- the MLP over hidden chunks: per chunk c, layer 1 (transposed)
  //      H_c^T[hidden][k] = relu(W1x[:, chunk]^T Y^T + b1[chunk]) -> Hc[k][entry], then layer 2
  //      acc2 += H_c W2x[chunk rows]
  f32x4 acc2[G::LMW][G::LNW];
#pragma unroll
  for (int m = 0; m < G::LMW; ++m)
#pragma unroll
    for (int n = 0; n < G::LNW; ++n) acc2[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
  for (int ch = 0; ch < Q::kChunks; ++ch) {
    {
      const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
      const int t0 = G::MT * ch + G::TMW * twm;  // the wave's first hidden tile of the chunk
      const uint32_t wvoff = lane * 16u;
      auto wload = [&](int s, int t) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(wb.r, wvoff,
                                                            (uint32_t)((s * Q::MH + t) * 64 * 16), 0);
        return make_uint4(v[0], v[1], v[2], v[3]);
      };
      f32x4 acc[G::TMW][G::TNW];
#pragma unroll
      for (int m = 0; m < G::TMW; ++m)
#pragma unroll
        for (int n = 0; n < G::TNW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
      uint4 wa[G::TMW];
#pragma unroll
      for (int m = 0; m < G::TMW; ++m) wa[m] = wload(0, t0 + m);
#pragma unroll
      for (int s = 0; s < G::WKS; ++s) {
        uint4 wn_[G::TMW], yb[G::TNW];
        if (s + 1 < G::WKS) {
#pragma unroll
          for (int m = 0; m < G::TMW; ++m) wn_[m] = wload(s + 1, t0 + m);
        }
#pragma unroll
        for (int n = 0; n < G::TNW; ++n) {
          const int k = 16 * (G::TNW * twn + n) + l16;
          yb[n] = *reinterpret_cast<const uint4*>(R + k * G::kLdy + 32 * s + 8 * g);
        }
#pragma unroll
        for (int m = 0; m < G::TMW; ++m)
#pragma unroll
          for (int n = 0; n < G::TNW; ++n) acc[m][n] = mma_bf16(wa[m], yb[n], acc[m][n]);
        if (s + 1 < G::WKS) {
#pragma unroll
          for (int m = 0; m < G::TMW; ++m) wa[m] = wn_[m];
        }
      }
#pragma unroll
      for (int m = 0; m < G::TMW; ++m) {
        const int jc = 16 * (G::TMW * twm + m) + 4 * g;  // entry within the chunk
        const uint32_t* bp =
            reinterpret_cast<const uint32_t*>(b1 + (int64_t)blk * HS * 2 + 2 * BS * ch + jc);
        const uint2 bb = make_uint2(bp[0], bp[1]);
        const float bias[4] = {__uint_as_float(bb.x << 16), __uint_as_float(bb.x & 0xffff0000u),
                               __uint_as_float(bb.y << 16), __uint_as_float(bb.y & 0xffff0000u)};
#pragma unroll
        for (int n = 0; n < G::TNW; ++n) {
          const int k = 16 * (G::TNW * twn + n) + l16;
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = fmaxf(acc[m][n][r] + bias[r], 0.f);
          *reinterpret_cast<uint2*>(Hc + k * G::kLdy + jc) =
              make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
        }
      }
    }
    __syncthreads();  // the chunk complete
    {
      const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
      const uint32_t wvoff = lane * 16u;
      auto wload = [&](int s, int t) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(
            wb.r, wvoff, kL2Off + (uint32_t)(((G::WKS * ch + s) * G::MT + t) * 64 * 16), 0);
        return make_uint4(v[0], v[1], v[2], v[3]);
      };
      uint4 wb_[G::LNW];
#pragma unroll
      for (int n = 0; n < G::LNW; ++n) wb_[n] = wload(0, G::LNW * lwn + n);
#pragma unroll
      for (int s = 0; s < G::WKS; ++s) {
        uint4 wn_[G::LNW], ha[G::LMW];
        if (s + 1 < G::WKS) {
#pragma unroll
          for (int n = 0; n < G::LNW; ++n) wn_[n] = wload(s + 1, G::LNW * lwn + n);
        }
#pragma unroll
        for (int m = 0; m < G::LMW; ++m) {
          const int k = 16 * (G::LMW * lwm + m) + l16;
          ha[m] = *reinterpret_cast<const uint4*>(Hc + k * G::kLdy + 32 * s + 8 * g);
        }
#pragma unroll
        for (int m = 0; m < G::LMW; ++m)
#pragma unroll
          for (int n = 0; n < G::LNW; ++n) acc2[m][n] = mma_bf16(ha[m], wb_[n], acc2[m][n]);
        if (s + 1 < G::WKS) {
#pragma unroll
          for (int n = 0; n < G::LNW; ++n) wb_[n] = wn_[n];
        }
      }
    }
    __syncthreads();  // the chunk read (and, after the last, Y no longer needed)
  }

  // ---- softshrink(acc2 + b2), cutoff -> planes O[rho][c][k] in R; the table back over the chunk
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    for (int i = opq((int)threadIdx.x); i < G::kTabWords; i += G::kThreads) tab[i] = dtab[i];
    float bias[G::LNW];
#pragma unroll
    for (int n = 0; n < G::LNW; ++n) bias[n] = (float)b2[(int64_t)blk * BS * 2 + 16 * (G::LNW * lwn + n) + l16];
    const bool all_rows = kept_h > H / 2;
#pragma unroll
    for (int m = 0; m < G::LMW; ++m) {
      const int k0 = 16 * (G::LMW * lwm + m) + 4 * g;
      bool keep[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) keep[r] = all_rows || row_kept(k0 + r, H, kept_h);
#pragma unroll
      for (int n = 0; n < G::LNW; ++n) {
        const int e = 16 * (G::LNW * lwn + n) + l16;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = keep[r] ? softshrink(acc2[m][n][r] + bias[n], lam) : 0.f;
        *reinterpret_cast<uint2*>(R + (e & 1) * G::kPlane + (e >> 1) * G::kLdx + k0) =
            make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
      }
    }
  }
  __syncthreads();

  // ---- inverse transform -> Z[h][entry] -> S rows h < H
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    dft_product<HP, BS>(R, tab, lane, twm, twn, 1, acc);
    __syncthreads();
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) {
        const int h = 16 * (G::TNW * twn + n) + l16;
        const int e0 = 16 * (G::TMW * twm + m) + 4 * g;
        *reinterpret_cast<uint2*>(R + h * G::kLdy + e0) =
            make_uint2(cvt_pk(acc[m][n][0], acc[m][n][1]), cvt_pk(acc[m][n][2], acc[m][n][3]));
      }
  }
  __syncthreads();
  constexpr int VPR = 2 * BS / 8;
  const Buf cb(col, cbytes);
  for (int it = tid; it < H * VPR; it += G::kThreads) {
    const int h = it / VPR, cv = it - h * VPR;
    cb.st128(*reinterpret_cast<const uint4*>(R + h * G::kLdy + cv * 8), cv * 16u + h * rsb, 0);
  }
}

}  // namespace afno
