// kernels_kept_mfma.h -- the bf16 matrix-core column kernel for a hard mode cutoff that keeps
// few spectral rows: 90 x 180 at keep 0.5 keeps 45 of 90 (|signed k| < 23).
//
// column_mfma runs its four products over every padded row and zeroes the dropped rows at
// the end of layer 2.  Here the rows the cutoff keeps are compacted: kept row k' < nkept =
// 2 kept_h - 1 is spectral row kept_row(k') (0, 1, .., kept_h - 1, then H - kept_h + 1, .., H - 1),
// padded to KP rows (16 <= KP <= 48, a multiple of 16).  With D the H-point DFT matrix as in
// kernels_mfma.h and two tables cut from it,
//   forward:  Y^T[(c, rho)][k'] = sum_(sigma, h) A[(c, rho)][(sigma, h)] Tf[(sigma, h)][k'],
//             Tf[(sigma, h)][k'] = Re / Im D[h][kept_row(k')]             (K = 2 HP, N = KP)
//   layer 1:  H1^T = relu(W1x^T Y^T + b1)                                  (N = KP)
//   layer 2:  O = softshrink(H1 W2x + b2)                                  (M = KP)
//   inverse:  Z^T[(c, rho)][h] = sum_(sigma, k') A'[(c, rho)][(sigma, k')] Ti[(sigma, k')][h],
//             Ti[(sigma, k')][h] = Re / Im D[kept_row(k')][h]              (K = 2 KP, N = HP)
// the forward producing only the kept rows and the inverse summing over them alone: the four
// products take KP / HP of column_mfma's matrix-core work (48 / 96 for 45 kept rows).  A and A'
// are column_mfma's operands (planes with per-lane plane choice and sign).  Ti's columns are
// rounded with dft_table_column's error carry over the kept rows.
//
// Six waves: products with 12 entry (or hidden) tiles of rows take two tiles each and every
// column tile (forward, layer 1, inverse); layer 2, with KP / 16 row tiles, takes two column
// tiles each and every row tile.
#pragma once
#include "kernels_mfma.h"

namespace afno {

template <int HP, int BS, int KP>
struct KeptCol {
  static constexpr int kThreads = 384;
  static constexpr int NW = 6;
  static constexpr int MT = 2 * BS / 16;    // 16-entry tiles
  static constexpr int HT = HP / 16;        // 16-row tiles over the field rows h
  static constexpr int KT = KP / 16;        // 16-row tiles over the kept rows k'
  static constexpr int DKS = 2 * HP / 32;   // k-steps of the forward (K = 2 HP)
  static constexpr int IKS = 2 * KP / 32;   // k-steps of the inverse (K = 2 KP)
  static constexpr int WKS = 2 * BS / 32;   // k-steps of a layer (K = 2 BS)
  static constexpr int MW = MT / NW;        // entry tiles per wave
  static_assert(HP == 96 && BS == 96 && KP % 16 == 0 && KP <= 48, "shapes of this kernel");
  static_assert(MT % NW == 0 && KP % 16 == 0, "wave split");
  static constexpr int kTfWords = DKS * KT * 64;   // kept_table_task's two tables
  static constexpr int kTiWords = IKS * HT * 64;
  static constexpr int kTabBytes = (kTfWords + kTiWords) * 16;
  // the column X as planes [rho][c][h] (column_mfma's strides), the row-major tiles
  // [k' or h][entry], and the mixed spectrum O as planes [rho][c][k']
  static constexpr int kLdx = HP + 8;
  static constexpr int kPlane = BS * kLdx + 64;
  static constexpr int kLdo = KP + 8;
  static constexpr int kPlaneO = BS * kLdo + 64;
  static constexpr int kLdy = 2 * BS + 8;
  static constexpr int kXBytes = (kPlane + BS * kLdx) * 2;
  static constexpr int kZBytes = HP * kLdy * 2;
  static constexpr int kRegionBytes = ((kXBytes > kZBytes ? kXBytes : kZBytes) + 15) / 16 * 16;
  static constexpr int kBytes = kTabBytes + kRegionBytes;
};

// grid B * KW * nb (block index fastest), 384 threads, dynamic LDS KeptCol<HP, BS, KP>::kBytes.
// S: spectrum [B][H][KW][C] complex bf16, updated in place; wfrag: column_mfma's weight
// fragments; dtab: Tf then Ti (kept_table_task, kernels_prep.h).  1 <= kept_h, 2 kept_h - 1 <= KP.
// stage: 0 full, 2 stop after the MLP (the mixed spectrum back to S: kept rows, zeros).
template <int HP, int BS, int KP>
__global__ void __launch_bounds__(384) __attribute__((amdgpu_waves_per_eu(3)))
column_mfma_kept(bf16* __restrict__ S, const uint4* __restrict__ wfrag,
                 const uint4* __restrict__ dtab, const bf16* __restrict__ b1,
                 const bf16* __restrict__ b2, int H, int C, int KW, int nb, int kept_h, float lam,
                 int stage) {
  typedef KeptCol<HP, BS, KP> G;
  extern __shared__ uint4 smem_kept[];
  uint4* tab = smem_kept;                    // Tf words, then Ti words
  bf16* R = reinterpret_cast<bf16*>(reinterpret_cast<char*>(smem_kept) + G::kTabBytes);
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int nkept = 2 * kept_h - 1;

  const int blk = blockIdx.x % nb;
  const int rest = blockIdx.x / nb;
  const int kw = rest % KW;
  const int64_t b = rest / KW;
  bf16* col = S + ((b * H) * KW + kw) * (int64_t)C * 2 + (int64_t)blk * BS * 2;
  const uint32_t rsb = (uint32_t)KW * (uint32_t)C * 4;
  const Buf cb(col, buf_bytes((uint64_t)H * rsb));

  // ---- both tables and the column (planes X[rho][c][h], rows >= H zero)
  constexpr int TW = G::kTfWords + G::kTiWords;
  {
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
    for (int i = tid; i < TW; i += G::kThreads) tab[i] = dtab[i];
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

  constexpr int64_t kBlockWords = frag_words_per_block<bf16>(BS);
  const Buf wb(wfrag + blk * kBlockWords, (uint32_t)(kBlockWords * 16));
  constexpr uint32_t kLayerBytes = (uint32_t)(kBlockWords / 2 * 16);

  // ---- forward: Y^T[entry][k'] -> tile Y[k'][entry]
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4, rho = l16 & 1;
    const uint32_t neg = rho == 0 ? 0x80008000u : 0u;
    f32x4 acc[G::MW][G::KT];
#pragma unroll
    for (int m = 0; m < G::MW; ++m)
#pragma unroll
      for (int n = 0; n < G::KT; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < G::DKS; ++s) {
      constexpr int kHalf = G::DKS / 2;
      const int sigma = s / kHalf, r0 = 32 * (s % kHalf);
      uint4 a[G::MW], bt[G::KT];
#pragma unroll
      for (int m = 0; m < G::MW; ++m) {
        const int c = (16 * (G::MW * wave + m) + l16) >> 1;
        a[m] = *reinterpret_cast<const uint4*>(R + (rho ^ sigma) * G::kPlane + c * G::kLdx + r0 + 8 * g);
        if (sigma) a[m] = xor4(a[m], neg);
      }
#pragma unroll
      for (int n = 0; n < G::KT; ++n) bt[n] = tab[(s * G::KT + n) * 64 + lane];
#pragma unroll
      for (int m = 0; m < G::MW; ++m)
#pragma unroll
        for (int n = 0; n < G::KT; ++n) acc[m][n] = mma_bf16(a[m], bt[n], acc[m][n]);
    }
    __syncthreads();  // X read by every wave
#pragma unroll
    for (int m = 0; m < G::MW; ++m)
#pragma unroll
      for (int n = 0; n < G::KT; ++n) {
        const int kp = 16 * n + l16;
        const int e0 = 16 * (G::MW * wave + m) + 4 * g;
        *reinterpret_cast<uint2*>(R + kp * G::kLdy + e0) =
            make_uint2(cvt_pk(acc[m][n][0], acc[m][n][1]), cvt_pk(acc[m][n][2], acc[m][n][3]));
      }
  }
  __syncthreads();

  // ---- layer 1 (transposed): H1^T[hidden][k'] = relu(W1x^T Y^T + b1) -> tile H[k'][hidden]
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    const uint32_t wvoff = lane * 16u;
    auto wload = [&](int s, int t) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(wb.r, wvoff,
                                                          (uint32_t)((s * G::MT + t) * 64 * 16), 0);
      return make_uint4(v[0], v[1], v[2], v[3]);
    };
    f32x4 acc[G::MW][G::KT];
#pragma unroll
    for (int m = 0; m < G::MW; ++m)
#pragma unroll
      for (int n = 0; n < G::KT; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    uint4 wa[G::MW];
#pragma unroll
    for (int m = 0; m < G::MW; ++m) wa[m] = wload(0, G::MW * wave + m);
#pragma unroll
    for (int s = 0; s < G::WKS; ++s) {
      uint4 wn_[G::MW], yb[G::KT];
      if (s + 1 < G::WKS) {
#pragma unroll
        for (int m = 0; m < G::MW; ++m) wn_[m] = wload(s + 1, G::MW * wave + m);
      }
#pragma unroll
      for (int n = 0; n < G::KT; ++n)
        yb[n] = *reinterpret_cast<const uint4*>(R + (16 * n + l16) * G::kLdy + 32 * s + 8 * g);
#pragma unroll
      for (int m = 0; m < G::MW; ++m)
#pragma unroll
        for (int n = 0; n < G::KT; ++n) acc[m][n] = mma_bf16(wa[m], yb[n], acc[m][n]);
      if (s + 1 < G::WKS) {
#pragma unroll
        for (int m = 0; m < G::MW; ++m) wa[m] = wn_[m];
      }
    }
    float bias[G::MW][4];
#pragma unroll
    for (int m = 0; m < G::MW; ++m) {
      const uint32_t* bp = reinterpret_cast<const uint32_t*>(b1 + (int64_t)blk * BS * 2 +
                                                             16 * (G::MW * wave + m) + 4 * g);
      const uint2 bb = make_uint2(bp[0], bp[1]);
      bias[m][0] = __uint_as_float(bb.x << 16);
      bias[m][1] = __uint_as_float(bb.x & 0xffff0000u);
      bias[m][2] = __uint_as_float(bb.y << 16);
      bias[m][3] = __uint_as_float(bb.y & 0xffff0000u);
    }
    __syncthreads();  // Y read by every wave
#pragma unroll
    for (int m = 0; m < G::MW; ++m)
#pragma unroll
      for (int n = 0; n < G::KT; ++n) {
        const int kp = 16 * n + l16;
        const int e0 = 16 * (G::MW * wave + m) + 4 * g;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = fmaxf(acc[m][n][r] + bias[m][r], 0.f);
        *reinterpret_cast<uint2*>(R + kp * G::kLdy + e0) =
            make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
      }
  }
  __syncthreads();

  // ---- layer 2: O[k'][entry] = softshrink(H W2x + b2) -> planes O[rho][c][k'] (rows k' >=
  //      nkept zero)
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    const uint32_t wvoff = lane * 16u;
    auto wload = [&](int s, int t) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(
          wb.r, wvoff, kLayerBytes + (uint32_t)((s * G::MT + t) * 64 * 16), 0);
      return make_uint4(v[0], v[1], v[2], v[3]);
    };
    f32x4 acc[G::KT][G::MW];
#pragma unroll
    for (int m = 0; m < G::KT; ++m)
#pragma unroll
      for (int n = 0; n < G::MW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    uint4 wv_[G::MW];
#pragma unroll
    for (int n = 0; n < G::MW; ++n) wv_[n] = wload(0, G::MW * wave + n);
#pragma unroll
    for (int s = 0; s < G::WKS; ++s) {
      uint4 wn_[G::MW], ha[G::KT];
      if (s + 1 < G::WKS) {
#pragma unroll
        for (int n = 0; n < G::MW; ++n) wn_[n] = wload(s + 1, G::MW * wave + n);
      }
#pragma unroll
      for (int m = 0; m < G::KT; ++m)
        ha[m] = *reinterpret_cast<const uint4*>(R + (16 * m + l16) * G::kLdy + 32 * s + 8 * g);
#pragma unroll
      for (int m = 0; m < G::KT; ++m)
#pragma unroll
        for (int n = 0; n < G::MW; ++n) acc[m][n] = mma_bf16(ha[m], wv_[n], acc[m][n]);
      if (s + 1 < G::WKS) {
#pragma unroll
        for (int n = 0; n < G::MW; ++n) wv_[n] = wn_[n];
      }
    }
    float bias[G::MW];
#pragma unroll
    for (int n = 0; n < G::MW; ++n) bias[n] = (float)b2[(int64_t)blk * BS * 2 + 16 * (G::MW * wave + n) + l16];
    __syncthreads();  // H read by every wave
#pragma unroll
    for (int m = 0; m < G::KT; ++m) {
      const int k0 = 16 * m + 4 * g;
#pragma unroll
      for (int n = 0; n < G::MW; ++n) {
        const int e = 16 * (G::MW * wave + n) + l16;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = k0 + r < nkept ? softshrink(acc[m][n][r] + bias[n], lam) : 0.f;
        *reinterpret_cast<uint2*>(R + (e & 1) * G::kPlaneO + (e >> 1) * G::kLdo + k0) =
            make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
      }
    }
  }
  __syncthreads();
  if (stage == 2) {  // diagnostic stop: the mixed spectrum back to S, zeros on dropped rows
    for (int it = tid; it < H * BS; it += G::kThreads) {
      const int h = it / BS, c = it - h * BS;
      const int kp = kept_index(h, H, kept_h);
      uint32_t re = 0, im = 0;
      if (kp >= 0) {
        re = *reinterpret_cast<const uint16_t*>(R + c * G::kLdo + kp);
        im = *reinterpret_cast<const uint16_t*>(R + G::kPlaneO + c * G::kLdo + kp);
      }
      cb.st32(re | (im << 16), c * 4u + h * rsb, 0);
    }
    return;
  }

  // ---- inverse: Z^T[entry][h] = A'(O) Ti -> tile Z[h][entry] -> S rows h < H
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4, rho = l16 & 1;
    const uint32_t neg = rho == 1 ? 0x80008000u : 0u;
    const uint4* ti = tab + G::kTfWords;
    f32x4 acc[G::MW][G::HT];
#pragma unroll
    for (int m = 0; m < G::MW; ++m)
#pragma unroll
      for (int n = 0; n < G::HT; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < G::IKS; ++s) {
      // this lane's 8 K rows: (sigma, k') = divmod(32 s + 8 g, KP), within one plane
      const int kap = 32 * s + 8 * g;
      const int sigma = kap >= KP ? 1 : 0, kp0 = kap - sigma * KP;
      uint4 a[G::MW], bt[G::HT];
#pragma unroll
      for (int m = 0; m < G::MW; ++m) {
        const int c = (16 * (G::MW * wave + m) + l16) >> 1;
        a[m] = *reinterpret_cast<const uint4*>(R + (rho ^ sigma) * G::kPlaneO + c * G::kLdo + kp0);
        a[m] = xor4(a[m], sigma ? neg : 0u);
      }
#pragma unroll
      for (int n = 0; n < G::HT; ++n) bt[n] = ti[(s * G::HT + n) * 64 + lane];
#pragma unroll
      for (int m = 0; m < G::MW; ++m)
#pragma unroll
        for (int n = 0; n < G::HT; ++n) acc[m][n] = mma_bf16(a[m], bt[n], acc[m][n]);
    }
    __syncthreads();  // O read by every wave
#pragma unroll
    for (int m = 0; m < G::MW; ++m)
#pragma unroll
      for (int n = 0; n < G::HT; ++n) {
        const int h = 16 * n + l16;
        const int e0 = 16 * (G::MW * wave + m) + 4 * g;
        *reinterpret_cast<uint2*>(R + h * G::kLdy + e0) =
            make_uint2(cvt_pk(acc[m][n][0], acc[m][n][1]), cvt_pk(acc[m][n][2], acc[m][n][3]));
      }
  }
  __syncthreads();
  constexpr int VPR = 2 * BS / 8;
  for (int it = tid; it < H * VPR; it += G::kThreads) {
    const int h = it / VPR, cv = it - h * VPR;
    cb.st128(*reinterpret_cast<const uint4*>(R + h * G::kLdy + cv * 8), cv * 16u + h * rsb, 0);
  }
}

}  // namespace afno
