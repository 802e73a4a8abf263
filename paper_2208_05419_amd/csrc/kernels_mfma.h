// kernels_mfma.h -- bf16 column kernel whose H-axis transforms run on the matrix cores.
//
// For a short column (H <= 96) the length-H DFT is a dense H x H complex matrix, and on
// gfx950 a bf16 MFMA product with it costs about as many matrix-core cycles as one layer of
// the block MLP, while the same transform as a radix FFT on the vector ALUs (fp32, unpacked)
// costs several times more issue slots than the whole MLP.  So all four contractions of a
// column -- forward DFT along H, the two block-MLP layers ("Model Innovations" steps 1-3 of
// AFNO: FFT, block-diagonal complex MLP with ReLU and softshrink, inverse FFT) and the
// inverse DFT -- are MFMA products here, chained through LDS.
//
// Notation: a column holds the spectrum X[h][c] (h < H rows, c < BS complex channels of one
// block), stored as bf16 (re, im) pairs.  "Entry" (c, rho) is the real component rho of
// channel c; entries are interleaved, e = 2 c + rho.  D[i][j] = exp(-2 pi i i j / H) / sqrt(H)
// (symmetric).  The real-ified transform table T has K index (sigma, i) in planes (sigma
// major) and column j:  T[(0, i)][j] = Re D[i][j],  T[(1, i)][j] = Im D[i][j]; zero for
// i >= H or j >= H.
//
//   forward:   Y^T[(c, rho)][k] = sum_(sigma, h) A[(c, rho)][(sigma, h)] T[(sigma, h)][k]
//              A = X(c, rho ^ sigma)[h], negated for (rho, sigma) = (0, 1)
//              (Re D X = Dr Xr - Di Xi, Im D X = Dr Xi + Di Xr)
//   layer 1:   H1^T = relu(W1x^T Y^T + b1)   (W1x: the real-ified complex block weight)
//   layer 2:   O = softshrink(H1 W2x + b2), zeroed outside the H-mode cutoff
//   inverse:   Z^T[(c, rho)][h] = sum_(sigma, k) A'[(c, rho)][(sigma, k)] T[(sigma, k)][h]
//              A' = O(c, rho ^ sigma)[k], negated for (rho, sigma) = (1, 1)
//              (conj(D) O: Re = Dr Or + Di Oi, Im = Dr Oi - Di Or)
//
// The MFMA result layout (lane = output column, four consecutive output rows) makes each
// product's result the next product's 16-byte operand read: Y^T lands in a row-major
// [k][entry] tile, H1^T in a [k][hidden] tile, O (untransposed layer) in planar
// [rho][c][k] planes for the inverse, Z^T goes to HBM as 8-byte (two channel) stores.
#pragma once
#include "kernel_common.h"
#include "kernels_prep.h"

namespace afno {

// An opaque copy of a value: expressions of the copy cannot be tied to expressions of the
// original, so each product phase of a column kernel derives its lane indices afresh rather
// than keeping every phase's index arithmetic live across the kernel.
__device__ __forceinline__ int opq(int v) {
  asm volatile("" : "+v"(v));
  return v;
}


// Geometry for padded height HP (H <= HP, HP a multiple of 32) and block size BS; NWR x NWC
// waves (transposed products: NWR along the channel entries, NWC along the rows; layer 2 the
// other way round).
template <int HP, int BS, int NWR = 4, int NWC = 2>
struct MfmaCol {
  static constexpr int kThreads = 64 * NWR * NWC;
  static constexpr int MT = 2 * BS / 16;   // 16-entry tiles over the 2 BS channel entries
  static constexpr int KT = HP / 16;       // 16-row tiles over H (spectral or spatial rows)
  static constexpr int DKS = 2 * HP / 32;  // k-steps of a transform product (K = 2 HP)
  static constexpr int WKS = 2 * BS / 32;  // k-steps of an MLP product (K = 2 BS)
  // products with channel-entry rows and field-row columns: NWR x NWC waves
  static constexpr int TWM = NWR, TWN = NWC, TMW = MT / TWM, TNW = KT / TWN;
  // layer 2 (field-row rows, channel-entry columns): NWC x NWR waves
  static constexpr int LWM = NWC, LWN = NWR, LMW = KT / LWM, LNW = MT / LWN;
  static_assert(HP % 32 == 0 && BS % 32 == 0, "HP and BS multiples of 32");
  static_assert(MT % TWM == 0 && KT % TWN == 0 && KT % LWM == 0 && MT % LWN == 0, "wave grid");
  static constexpr int kTabWords = DKS * KT * 64;  // 16-byte table fragments
  static constexpr int kTabBytes = kTabWords * 16;
  // planar transposed planes [rho][c][row]: row stride kLdx, plane stride kPlane (bf16);
  // kLdx * 2 bytes is a multiple of 16 and the plane offset lands 32 banks away, so the
  // 16 lanes of a fragment read (8 channels x 2 planes) hit 64 distinct banks
  static constexpr int kLdx = HP + 8;
  static constexpr int kPlane = BS * kLdx + 64;
  // row-major tiles [row][entry]: stride kLdy (bf16)
  static constexpr int kLdy = 2 * BS + 8;
  static constexpr int kXBytes = (kPlane + BS * kLdx) * 2;
  static constexpr int kYBytes = HP * kLdy * 2;
  static constexpr int kRegionBytes = ((kXBytes > kYBytes ? kXBytes : kYBytes) + 15) / 16 * 16;
  static constexpr int kBytes = kTabBytes + kRegionBytes;
};

__device__ __forceinline__ bf16x8 as_frag(uint4 u) {
  union { uint4 u; bf16x8 f; } r;
  r.u = u;
  return r.f;
}
__device__ __forceinline__ uint4 xor4(uint4 u, uint32_t m) {
  return make_uint4(u.x ^ m, u.y ^ m, u.z ^ m, u.w ^ m);
}
typedef float f32x2v __attribute__((ext_vector_type(2)));
typedef bf16 bf16x2v __attribute__((ext_vector_type(2)));
// two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32
__device__ __forceinline__ uint32_t cvt_pk(float lo, float hi) {
  union { bf16x2v v; uint32_t u; } w;
  w.v = __builtin_convertvector((f32x2v){lo, hi}, bf16x2v);
  return w.u;
}
__device__ __forceinline__ f32x4 mma_bf16(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_frag(a), as_frag(b), c, 0, 0, 0);
}

// A transform product over the planar planes P (X for the forward, O for the inverse):
// acc[m][n] += A (channel-entry tile TMW wm + m) x T (row tile TNW wn + n), the A operand
// taking plane rho ^ sigma, negated where rho == neg_rho on the sigma = 1 planes.
template <int HP, int BS, class G = MfmaCol<HP, BS>>
__device__ __forceinline__ void dft_product(const bf16* P, const uint4* tab, int lane, int wm,
                                            int wn, int neg_rho, f32x4 (&acc)[G::TMW][G::TNW]) {
  const int l16 = lane & 15, g = lane >> 4, rho = l16 & 1;
  const uint32_t neg = rho == neg_rho ? 0x80008000u : 0u;
  const bf16* pl0 = P + rho * G::kPlane + 8 * g;          // plane rho (sigma = 0)
  const bf16* pl1 = P + (rho ^ 1) * G::kPlane + 8 * g;    // plane rho ^ 1 (sigma = 1)
#pragma unroll
  for (int m = 0; m < G::TMW; ++m)
#pragma unroll
    for (int n = 0; n < G::TNW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < G::DKS; ++s) {
    constexpr int kHalf = G::DKS / 2;  // k-steps per plane (HP % 32 == 0)
    const int sigma = s / kHalf;
    const int r0 = 32 * (s % kHalf);
    uint4 a[G::TMW], b[G::TNW];
#pragma unroll
    for (int m = 0; m < G::TMW; ++m) {
      const int c = (16 * (G::TMW * wm + m) + l16) >> 1;
      const bf16* p = (sigma ? pl1 : pl0) + c * G::kLdx + r0;
      a[m] = *reinterpret_cast<const uint4*>(p);
      if (sigma) a[m] = xor4(a[m], neg);
    }
#pragma unroll
    for (int n = 0; n < G::TNW; ++n) b[n] = tab[(s * G::KT + G::TNW * wn + n) * 64 + lane];
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) acc[m][n] = mma_bf16(a[m], b[n], acc[m][n]);
  }
}

// grid B * KW * nb (block index fastest), 512 threads, dynamic LDS MfmaCol<HP, BS>::kBytes.
// S: spectrum [B][H][KW][C] complex bf16, updated in place.  wfrag: fragment-ordered
// weights; dtab: transform table (both from prep_operands).  stage: 0 full, 1 stop after the
// forward transform, 2 stop after the MLP (the column goes back to S as it is).
template <int HP, int BS, int NWR = 4, int NWC = 2>
__global__ void __launch_bounds__(64 * NWR * NWC) __attribute__((amdgpu_waves_per_eu(NWR * NWC / 2)))
column_mfma(bf16* __restrict__ S, const uint4* __restrict__ wfrag, const uint4* __restrict__ dtab,
            const bf16* __restrict__ b1, const bf16* __restrict__ b2, int H, int C, int KW,
            int nb, int kept_h, float lam, int stage) {
  typedef MfmaCol<HP, BS, NWR, NWC> G;
  extern __shared__ uint4 smem_mfma[];
  uint4* tab = smem_mfma;
  bf16* R = reinterpret_cast<bf16*>(reinterpret_cast<char*>(smem_mfma) + G::kTabBytes);
  const int tid = threadIdx.x, lane = tid & 63;  // the products take their own lane indices
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  const int blk = blockIdx.x % nb;  // consecutive workgroups -> different XCDs -> blocks
  const int rest = blockIdx.x / nb;
  const int kw = rest % KW;
  const int64_t b = rest / KW;
  bf16* col = S + ((b * H) * KW + kw) * (int64_t)C * 2 + (int64_t)blk * BS * 2;
  const uint32_t rsb = (uint32_t)KW * (uint32_t)C * 4;  // bytes per row of S
  const Buf cb(col, buf_bytes((uint64_t)H * rsb));

  // ---- transform table and the column into LDS; the column as planar transposed planes
  //      X[rho][c][h] (rows h >= H zero), from 8 rows x 1 channel per task
  constexpr int XT = BS * (HP / 8);
  constexpr int XR = (XT + G::kThreads - 1) / G::kThreads;
  constexpr int TR = (G::kTabWords + G::kThreads - 1) / G::kThreads;
  {
    uint32_t xv[XR][8];
#pragma unroll
    for (int u = 0; u < XR; ++u) {
      const int task = tid + u * G::kThreads;
      const int c = task % BS, r0 = 8 * (task / BS);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // branch-free: rows outside the column load its first word and are zeroed
        const bool ok = task < XT && r0 + e < H;
        const uint32_t wv = cb.ld32(ok ? c * 4u + (uint32_t)(r0 + e) * rsb : 0u, 0);
        xv[u][e] = ok ? wv : 0u;
      }
    }
    uint4 tv[TR];
#pragma unroll
    for (int u = 0; u < TR; ++u) tv[u] = dtab[min(tid + u * G::kThreads, G::kTabWords - 1)];
#pragma unroll
    for (int u = 0; u < TR; ++u) {
      const int i = tid + u * G::kThreads;
      if (i < G::kTabWords) tab[i] = tv[u];
    }
#pragma unroll
    for (int u = 0; u < XR; ++u) {
      const int task = tid + u * G::kThreads;
      if (task < XT) {
        const int c = task % BS, r0 = 8 * (task / BS);
        uint4 re, im;  // low halves (re) and high halves (im) of 8 consecutive rows
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

  const int twm = wave / G::TWN, twn = wave % G::TWN;
  const int lwm = wave / G::LWN, lwn = wave % G::LWN;
  constexpr int64_t kBlockWords = frag_words_per_block<bf16>(BS);
  const Buf wb(wfrag + blk * kBlockWords, (uint32_t)(kBlockWords * 16));
  constexpr uint32_t kLayerBytes = (uint32_t)(kBlockWords / 2 * 16);
  const uint32_t wvoff = lane * 16u;
  auto wload = [&](uint32_t layer_off, int s, int t) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(wb.r, wvoff,
                                                        layer_off + (uint32_t)((s * G::MT + t) * 64 * 16), 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
  };

  // ---- forward transform: Y^T = A(X) T -> tile Y[k][entry] (scaled by 1/sqrt(H) via T)
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    dft_product<HP, BS, G>(R, tab, lane, twm, twn, 0, acc);
    __syncthreads();  // every wave has read its X fragments
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
  if (stage == 1) {  // diagnostic stop: spectrum rows back to S
    constexpr int VPR = 2 * BS / 8;
    for (int it = tid; it < H * VPR; it += G::kThreads) {
      const int h = it / VPR, cv = it - h * VPR;
      cb.st128(*reinterpret_cast<const uint4*>(R + h * G::kLdy + cv * 8), cv * 16u + h * rsb, 0);
    }
    return;
  }

  // ---- layer 1 (transposed): H1^T[hidden][k] = relu(W1x^T Y^T + b1) -> tile H[k][hidden]
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    uint4 wa[G::TMW];
#pragma unroll
    for (int m = 0; m < G::TMW; ++m) wa[m] = wload(0, 0, G::TMW * twm + m);
#pragma unroll
    for (int s = 0; s < G::WKS; ++s) {
      uint4 wn_[G::TMW], yb[G::TNW];
      if (s + 1 < G::WKS) {
#pragma unroll
        for (int m = 0; m < G::TMW; ++m) wn_[m] = wload(0, s + 1, G::TMW * twm + m);
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
    float bias[G::TMW][4];
#pragma unroll
    for (int m = 0; m < G::TMW; ++m) {
      const uint32_t* bp = reinterpret_cast<const uint32_t*>(b1 + (int64_t)blk * BS * 2 +
                                                             16 * (G::TMW * twm + m) + 4 * g);
      const uint2 bb = make_uint2(bp[0], bp[1]);  // the biases are only 4-byte aligned
      bias[m][0] = __uint_as_float(bb.x << 16);
      bias[m][1] = __uint_as_float(bb.x & 0xffff0000u);
      bias[m][2] = __uint_as_float(bb.y << 16);
      bias[m][3] = __uint_as_float(bb.y & 0xffff0000u);
    }
    __syncthreads();  // every wave has read its Y fragments
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) {
        const int k = 16 * (G::TNW * twn + n) + l16;
        const int e0 = 16 * (G::TMW * twm + m) + 4 * g;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = fmaxf(acc[m][n][r] + bias[m][r], 0.f);
        *reinterpret_cast<uint2*>(R + k * G::kLdy + e0) =
            make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
      }
  }
  __syncthreads();

  // ---- layer 2: O[k][entry] = softshrink(H W2x + b2), cutoff -> planes O[rho][c][k]
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::LMW][G::LNW];
#pragma unroll
    for (int m = 0; m < G::LMW; ++m)
#pragma unroll
      for (int n = 0; n < G::LNW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    uint4 wb_[G::LNW];
#pragma unroll
    for (int n = 0; n < G::LNW; ++n) wb_[n] = wload(kLayerBytes, 0, G::LNW * lwn + n);
#pragma unroll
    for (int s = 0; s < G::WKS; ++s) {
      uint4 wn_[G::LNW], ha[G::LMW];
      if (s + 1 < G::WKS) {
#pragma unroll
        for (int n = 0; n < G::LNW; ++n) wn_[n] = wload(kLayerBytes, s + 1, G::LNW * lwn + n);
      }
#pragma unroll
      for (int m = 0; m < G::LMW; ++m) {
        const int k = 16 * (G::LMW * lwm + m) + l16;
        ha[m] = *reinterpret_cast<const uint4*>(R + k * G::kLdy + 32 * s + 8 * g);
      }
#pragma unroll
      for (int m = 0; m < G::LMW; ++m)
#pragma unroll
        for (int n = 0; n < G::LNW; ++n) acc[m][n] = mma_bf16(ha[m], wb_[n], acc[m][n]);
      if (s + 1 < G::WKS) {
#pragma unroll
        for (int n = 0; n < G::LNW; ++n) wb_[n] = wn_[n];
      }
    }
    float bias[G::LNW];
#pragma unroll
    for (int n = 0; n < G::LNW; ++n) bias[n] = (float)b2[(int64_t)blk * BS * 2 + 16 * (G::LNW * lwn + n) + l16];
    // every row kept (padding rows h >= H meet zero rows of T in the inverse)
    const bool all_rows = kept_h > H / 2;
    __syncthreads();  // every wave has read its H fragments
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
        for (int r = 0; r < 4; ++r) v[r] = keep[r] ? softshrink(acc[m][n][r] + bias[n], lam) : 0.f;
        *reinterpret_cast<uint2*>(R + (e & 1) * G::kPlane + (e >> 1) * G::kLdx + k0) =
            make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
      }
    }
  }
  __syncthreads();
  if (stage == 2) {  // diagnostic stop: mixed spectrum rows back to S
    for (int it = tid; it < H * BS; it += G::kThreads) {
      const int h = it / BS, c = it - h * BS;
      const uint32_t re = *reinterpret_cast<const uint16_t*>(R + c * G::kLdx + h);
      const uint32_t im = *reinterpret_cast<const uint16_t*>(R + G::kPlane + c * G::kLdx + h);
      cb.st32(re | (im << 16), c * 4u + h * rsb, 0);
    }
    return;
  }

  // ---- inverse transform: Z^T = A'(O) T -> tile Z[h][entry] -> S rows h < H in 16-byte
  //      vectors (whole row segments per store instruction)
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    dft_product<HP, BS, G>(R, tab, lane, twm, twn, 1, acc);
    __syncthreads();  // every wave has read its O fragments
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
  for (int it = tid; it < H * VPR; it += G::kThreads) {
    const int h = it / VPR, cv = it - h * VPR;
    cb.st128(*reinterpret_cast<const uint4*>(R + h * G::kLdy + cv * 8), cv * 16u + h * rsb, 0);
  }
}

}  // namespace afno
