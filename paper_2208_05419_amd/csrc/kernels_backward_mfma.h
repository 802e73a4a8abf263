// kernels_backward_mfma.h -- bf16 backward column kernel with every contraction on the
// matrix cores (short columns, H <= 96, block sizes 32 / 64 / 96).
//
// The backward column pass of the filter (the transposes of "Model Innovations" steps 1-3,
// taken in reverse) chains seven MFMA products through one LDS region, in the forward
// column kernel's geometry (MfmaCol) and with its real-ified operands: the DFT table T and
// block weights in fragment order.  With W1x, W2x the real-ified complex block weights
// (x W1 = x_entries W1x), the gradient of a real-ified product y = x M is dx = dy M^T, and
// M^T is the real-ified conjugate transpose, so the prepared fragments of conj(W)^T serve the
// backward products as the forward's fragments of W serve the forward.
//
//   P1  X^T  = DFT(x column), table hi + lo     -> tile Y[k][entry]        (per-mode X out)
//   P2  H^T  = relu(W1x^T Y^T + b1)             -> tile H[k][hidden], bits v > 0  (h out)
//   P3  O    = H W2x + b2                       -> bits |o| > lam and the row kept
//   P4  dz^T = c_kw DFT(g column), do = masked  -> tile DO[k][entry]       (do out, db2)
//   P5  dh^T = W2x do^T, dv = dh where v > 0    -> tile DV[k][hidden]      (dv out, db1)
//   P6  dX   = DV W1x^T                         -> planes [rho][c][k]
//   P7  Z^T  = IDFT(dX) / c_kw                  -> the gradient spectrum column, in place
//
// Per-mode factors (X, h, do, dv) go to HBM in 8-mode groups: modes[t][blk][G][entry][8],
// G = mode / 8, so that the weight-gradient product loads each matrix-core operand (one
// entry, eight consecutive modes) as one 16-byte word.  A column's modes are
// (b KW + kw) HP .. + HP - 1; rows h >= H hold X = 0 and do = dv = 0.
#pragma once
#include "kernels_mfma.h"

namespace afno {
template <int HP, int BS>
struct MfmaBwd {
  typedef MfmaCol<HP, BS> G;
  static constexpr int NB2 = 2 * BS;
  static constexpr int NW1 = NB2 / 32;  // words of a row's hidden-entry bits
  static constexpr int NW2 = HP / 32;   // words of an entry's mode bits
  static constexpr int kMaskWords = HP * NW1 + NB2 * NW2;
  static constexpr int kBytes = G::kTabBytes + G::kRegionBytes + kMaskWords * 4;
};

// The DFT table's rounding remainders: the same words as dft_table_word with each entry
// v replaced by bf16(v - bf16(v)), so that T_hi + T_lo carries T to about 2^-16.  The
// spectrum that decides the two masks is taken with both: its error is then the bf16
// storage rounding alone (as with the vector-ALU FFT), not the table's 2^-9.
__device__ __forceinline__ uint4 dft_table_word_lo(int64_t i, int H, int HP) {
  const int KT = HP / 16;
  const int lane = (int)(i & 63);
  const int64_t f = i >> 6;
  const int t = (int)(f % KT), s = (int)(f / KT);
  const int j = 16 * t + (lane & 15);
  const float sc = 1.0f / sqrtf((float)H);
  union { uint4 u; bf16 h[8]; } w;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int kap = 32 * s + 8 * (lane >> 4) + e;
    const int sigma = kap / HP, r = kap % HP;
    float v = 0.f;
    if (r < H && j < H) {
      const int m = (r * j) % H;
      float sn, cs;
      sincospif(2.0f * (float)m / (float)H, &sn, &cs);
      v = sigma == 0 ? cs * sc : -sn * sc;
    }
    w.h[e] = (bf16)(v - (float)(bf16)v);
  }
  return w.u;
}

// The backward's independent preparations in one launch, index ranges in turn: the forward
// operands (block weights in fragment order and the DFT table, PrepJob pf), the table's
// rounding remainders, and the conjugate-transposed weights.  The fragments of the
// conjugate-transposed weights read wt1 / wt2 and follow in a launch of their own.
struct BwdPrep {
  PrepJob<bf16> pf;
  const bf16 *w1, *w2;
  bf16 *wt1, *wt2;
  uint4* tab_lo;
  int nb, bs, H, HP;
  int64_t n_pf, n_lo, n_ct;
};

__global__ void __launch_bounds__(256) bwd_prep_kernel(BwdPrep p) {
  const int64_t e1 = p.n_pf, e2 = e1 + p.n_lo, e3 = e2 + p.n_ct;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < e3;
       t += (int64_t)gridDim.x * blockDim.x) {
    if (t < e1)
      prep_operands<bf16>(t, e3, p.pf, nullptr);  // this word only (the next: t + e3 >= e1)
    else if (t < e2)
      p.tab_lo[t - e1] = dft_table_word_lo(t - e1, p.H, p.HP);
    else
      conj_transpose_one<bf16>(t - e2, p.w1, p.w2, p.wt1, p.wt2, p.nb, p.bs);
  }
}

// dft_product's sum accumulated onto acc, the table read from global memory (L2-resident)
template <int HP, int BS>
__device__ __forceinline__ void bwd_dft_acc(const bf16* P, const uint4* __restrict__ tabg, int lane,
                                            int wm, int wn, int neg_rho,
                                            f32x4 (&acc)[MfmaCol<HP, BS>::TMW][MfmaCol<HP, BS>::TNW]) {
  typedef MfmaCol<HP, BS> G;
  const int l16 = lane & 15, g = lane >> 4, rho = l16 & 1;
  const uint32_t neg = rho == neg_rho ? 0x80008000u : 0u;
  const bf16* pl0 = P + rho * G::kPlane + 8 * g;
  const bf16* pl1 = P + (rho ^ 1) * G::kPlane + 8 * g;
  // one k-step at a time: the global table words stay few registers
#pragma unroll 1
  for (int s = 0; s < G::DKS; ++s) {
    constexpr int kHalf = G::DKS / 2;
    const int sigma = s / kHalf;
    const int r0 = 32 * (s % kHalf);
    uint4 a[G::TMW], b[G::TNW];
#pragma unroll
    for (int n = 0; n < G::TNW; ++n) b[n] = tabg[(s * G::KT + G::TNW * wn + n) * 64 + lane];
#pragma unroll
    for (int m = 0; m < G::TMW; ++m) {
      const int c = (16 * (G::TMW * wm + m) + l16) >> 1;
      const bf16* p = (sigma ? pl1 : pl0) + c * G::kLdx + r0;
      a[m] = *reinterpret_cast<const uint4*>(p);
      if (sigma) a[m] = xor4(a[m], neg);
    }
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) acc[m][n] = mma_bf16(a[m], b[n], acc[m][n]);
  }
}

// rows h < H of one column (bf16 complex) -> planar planes P[rho][c][h], rows >= H zero
template <int HP, int BS>
__device__ __forceinline__ void bwd_load_planes(bf16* P, const Buf& cb, int H, uint32_t rsb) {
  typedef MfmaCol<HP, BS> G;
  constexpr int XT = BS * (HP / 8);
  constexpr int XR = (XT + G::kThreads - 1) / G::kThreads;
  const int tid = opq((int)threadIdx.x);  // not shared with the other column load's offsets
  uint32_t xv[XR][8];
#pragma unroll
  for (int u = 0; u < XR; ++u) {
    const int task = tid + u * G::kThreads;
    const int c = task % BS, r0 = 8 * (task / BS);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool ok = task < XT && r0 + e < H;
      // non-temporal: each spectrum column is read once here (Sg is rewritten by P7 anyway)
      const uint32_t wv = cb.ld32<kNonTemporal>(ok ? c * 4u + (uint32_t)(r0 + e) * rsb : 0u, 0);
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
      *reinterpret_cast<uint4*>(P + c * G::kLdx + r0) = re;
      *reinterpret_cast<uint4*>(P + G::kPlane + c * G::kLdx + r0) = im;
    }
  }
}

// Products whose A operand is a weight fragment (rows: output entries) and whose B operand is
// a row-major tile (column k = tile row, K = entries): acc[m][n] over the wave's TMW x TNW
// tiles.  The forward layer-1 shape.
template <int HP, int BS>
__device__ __forceinline__ void bwd_prod_wt(const Buf& wb, uint32_t layer_off, const bf16* Rt,
                                            int lane, int twm, int twn,
                                            f32x4 (&acc)[MfmaCol<HP, BS>::TMW][MfmaCol<HP, BS>::TNW]) {
  typedef MfmaCol<HP, BS> G;
  const int l16 = lane & 15, g = lane >> 4;
  const uint32_t wvoff = lane * 16u;
  auto wload = [&](int s, int t) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(wb.r, wvoff,
                                                        layer_off + (uint32_t)((s * G::MT + t) * 64 * 16), 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
  };
#pragma unroll
  for (int m = 0; m < G::TMW; ++m)
#pragma unroll
    for (int n = 0; n < G::TNW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
  uint4 wa[G::TMW];
#pragma unroll
  for (int m = 0; m < G::TMW; ++m) wa[m] = wload(0, G::TMW * twm + m);
#pragma unroll
  for (int s = 0; s < G::WKS; ++s) {
    uint4 wn_[G::TMW], yb[G::TNW];
    if (s + 1 < G::WKS) {
#pragma unroll
      for (int m = 0; m < G::TMW; ++m) wn_[m] = wload(s + 1, G::TMW * twm + m);
    }
#pragma unroll
    for (int n = 0; n < G::TNW; ++n) {
      const int k = 16 * (G::TNW * twn + n) + l16;
      yb[n] = *reinterpret_cast<const uint4*>(Rt + k * G::kLdy + 32 * s + 8 * g);
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
}

// Products whose A operand is a row-major tile (row k, K = entries) and whose B operand is a
// weight fragment (columns: output entries): acc[m][n] over the wave's LMW x LNW tiles.  The
// forward layer-2 shape.
template <int HP, int BS>
__device__ __forceinline__ void bwd_prod_tw(const Buf& wb, uint32_t layer_off, const bf16* Rt,
                                            int lane, int lwm, int lwn,
                                            f32x4 (&acc)[MfmaCol<HP, BS>::LMW][MfmaCol<HP, BS>::LNW]) {
  typedef MfmaCol<HP, BS> G;
  const int l16 = lane & 15, g = lane >> 4;
  const uint32_t wvoff = lane * 16u;
  auto wload = [&](int s, int t) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(wb.r, wvoff,
                                                        layer_off + (uint32_t)((s * G::MT + t) * 64 * 16), 0);
    return make_uint4(v[0], v[1], v[2], v[3]);
  };
#pragma unroll
  for (int m = 0; m < G::LMW; ++m)
#pragma unroll
    for (int n = 0; n < G::LNW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
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
      ha[m] = *reinterpret_cast<const uint4*>(Rt + k * G::kLdy + 32 * s + 8 * g);
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
}

// A row-major tile [k][entry] (rows k < HP) -> its modes in 8-mode groups: 16 bytes of
// dst[(g0 + q) 2 BS + e][0..7] per task (8 two-byte LDS reads down the column)
template <int HP, int BS>
__device__ __forceinline__ void bwd_modes_out(const bf16* Rt, bf16* dst, int64_t g0) {
  typedef MfmaCol<HP, BS> G;
  constexpr int NB2 = 2 * BS, TASKS = (HP / 8) * NB2;
  const uint16_t* t16 = reinterpret_cast<const uint16_t*>(Rt);
  for (int t = threadIdx.x; t < TASKS; t += G::kThreads) {
    const int q = t / NB2, e = t - q * NB2;
    const uint16_t* p = t16 + (8 * q) * G::kLdy + e;
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)p[(2 * i) * G::kLdy] | ((uint32_t)p[(2 * i + 1) * G::kLdy] << 16);
    // non-temporal: 429 MB at the benchmark shape, read once, later, by the weight product;
    // normal stores would push the spectra the next passes read out of the caches
    typedef uint32_t u4v __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(u4v{w[0], w[1], w[2], w[3]},
                                reinterpret_cast<u4v*>(dst + ((g0 + q) * NB2 + e) * 8));
  }
}

// grid B * KW * nb (block index fastest), 512 threads, dynamic LDS MfmaBwd<HP, BS>::kBytes.
// Sx: spectrum of x; Sg: spectrum of g, replaced by IDFT_H(dX) / c_kw.  wfwd: fragments of
// (w1, w2); wbwd: fragments of (conj(w2)^T, conj(w1)^T); dtab, dtab_lo: the DFT table and its
// rounding remainders.  modes: the four
// per-mode factor tensors (the weight-product pass takes the weight and bias gradients from
// them).
template <int HP, int BS>
__global__ void __launch_bounds__(512) __attribute__((amdgpu_waves_per_eu(4)))
column_bwd_mfma(const bf16* __restrict__ Sx, bf16* __restrict__ Sg, const uint4* __restrict__ wfwd,
                const uint4* __restrict__ wbwd, const uint4* __restrict__ dtab,
                const uint4* __restrict__ dtab_lo, const bf16* __restrict__ b1, const bf16* __restrict__ b2, int H, int C, int KW,
                int nb, int kept_h, float lam, int W, bf16* __restrict__ modes, int64_t mpad) {
  typedef MfmaCol<HP, BS> G;
  typedef MfmaBwd<HP, BS> Q;
  constexpr int NB2 = Q::NB2, NW1 = Q::NW1, NW2 = Q::NW2;
  extern __shared__ uint4 smem_bmfma[];
  uint4* tab = smem_bmfma;
  bf16* R = reinterpret_cast<bf16*>(reinterpret_cast<char*>(smem_bmfma) + G::kTabBytes);
  uint32_t* M1 = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(R) + G::kRegionBytes);
  uint32_t* M2 = M1 + HP * NW1;  // M1[k][NW1]: v > 0;  M2[entry][NW2]: |o| > lam, kept
  const int tid = threadIdx.x;  // each phase takes its own lane indices (opq)
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int twm = wave / G::TWN, twn = wave % G::TWN;
  const int lwm = wave / G::LWN, lwn = wave % G::LWN;

  const int blk = blockIdx.x % nb;
  const int rest = blockIdx.x / nb;
  const int kw = rest % KW;
  const int64_t b = rest / KW;
  const int64_t coff = ((b * H) * KW + kw) * (int64_t)C * 2 + (int64_t)blk * BS * 2;
  const uint32_t rsb = (uint32_t)KW * (uint32_t)C * 4;
  const uint32_t cbytes = buf_bytes((uint64_t)H * rsb);
  constexpr int64_t kBlockWords = frag_words_per_block<bf16>(BS);
  constexpr uint32_t kLayerBytes = (uint32_t)(kBlockWords / 2 * 16);
  // buffer resources are built where used (each holds four scalar registers)
  const float ckw = (kw == 0 || 2 * kw == W) ? 1.f : 2.f;
  const int64_t g0 = (b * KW + kw) * (HP / 8);  // first 8-mode group of the column
  auto tensor = [&](int t) { return modes + ((int64_t)t * nb + blk) * NB2 * mpad; };

  // ---- masks cleared; the table and the x column into LDS
  for (int i = tid; i < Q::kMaskWords; i += G::kThreads) M1[i] = 0u;
  for (int i = tid; i < G::kTabWords; i += G::kThreads) tab[i] = dtab[i];
  bwd_load_planes<HP, BS>(R, Buf(Sx + coff, cbytes), H, rsb);
  __syncthreads();

  // ---- P1: X^T = DFT(x) -> Y[k][entry]
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    dft_product<HP, BS>(R, tab, lane, twm, twn, 0, acc);
    bwd_dft_acc<HP, BS>(R, dtab_lo, lane, twm, twn, 0, acc);
    __syncthreads();
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
  bwd_modes_out<HP, BS>(R, tensor(0), g0);

  // ---- P2: H^T = relu(W1x^T Y^T + b1) -> H[k][hidden]; bits v > 0
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    bwd_prod_wt<HP, BS>(Buf(wfwd + blk * kBlockWords, (uint32_t)(kBlockWords * 16)), 0, R, lane,
                        twm, twn, acc);
    float bias[G::TMW][4];
#pragma unroll
    for (int m = 0; m < G::TMW; ++m) {
      const uint32_t* bp = reinterpret_cast<const uint32_t*>(b1 + (int64_t)blk * BS * 2 +
                                                             16 * (G::TMW * twm + m) + 4 * g);
      const uint2 bb = make_uint2(bp[0], bp[1]);
      bias[m][0] = __uint_as_float(bb.x << 16);
      bias[m][1] = __uint_as_float(bb.x & 0xffff0000u);
      bias[m][2] = __uint_as_float(bb.y << 16);
      bias[m][3] = __uint_as_float(bb.y & 0xffff0000u);
    }
    __syncthreads();  // Y read by every wave (products and the X modes)
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) {
        const int k = 16 * (G::TNW * twn + n) + l16;
        const int j0 = 16 * (G::TMW * twm + m) + 4 * g;
        float v[4];
        uint32_t bits = 0u;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float pre = acc[m][n][r] + bias[m][r];
          bits |= (pre > 0.f ? 1u : 0u) << r;
          v[r] = fmaxf(pre, 0.f);
        }
        *reinterpret_cast<uint2*>(R + k * G::kLdy + j0) =
            make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
        if (bits) atomicOr(M1 + k * NW1 + (j0 >> 5), bits << (j0 & 31));
      }
  }
  __syncthreads();
  bwd_modes_out<HP, BS>(R, tensor(1), g0);

  // ---- P3: O = H W2x + b2 -> bits |o| > lam on kept rows
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::LMW][G::LNW];
    bwd_prod_tw<HP, BS>(Buf(wfwd + blk * kBlockWords, (uint32_t)(kBlockWords * 16)), kLayerBytes,
                        R, lane, lwm, lwn, acc);
    const bool all_rows = kept_h > H / 2;
#pragma unroll
    for (int m = 0; m < G::LMW; ++m) {
      const int k0 = 16 * (G::LMW * lwm + m) + 4 * g;
      bool keep[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) keep[r] = k0 + r < H && (all_rows || row_kept(k0 + r, H, kept_h));
#pragma unroll
      for (int n = 0; n < G::LNW; ++n) {
        const int e = 16 * (G::LNW * lwn + n) + l16;
        const float bias = (float)b2[(int64_t)blk * BS * 2 + e];
        uint32_t bits = 0u;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          bits |= (keep[r] && fabsf(acc[m][n][r] + bias) > lam ? 1u : 0u) << r;
        if (bits) atomicOr(M2 + e * NW2 + (k0 >> 5), bits << (k0 & 31));
      }
    }
  }
  __syncthreads();  // H read by every wave; both masks complete

  // ---- P4: dz^T = c_kw DFT(g), do = dz masked -> DO[k][entry]
  bwd_load_planes<HP, BS>(R, Buf(Sg + coff, cbytes), H, rsb);
  __syncthreads();
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    dft_product<HP, BS>(R, tab, lane, twm, twn, 0, acc);
    __syncthreads();
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) {
        const int k = 16 * (G::TNW * twn + n) + l16;
        const int e0 = 16 * (G::TMW * twm + m) + 4 * g;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool on = (M2[(e0 + r) * NW2 + (k >> 5)] >> (k & 31)) & 1u;
          v[r] = on ? acc[m][n][r] * ckw : 0.f;
        }
        *reinterpret_cast<uint2*>(R + k * G::kLdy + e0) =
            make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
      }
  }
  __syncthreads();
  bwd_modes_out<HP, BS>(R, tensor(2), g0);

  // ---- P5: dh^T = W2x do^T, dv = dh where v > 0 -> DV[k][hidden]
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    bwd_prod_wt<HP, BS>(Buf(wbwd + blk * kBlockWords, (uint32_t)(kBlockWords * 16)), 0, R, lane,
                        twm, twn, acc);
    __syncthreads();  // DO read by every wave (products, modes)
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) {
        const int k = 16 * (G::TNW * twn + n) + l16;
        const int j0 = 16 * (G::TMW * twm + m) + 4 * g;
        const uint32_t bits = M1[k * NW1 + (j0 >> 5)] >> (j0 & 31);
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = (bits >> r) & 1u ? acc[m][n][r] : 0.f;
        *reinterpret_cast<uint2*>(R + k * G::kLdy + j0) =
            make_uint2(cvt_pk(v[0], v[1]), cvt_pk(v[2], v[3]));
      }
  }
  __syncthreads();
  bwd_modes_out<HP, BS>(R, tensor(3), g0);

  // ---- P6: dX = DV W1x^T -> planes [rho][c][k]
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::LMW][G::LNW];
    bwd_prod_tw<HP, BS>(Buf(wbwd + blk * kBlockWords, (uint32_t)(kBlockWords * 16)), kLayerBytes,
                        R, lane, lwm, lwn, acc);
    __syncthreads();  // DV read by every wave
#pragma unroll
    for (int m = 0; m < G::LMW; ++m) {
      const int k0 = 16 * (G::LMW * lwm + m) + 4 * g;
#pragma unroll
      for (int n = 0; n < G::LNW; ++n) {
        const int e = 16 * (G::LNW * lwn + n) + l16;
        *reinterpret_cast<uint2*>(R + (e & 1) * G::kPlane + (e >> 1) * G::kLdx + k0) =
            make_uint2(cvt_pk(acc[m][n][0], acc[m][n][1]), cvt_pk(acc[m][n][2], acc[m][n][3]));
      }
    }
  }
  __syncthreads();

  // ---- P7: Z^T = IDFT(dX) / c_kw -> Z[h][entry] -> the column of Sg
  {
    const int lane = opq((int)threadIdx.x) & 63, l16 = lane & 15, g = lane >> 4;
    f32x4 acc[G::TMW][G::TNW];
    dft_product<HP, BS>(R, tab, lane, twm, twn, 1, acc);
    __syncthreads();
    const float inv_c = 1.f / ckw;
#pragma unroll
    for (int m = 0; m < G::TMW; ++m)
#pragma unroll
      for (int n = 0; n < G::TNW; ++n) {
        const int h = 16 * (G::TNW * twn + n) + l16;
        const int e0 = 16 * (G::TMW * twm + m) + 4 * g;
        *reinterpret_cast<uint2*>(R + h * G::kLdy + e0) =
            make_uint2(cvt_pk(acc[m][n][0] * inv_c, acc[m][n][1] * inv_c),
                       cvt_pk(acc[m][n][2] * inv_c, acc[m][n][3] * inv_c));
      }
  }
  __syncthreads();
  constexpr int VPR = 2 * BS / 8;
  const Buf cg(Sg + coff, cbytes);
  for (int it = tid; it < H * VPR; it += G::kThreads) {
    const int h = it / VPR, cv = it - h * VPR;
    cg.st128(*reinterpret_cast<const uint4*>(R + h * G::kLdy + cv * 8), cv * 16u + h * rsb, 0);
  }
}

}  // namespace afno
