// kernels_fast.h -- size-specialised kernels of the AFNO filter.
//
// The same three HBM passes as kernels_generic.h, with every transform length fixed
// at compile time and split as N = N1 * N2 into two register-resident DFT stages
// (dft_reg.h) around one exchange through LDS:
//   n = n1 + N1 n2, k = k2 + N2 k1:
//   X[k2 + N2 k1] = sum_n1 w_N1^(n1 k1) [ w_N^(n1 k2) sum_n2 x[n1 + N1 n2] w_N2^(n2 k2) ],
// so a thread loads N2 strided inputs straight from HBM into registers, takes an
// N2-point DFT, applies the twiddles w_N^(n1 k2), writes to LDS; after one barrier a
// thread gathers N1 values and takes the N1-point DFT.  Channels are on the lanes, so
// every global access of a wave covers consecutive channels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "afno_internal.h"
#include "dft_reg.h"
#include "kernel_common.h"
#include "kernels_prep.h"

namespace afno {

// tw[m] = exp(-2 pi i m / N), m in [0, N), from double-precision sincospi (no barrier)
template <int N, int NT>
__device__ __forceinline__ void fill_roots(float2* tw) {
  for (int m = threadIdx.x; m < N; m += NT) {
    double s, c;
    sincospi(2.0 * (double)m / (double)N, &s, &c);
    tw[m] = make_float2((float)c, (float)(-s));
  }
}

// v * w^m (forward) or v * conj(w)^m (inverse).  The two-stage transforms pass m = j k2
// with j < N1 and k2 < N2, so m < N1 N2 needs no reduction.
template <bool INV>
__device__ __forceinline__ float2 twiddle(float2 v, const float2* tw, int m) {
  float2 w = tw[m];
  if (INV) w.y = -w.y;
  return c_mul(v, w);
}

// two consecutive elements of T in their storage form, and their widening to float
template <typename T> struct Raw2;
template <> struct Raw2<float> { typedef float2 type; };
template <> struct Raw2<bf16> { typedef uint32_t type; };
__device__ __forceinline__ float2 ld_raw2(const float* p) { return *reinterpret_cast<const float2*>(p); }
__device__ __forceinline__ uint32_t ld_raw2(const bf16* p) { return *reinterpret_cast<const uint32_t*>(p); }
__device__ __forceinline__ float2 widen2(float2 v) { return v; }
__device__ __forceinline__ float2 widen2(uint32_t v) {
  return make_float2(__uint_as_float(v << 16), __uint_as_float(v & 0xffff0000u));
}

// complex values of storage type T through a buffer descriptor (byte offsets)
template <typename T> struct CBuf;
template <> struct CBuf<bf16> {
  Buf b;
  __device__ __forceinline__ CBuf(const bf16* base, uint32_t bytes) : b(base, bytes) {}
  __device__ __forceinline__ float2 ld(uint32_t voff, uint32_t soff) const {
    return unpack_c(b.ld32(voff, soff), (const bf16*)nullptr);
  }
  __device__ __forceinline__ void st(uint32_t voff, uint32_t soff, float2 z) const {
    b.st32(pack_c(z, (const bf16*)nullptr), voff, soff);
  }
};
template <> struct CBuf<float> {
  Buf b;
  __device__ __forceinline__ CBuf(const float* base, uint32_t bytes) : b(base, bytes) {}
  __device__ __forceinline__ float2 ld(uint32_t voff, uint32_t soff) const {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(b.r, voff, soff, 0);
    return make_float2(__uint_as_float(v[0]), __uint_as_float(v[1]));
  }
  __device__ __forceinline__ void st(uint32_t voff, uint32_t soff, float2 z) const {
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    u2 v = {__float_as_uint(z.x), __float_as_uint(z.y)};
    __builtin_amdgcn_raw_buffer_store_b64(v, b.r, voff, soff, 0);
  }
};

// two consecutive real channels (c, c+1) through a buffer, as the complex value x_c + i x_{c+1}
__device__ __forceinline__ float2 ld_pair(const Buf& b, const float*, uint32_t voff, uint32_t soff) {
  const uint2 v = b.ld64(voff, soff);
  return make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
}
__device__ __forceinline__ float2 ld_pair(const Buf& b, const bf16*, uint32_t voff, uint32_t soff) {
  return widen2(b.ld32(voff, soff));
}
__device__ __forceinline__ void st_pair(const Buf& b, const float*, uint32_t voff, uint32_t soff, float2 v) {
  b.st64(make_uint2(__float_as_uint(v.x), __float_as_uint(v.y)), voff, soff);
}
__device__ __forceinline__ void st_pair(const Buf& b, const bf16*, uint32_t voff, uint32_t soff, float2 v) {
  b.st32(pack_c(v, (const bf16*)nullptr), voff, soff);
}
__device__ __forceinline__ typename Raw2<float>::type ld_raw_pair(const Buf& b, const float*, uint32_t voff, uint32_t soff) {
  return ld_pair(b, (const float*)nullptr, voff, soff);
}
__device__ __forceinline__ typename Raw2<bf16>::type ld_raw_pair(const Buf& b, const bf16*, uint32_t voff, uint32_t soff) {
  return b.ld32(voff, soff);
}
// two complex values (re, im of channel c, re, im of channel c+1)
__device__ __forceinline__ float4 ld_cpair(const Buf& b, const float*, uint32_t voff, uint32_t soff) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b128(b.r, voff, soff, 0);
  return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]), __uint_as_float(v[3]));
}
__device__ __forceinline__ float4 ld_cpair(const Buf& b, const bf16*, uint32_t voff, uint32_t soff) {
  const uint2 v = b.ld64(voff, soff);
  const float2 a = widen2(v.x), c = widen2(v.y);
  return make_float4(a.x, a.y, c.x, c.y);
}
__device__ __forceinline__ void st_cpair(const Buf& b, const float*, uint32_t voff, uint32_t soff, float4 v) {
  b.st128(make_uint4(__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)), voff, soff);
}
__device__ __forceinline__ void st_cpair(const Buf& b, const bf16*, uint32_t voff, uint32_t soff, float4 v) {
  b.st64(make_uint2(pack_c(make_float2(v.x, v.y), (const bf16*)nullptr),
                    pack_c(make_float2(v.z, v.w), (const bf16*)nullptr)), voff, soff);
}

// X_c = (Z[k] + conj Z[W-k]) s,  X_{c+1} = (Z[k] - conj Z[W-k]) s / i  with s = 1/(2 sqrt W)
__device__ __forceinline__ float4 split_pair(float2 z, float2 zm, float s) {
  return make_float4((z.x + zm.x) * s, (z.y - zm.y) * s, (z.y + zm.y) * s, (zm.x - z.x) * s);
}

// ------------------------------------------------------------------ W-axis slices

// Workgroup g -> (row b H + h, first channel c0) of a W-axis kernel over nrows rows of
// nchunk slices of 2 NP channels.  A slice narrower than a 128-byte L2 line (bf16 with
// 2 NP = 32 channels: 64 bytes per position) shares each line with the next slice, and
// consecutive workgroups land on different XCDs, each with its own L2; so workgroups g and
// g + 8, which the hardware deals to the same XCD (workgroups go to the 8 XCDs in turn),
// take the two slices of one line, and each line is fetched into one L2 only.  That grid
// is a multiple of 16 (row_grid); workgroups past the last slice pair get no slice.
template <int NP, int ES>
__host__ __device__ constexpr bool row_slices_paired(int nchunk) {
  return 2 * NP * ES < 128 && nchunk % 2 == 0;
}
template <int NP, int ES>
__host__ __device__ inline int64_t row_grid(int64_t nrows, int nchunk) {
  return row_slices_paired<NP, ES>(nchunk) ? (nrows * nchunk + 15) / 16 * 16 : nrows * nchunk;
}
template <int NP, int ES>
__device__ __forceinline__ bool row_slice(int g, int nchunk, int64_t nrows, int64_t& row, int& c0) {
  if (row_slices_paired<NP, ES>(nchunk)) {
    const int pairs = nchunk / 2;
    const int64_t unit = (int64_t)(g >> 4) * 8 + (g & 7);
    if (unit >= nrows * pairs) return false;
    row = unit / pairs;
    c0 = (int)(2 * (unit % pairs) + ((g >> 3) & 1)) * (2 * NP);
    return true;
  }
  row = g / nchunk;
  c0 = (g % nchunk) * (2 * NP);
  return true;
}

// ------------------------------------------------------------------ W-axis forward

// grid pj.nprep (a multiple of 8: the preparation job's workgroups, dispatched first so that
// their longer tasks overlap the transforms) + row_grid(B H, C / (2 NP)), block NP * N1.  NP
// complex signals (2 NP channels) per workgroup; signal p of thread t = t % NP.
template <typename T, int W, int N1, int N2, int NP>
__global__ void __launch_bounds__(NP * N1)
row_r2c_fast(const T* __restrict__ x, T* __restrict__ S, int C, int KW, float scale,
             int64_t nrows, PrepJob<T> pj) {
  static_assert(N1 * N2 == W && W % 2 == 0, "W = N1 N2, even");
  static_assert(N2 * N1 * NP >= 96, "room for the table's roots");
  constexpr int NT = NP * N1;
  __shared__ float2 F[N2 * N1 * NP];
  __shared__ float2 tw[W];
  if ((int)blockIdx.x < pj.nprep) {  // the column kernel's operands
    if (pj.tout && pj.kept_h >= 0) dft_roots(F, pj.H);
    prep_operands<T>((int64_t)blockIdx.x * NT + threadIdx.x, (int64_t)pj.nprep * NT, pj, F);
    return;
  }
  const int tid = threadIdx.x;
  // the workgroup's row b H + h and channel slice (pj.nprep is a multiple of 8, so workgroup
  // g keeps its XCD: consecutive workgroups go to consecutive XCDs)
  int64_t row;
  int c0;
  if (!row_slice<NP, (int)sizeof(T)>(blockIdx.x - pj.nprep, C / (2 * NP), nrows, row, c0)) return;
  constexpr uint32_t es = sizeof(T);
  const uint32_t xrow = (uint32_t)C * es;        // bytes between consecutive w
  const uint32_t srow = (uint32_t)C * 2 * es;    // bytes between consecutive kw of S
  const Buf xb(x + row * (int64_t)W * C + c0, (uint32_t)W * xrow);
  const Buf sb(S + (row * (int64_t)KW * C + c0) * 2, (uint32_t)KW * srow);
  {
    const int p = tid % NP, j = tid / NP;
    const uint32_t voff = 2 * p * es + j * xrow;
    float2 v[N2];
#pragma unroll
    for (int t = 0; t < N2; ++t) v[t] = ld_pair(xb, (const T*)nullptr, voff, N1 * t * xrow);
    fill_roots<W, NT>(tw);
    __syncthreads();
    DftReg<N2, false>::run(v);
#pragma unroll
    for (int k2 = 0; k2 < N2; ++k2)
      F[(k2 * N1 + j) * NP + p] = k2 == 0 ? v[0] : twiddle<false>(v[k2], tw, j * k2);
  }
  __syncthreads();
  // One task per pair of residues {q, N2 - q}: it holds Z[k] and its partner Z[W - k]
  // for every k of both residue classes, so the two real spectra separate in registers.
  constexpr int NPT = N2 / 2 + 1;
  for (int task = tid; task < NP * NPT; task += NT) {
    const int p = task % NP, q = task / NP;
    const int qa = q, qb = (N2 - q) % N2;
    float2 a[N1], b[N1];
#pragma unroll
    for (int j = 0; j < N1; ++j) {
      a[j] = F[(qa * N1 + j) * NP + p];
      b[j] = F[(qb * N1 + j) * NP + p];
    }
    DftReg<N1, false>::run(a);  // a[k1] = Z[qa + N2 k1]
    DftReg<N1, false>::run(b);  // b[k1] = Z[qb + N2 k1]
    const uint32_t va = 4 * p * es + qa * srow, vb = 4 * p * es + qb * srow;
#pragma unroll
    for (int k1 = 0; k1 < N1; ++k1) {
      // partner of qa + N2 k1: N2 (N1 - k1) for q = 0, else qb + N2 (N1 - 1 - k1)
      const int ka = qa + N2 * k1;
      const float2 zam = (q == 0) ? a[(N1 - k1) % N1] : b[N1 - 1 - k1];
      if (ka <= W / 2 && ka < KW)
        st_cpair(sb, (const T*)nullptr, va, N2 * k1 * srow, split_pair(a[k1], zam, scale));
      const int kb = qb + N2 * k1;
      if (qb != qa && kb <= W / 2 && kb < KW)
        st_cpair(sb, (const T*)nullptr, vb, N2 * k1 * srow, split_pair(b[k1], a[N1 - 1 - k1], scale));
    }
  }
}

// ------------------------------------------------------------------ W-axis inverse + residual

// grid row_grid(B H, C / (2 NP)), block NP * N1.  mode 0: out = x + y (dtype T); mode 1:
// dst = y.
// Global traffic goes through LDS in 16-byte vectors: the kept half spectrum of the
// workgroup's 2 NP channels is staged once (each stored bin feeds both Z[k] and Z[W-k]),
// the residual is prefetched at kernel start, and the output leaves in 16-byte stores.
template <typename T, int W, int N1, int N2, int NP>
__global__ void __launch_bounds__(NP * N1)
row_c2r_fast(const T* __restrict__ S, const T* __restrict__ x, T* __restrict__ out,
             float* __restrict__ dst, int C, int KW, float scale, int mode, int64_t nrows) {
  static_assert(N1 * N2 == W && W % 2 == 0, "W = N1 N2, even");
  constexpr int NT = NP * N1;
  constexpr int HALF = W / 2;
  constexpr uint32_t es = sizeof(T);
  constexpr int XV = 16 / es;                          // channels per 16-byte vector of x / out
  constexpr int XPR = 2 * NP / XV;                     // 16-byte vectors per row of the slice
  constexpr int TX = (W * XPR + NT - 1) / NT;          // residual vectors per thread
  constexpr int SPR = 2 * NP * 2 * es / 16;            // 16-byte vectors per spectrum row
  constexpr int TP2 = (NP * N2 + NT - 1) / NT;         // second-stage tasks per thread
  constexpr int FN = (HALF + 1) * SPR * 2 > W * NP ? (HALF + 1) * SPR * 2 : W * NP;
  __shared__ float2 F[FN];                             // staged spectrum / stage-1 output / y
  __shared__ float2 tw[W];
  const int tid = threadIdx.x;
  int64_t row;
  int c0;
  if (!row_slice<NP, (int)sizeof(T)>(blockIdx.x, C / (2 * NP), nrows, row, c0)) return;
  const uint32_t xrow = (uint32_t)C * es;
  const uint32_t srow = (uint32_t)C * 2 * es;
  const int64_t xbase = row * (int64_t)W * C + c0;
  const Buf xb(x + xbase, (uint32_t)W * xrow);
  const Buf ob(out + xbase, (uint32_t)W * xrow);
  const Buf db(dst + xbase, (uint32_t)W * C * 4);
  const Buf sb(S + (row * (int64_t)KW * C + c0) * 2, (uint32_t)KW * srow);
  uint4* F4 = reinterpret_cast<uint4*>(F);
  // ---- the kept half spectrum of the slice and the residual, 16-byte loads
  {
    uint4 sv[((HALF + 1) * SPR + NT - 1) / NT];
#pragma unroll
    for (int u = 0; u < ((HALF + 1) * SPR + NT - 1) / NT; ++u) {
      const int i = tid + u * NT;
      const int r = i / SPR, v = i % SPR;
      sv[u] = make_uint4(0, 0, 0, 0);
      if (r < KW && r <= HALF) {
        const auto q = __builtin_amdgcn_raw_buffer_load_b128(sb.r, v * 16 + r * srow, 0, 0);
        sv[u] = make_uint4(q[0], q[1], q[2], q[3]);
      }
    }
    fill_roots<W, NT>(tw);
#pragma unroll
    for (int u = 0; u < ((HALF + 1) * SPR + NT - 1) / NT; ++u) {
      const int i = tid + u * NT;
      if (i < (HALF + 1) * SPR) F4[i] = sv[u];  // row r of the stored half at r * SPR
    }
  }
  uint4 xres[TX];
  if (mode == 0) {
#pragma unroll
    for (int u = 0; u < TX; ++u) {
      const int i = min(tid + u * NT, W * XPR - 1);
      const auto q = __builtin_amdgcn_raw_buffer_load_b128(xb.r, (i % XPR) * 16 + (i / XPR) * xrow, 0, 0);
      xres[u] = make_uint4(q[0], q[1], q[2], q[3]);
    }
  }
  __syncthreads();
  // ---- first stage: task (p, j) gathers Z[j + N1 t] from the staged half spectrum
  float2 v[N2];
  const int p = tid % NP, j = tid / NP;
  {
    const char* Fb = reinterpret_cast<const char*>(F);
#pragma unroll
    for (int t = 0; t < N2; ++t) {
      // Z[k] = Y_c[k] + i Y_{c+1}[k] over the full length: Y[W - k] = conj Y[k]; only the
      // real parts of the k = 0 and k = W/2 bins count
      const int k = j + N1 * t;
      const int kk = k <= HALF ? k : W - k;
      float4 y;
      if constexpr (es == 2) {
        const uint2 q = *reinterpret_cast<const uint2*>(Fb + kk * SPR * 16 + p * 8);
        const float2 a = widen2(q.x), c = widen2(q.y);
        y = make_float4(a.x, a.y, c.x, c.y);
      } else {
        y = *reinterpret_cast<const float4*>(Fb + kk * SPR * 16 + p * 16);
      }
      v[t] = (k == 0 || k == HALF) ? make_float2(y.x, y.z)
             : (k < HALF ? make_float2(y.x - y.w, y.y + y.z) : make_float2(y.x + y.w, y.z - y.y));
    }
  }
  __syncthreads();  // the staged spectrum has been read; F is overwritten below
  DftReg<N2, true>::run(v);
#pragma unroll
  for (int k2 = 0; k2 < N2; ++k2)
    F[(k2 * N1 + j) * NP + p] = k2 == 0 ? v[0] : twiddle<true>(v[k2], tw, j * k2);
  __syncthreads();
  // ---- second stage: task (p, k2) -> y at w = k2 + N2 k1, held until F is free
  float2 yv[TP2][N1];
#pragma unroll
  for (int u = 0; u < TP2; ++u) {
    const int task = min(tid + u * NT, NP * N2 - 1);
    const int pp = task % NP, k2 = task / NP;
#pragma unroll
    for (int jj = 0; jj < N1; ++jj) yv[u][jj] = F[(k2 * N1 + jj) * NP + pp];
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < TP2; ++u) {
    const int task = tid + u * NT;
    if (task < NP * N2) {
      const int pp = task % NP, k2 = task / NP;
      DftReg<N1, true>::run(yv[u]);  // yv[k1] = z[k2 + N2 k1] = y_c + i y_{c+1}
#pragma unroll
      for (int k1 = 0; k1 < N1; ++k1) F[(k2 + N2 * k1) * NP + pp] = yv[u][k1];  // y[w][pair]
    }
  }
  __syncthreads();
  // ---- out = x + y / sqrt(W) (or dst = y), 16-byte vectors along each row
  if (mode == 0) {
#pragma unroll
    for (int u = 0; u < TX; ++u) {
      const int i = tid + u * NT;
      if (i < W * XPR) {
        const int w = i / XPR, g = i % XPR;
        const float* yr = reinterpret_cast<const float*>(F + w * NP) + g * XV;  // XV channels
        union { uint4 u4; uint32_t w32[4]; } xo, ov;
        xo.u4 = xres[u];
        if constexpr (es == 2) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float2 xv = widen2(xo.w32[e]);
            ov.w32[e] = pack_c(make_float2(xv.x + yr[2 * e] * scale, xv.y + yr[2 * e + 1] * scale),
                               (const bf16*)nullptr);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            ov.w32[e] = __float_as_uint(__uint_as_float(xo.w32[e]) + yr[e] * scale);
        }
        ob.st128(ov.u4, g * 16 + w * xrow, 0);
      }
    }
  } else {
    constexpr int DPR = 2 * NP / 4;  // 16-byte float vectors per row of dst
    for (int i = tid; i < W * DPR; i += NT) {
      const int w = i / DPR, g = i % DPR;
      const float4 y = *reinterpret_cast<const float4*>(reinterpret_cast<const float*>(F + w * NP) + 4 * g);
      db.st128(make_uint4(__float_as_uint(y.x * scale), __float_as_uint(y.y * scale),
                          __float_as_uint(y.z * scale), __float_as_uint(y.w * scale)),
               g * 16 + w * (uint32_t)C * 4, 0);
    }
  }
}

// ------------------------------------------------------------------ column kernel

template <int BS> struct ColShape {
  static constexpr int kThreads = 4 * BS < 64 ? 64 : 4 * BS;  // bs / 16 MFMA waves
};

template <typename T, typename FT, int H, int BS>
struct ColLds {
  static constexpr int kH16 = (H + 15) / 16 * 16;
  static constexpr int kLdt = 2 * BS + (sizeof(T) == 2 ? 8 : 4);
  static constexpr int kTile = kH16 * kLdt * (int)sizeof(T);
  static constexpr int kF = H * BS * 2 * (int)sizeof(FT);
  static constexpr int kRegion = ((kTile > kF ? kTile : kF) + 15) / 16 * 16;
  static constexpr int kBytes = kRegion + H * 8;
};

template <typename FT>
__device__ __forceinline__ void st_f(FT* p, float2 v);
template <> __device__ __forceinline__ void st_f<float>(float* p, float2 v) { st_c(p, v); }
template <> __device__ __forceinline__ void st_f<bf16>(bf16* p, float2 v) { st_c(p, v); }

// Wave grid of the block MLP: WM row groups x WN column groups.  Wave (wm, wn) computes
// MW = MT / WM m-tiles (rows 16 MW wm ...) by NW = (2 BS / 16) / WN n-tiles (real output
// columns 16 NW wn ...).  Two row groups halve the LDS traffic of the A tile (each wave
// reads only its rows) against re-reading each weight column from L2 twice.
template <int NT, int BS, int MT>
struct MlpGrid {
  static constexpr int kWaves = NT / 64;
  static constexpr int WM = (kWaves >= 4 && MT % 2 == 0) ? 2 : 1;
  static constexpr int WN = kWaves / WM;
  static constexpr int MW = MT / WM;
  static constexpr int NW = (2 * BS / 16) / WN;
  static_assert(WM * WN == kWaves && MW * WM == MT && NW * WN * 16 == 2 * BS, "MLP wave grid");
};

// One layer: acc[m][n] = (rows of the wave's m-tile m) x (real-ified complex weight of its
// n-tile n), the weight fragments read from the prepared buffer wb (this block, this
// layer).  Every m-tile is computed (rows outside the cutoff are zeroed by the caller).
template <typename T, int NT, int BS, int MT>
__device__ __forceinline__ void gemm_layer(const T* tile, const Buf& wb, uint32_t layer_off,
                                           int lane, int wm, int wn,
                                           f32x4 (&acc)[MlpGrid<NT, BS, MT>::MW][MlpGrid<NT, BS, MT>::NW]) {
  typedef Mma<T> M;
  typedef MlpGrid<NT, BS, MT> G;
  typedef typename FragWord<T>::type Word;
  constexpr int LDT = 2 * BS + (sizeof(T) == 2 ? 8 : 4);
  constexpr int KSTEPS = 2 * BS / M::kK;
  constexpr int NT16 = 2 * BS / 16;
  constexpr int KCH0 = sizeof(T) == 2 ? 2 : 4;
  constexpr int KCH = KSTEPS < KCH0 ? KSTEPS : KCH0;
  static_assert(KSTEPS % KCH == 0, "k-step chunking");
  const uint32_t voff = lane * (uint32_t)sizeof(Word);
#pragma unroll
  for (int m = 0; m < G::MW; ++m)
#pragma unroll
    for (int n = 0; n < G::NW; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
  const T* arow = tile + (16 * G::MW * wm + (lane & 15)) * LDT;
#pragma unroll 1
  for (int s0 = 0; s0 < KSTEPS; s0 += KCH) {
    typename M::Frag bfr[KCH][G::NW];
#pragma unroll
    for (int s = 0; s < KCH; ++s)
#pragma unroll
      for (int n = 0; n < G::NW; ++n) {
        const uint32_t soff = layer_off + ((s0 + s) * NT16 + wn * G::NW + n) * 64 * (uint32_t)sizeof(Word);
        if constexpr (sizeof(T) == 2) {
          union { uint4 u; typename M::Frag f; } r;
          const auto v = __builtin_amdgcn_raw_buffer_load_b128(wb.r, voff, soff, 0);
          r.u = make_uint4(v[0], v[1], v[2], v[3]);
          bfr[s][n] = r.f;
        } else {
          bfr[s][n] = __uint_as_float(wb.ld32(voff, soff));
        }
      }
#pragma unroll
    for (int s = 0; s < KCH; ++s) {
      typename M::Frag a[G::MW];
#pragma unroll
      for (int m = 0; m < G::MW; ++m) a[m] = M::load_a(arow + 16 * m * LDT, (s0 + s) * M::kK, lane);
#pragma unroll
      for (int m = 0; m < G::MW; ++m)
#pragma unroll
        for (int n = 0; n < G::NW; ++n) acc[m][n] = M::mma(a[m], bfr[s][n], acc[m][n]);
    }
  }
}

// grid B * KW * nb, block NT threads, dynamic LDS ColLds<...>::kBytes.
// WPE: waves per SIMD the register budget must allow (the workgroups per CU that the
// LDS admits times the waves per workgroup, over 4 SIMDs).
// The transform intermediate (FT: float, or bf16 where float would not fit the LDS)
// shares its LDS with the MFMA tile; the passes that switch between the two read all
// of their inputs, synchronise, then write.
// stage: 0 full, 1 stop after the forward transform, 2 stop after the MLP.
template <typename T, typename FT, int H, int N1, int N2, int BS, int WPE, int NT>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(WPE)))
column_fast(T* __restrict__ S, const typename FragWord<T>::type* __restrict__ wfrag,
            const T* __restrict__ b1, const T* __restrict__ b2, int C, int KW, int nb,
            int kept_h, float lam, float scale, int stage) {
  static_assert(N1 * N2 == H, "H = N1 N2");
  static_assert(BS % 16 == 0, "block size multiple of 16");
  typedef ColLds<T, FT, H, BS> L;
  constexpr int MT = L::kH16 / 16;
  constexpr int LDT = L::kLdt;
  extern __shared__ float4 smem_raw[];
  T* tile = reinterpret_cast<T*>(smem_raw);
  FT* F = reinterpret_cast<FT*>(smem_raw);
  float2* tw = reinterpret_cast<float2*>(reinterpret_cast<char*>(smem_raw) + L::kRegion);
  const int tid = threadIdx.x, lane = tid & 63;
  // the wave index is uniform across the wave: held in a scalar register, offsets derived
  // from it can be buffer soffsets
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

  const int blk = blockIdx.x % nb;  // consecutive workgroups -> different XCDs -> blocks
  const int rest = blockIdx.x / nb;
  const int kw = rest % KW;
  const int64_t b = rest / KW;
  const int64_t rs = (int64_t)KW * C * 2;  // row stride of S, elements
  T* col = S + ((b * H) * KW + kw) * (int64_t)C * 2 + (int64_t)blk * BS * 2;
  const uint32_t rsb = (uint32_t)(rs * sizeof(T));  // row stride of S, bytes
  const CBuf<T> cb(col, buf_bytes((uint64_t)H * rsb));

  // ---- forward, first stage: task (c, j): rows j + N1 t of channel c from HBM
  constexpr int TA = (BS * N1 + NT - 1) / NT;
  {
    float2 va[TA][N2];
#pragma unroll
    for (int u = 0; u < TA; ++u) {
      const int task = tid + u * NT;
      if (task < BS * N1) {
        const int c = task % BS, j = task / BS;
#pragma unroll
        for (int t = 0; t < N2; ++t)
          va[u][t] = cb.ld(2 * c * (uint32_t)sizeof(T) + j * rsb, N1 * t * rsb);
      }
    }
    fill_roots<H, NT>(tw);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < TA; ++u) {
      const int task = tid + u * NT;
      if (task < BS * N1) {
        const int c = task % BS, j = task / BS;
        DftReg<N2, false>::run(va[u]);
#pragma unroll
        for (int k2 = 0; k2 < N2; ++k2)
          st_f(F + ((k2 * N1 + j) * BS + c) * 2,
               k2 == 0 ? va[u][0] : twiddle<false>(va[u][k2], tw, j * k2));
      }
    }
  }
  __syncthreads();
  // ---- forward, second stage: task (c, k2) -> spectrum rows k2 + N2 k1 into the tile
  constexpr int TB = (BS * N2 + NT - 1) / NT;
  {
    float2 vb[TB][N1];
#pragma unroll
    for (int u = 0; u < TB; ++u) {
      const int task = tid + u * NT;
      if (task < BS * N2) {
        const int c = task % BS, k2 = task / BS;
#pragma unroll
        for (int j = 0; j < N1; ++j) vb[u][j] = ld_c(F + ((k2 * N1 + j) * BS + c) * 2);
      }
    }
    __syncthreads();  // the tile overwrites F
#pragma unroll
    for (int u = 0; u < TB; ++u) {
      const int task = tid + u * NT;
      if (task < BS * N2) {
        const int c = task % BS, k2 = task / BS;
        DftReg<N1, false>::run(vb[u]);
#pragma unroll
        for (int k1 = 0; k1 < N1; ++k1)
          st_c(tile + (k2 + N2 * k1) * LDT + 2 * c,
               make_float2(vb[u][k1].x * scale, vb[u][k1].y * scale));
      }
    }
    for (int e = tid; e < (L::kH16 - H) * 2 * BS; e += NT)
      tile[(H + e / (2 * BS)) * LDT + e % (2 * BS)] = Store<T>::to(0.f);
  }
  __syncthreads();

  if (stage != 1) {
    // ---- block MLP on the wave grid
    typedef MlpGrid<NT, BS, MT> G;
    const int wm = wave / G::WN, wn = wave % G::WN;
    constexpr int64_t kBlockWords = frag_words_per_block<T>(BS);
    const Buf wb(wfrag + blk * kBlockWords, (uint32_t)(kBlockWords * sizeof(typename FragWord<T>::type)));
    constexpr uint32_t kLayerBytes = (uint32_t)(kBlockWords / 2 * sizeof(typename FragWord<T>::type));
    const T* B1 = b1 + (int64_t)blk * BS * 2;
    const T* B2 = b2 + (int64_t)blk * BS * 2;
    const int col0 = 16 * G::NW * wn + (lane & 15);  // real output column of n-tile 0
    const int row0 = 16 * G::MW * wm + 4 * (lane >> 4);
    const bool all_rows = kept_h > H / 2;  // cutoff keeps every row
    f32x4 acc[G::MW][G::NW];
    gemm_layer<T, NT, BS, MT>(tile, wb, 0, lane, wm, wn, acc);
    float bias[G::NW];
#pragma unroll
    for (int n = 0; n < G::NW; ++n) bias[n] = ld_f(B1 + col0 + 16 * n);
    __syncthreads();  // every wave has read its spectrum rows
#pragma unroll
    for (int m = 0; m < G::MW; ++m)
#pragma unroll
      for (int n = 0; n < G::NW; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          tile[(row0 + 16 * m + r) * LDT + col0 + 16 * n] =
              Store<T>::to(fmaxf(acc[m][n][r] + bias[n], 0.f));
    __syncthreads();  // hidden layer complete
    gemm_layer<T, NT, BS, MT>(tile, wb, kLayerBytes, lane, wm, wn, acc);
#pragma unroll
    for (int n = 0; n < G::NW; ++n) bias[n] = ld_f(B2 + col0 + 16 * n);
    __syncthreads();  // every wave has read its hidden rows
#pragma unroll
    for (int m = 0; m < G::MW; ++m) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = row0 + 16 * m + r;
        const bool keep = all_rows || row_kept(row, H, kept_h);
#pragma unroll
        for (int n = 0; n < G::NW; ++n) {
          const float o = softshrink(acc[m][n][r] + bias[n], lam);
          tile[row * LDT + col0 + 16 * n] = Store<T>::to(keep ? o : 0.f);
        }
      }
    }
    __syncthreads();
  }

  if (stage != 0) {  // diagnostic stop: the tile goes back to S as it is
    constexpr int V = Store<T>::kVec;
    constexpr int VPR = 2 * BS / V;
    for (int it = tid; it < H * VPR; it += NT) {
      const int h = it / VPR, cv = it - h * VPR;
      *reinterpret_cast<uint4*>(col + h * rs + cv * V) =
          *reinterpret_cast<const uint4*>(tile + h * LDT + cv * V);
    }
    return;
  }

  // ---- inverse, first stage: task (c, j): tile rows j + N1 t
  constexpr int TC = (BS * N1 + NT - 1) / NT;
  {
    float2 vc[TC][N2];
#pragma unroll
    for (int u = 0; u < TC; ++u) {
      const int task = tid + u * NT;
      if (task < BS * N1) {
        const int c = task % BS, j = task / BS;
#pragma unroll
        for (int t = 0; t < N2; ++t) vc[u][t] = ld_c(tile + (j + N1 * t) * LDT + 2 * c);
      }
    }
    __syncthreads();  // F overwrites the tile
#pragma unroll
    for (int u = 0; u < TC; ++u) {
      const int task = tid + u * NT;
      if (task < BS * N1) {
        const int c = task % BS, j = task / BS;
        DftReg<N2, true>::run(vc[u]);
#pragma unroll
        for (int k2 = 0; k2 < N2; ++k2)
          st_f(F + ((k2 * N1 + j) * BS + c) * 2,
               k2 == 0 ? vc[u][0] : twiddle<true>(vc[u][k2], tw, j * k2));
      }
    }
  }
  __syncthreads();
  // ---- inverse, second stage: task (c, k2) -> rows k2 + N2 k1 of S
  for (int task = tid; task < BS * N2; task += NT) {
    const int c = task % BS, k2 = task / BS;
    float2 vd[N1];
#pragma unroll
    for (int j = 0; j < N1; ++j) vd[j] = ld_c(F + ((k2 * N1 + j) * BS + c) * 2);
    DftReg<N1, true>::run(vd);
#pragma unroll
    for (int k1 = 0; k1 < N1; ++k1)
      cb.st(2 * c * (uint32_t)sizeof(T) + k2 * rsb, N2 * k1 * rsb,
           make_float2(vd[k1].x * scale, vd[k1].y * scale));
  }
}

}  // namespace afno
