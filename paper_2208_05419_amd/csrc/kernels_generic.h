// kernels_generic.h -- size-generic kernels of the AFNO filter: any H, W of the form
// 2^a 3^b 5^c within the plan limits.  Transforms run as radix-2/3/4/5 Stockham passes
// over LDS (fft_lds.h); the size-specialised kernels of kernels_fast.h replace them for
// the grids the filter is usually run on.
//
// Three passes over HBM, all on one spectrum workspace S [B][H][KW][C] (complex,
// (re, im) interleaved, stored in the filter's dtype; KW = kept_w columns):
//   row_r2c   x -> S       real-to-complex DFT along W of every (b, h, c) line
//                          (FourCastNet, "Implementation Details" (b): R2C transform
//                          batched over batch and channels), scaled 1/sqrt(W)
//   column    S -> S       per (b, kw, channel block): DFT along H, the block complex
//                          MLP on MFMA with bias/ReLU/bias/softshrink/cutoff in the
//                          epilogues, inverse DFT along H ("Model Innovations" steps
//                          1-3; the MLP weights shared by every mode), in place
//   row_c2r   S, x -> out  complex-to-real inverse along W plus the residual add,
//                          rounded once to the dtype
// Two real channels (c, c+1) travel through the W transforms as one complex signal
// z = x_c + i x_{c+1}; their half spectra are separated (forward) and recombined
// (inverse) through the conjugate symmetry of a real signal's spectrum.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "afno_internal.h"
#include "fft_lds.h"
#include "kernel_common.h"

namespace afno {

// ------------------------------------------------------------------ kernel 1: W-axis R2C

// grid (B * H, C / rc), block kRowThreads.  LDS: W x (rc/2) float2 signals + W twiddles.
template <typename T>
__global__ void __launch_bounds__(kRowThreads)
row_r2c_kernel(const T* __restrict__ x, T* __restrict__ S, RowParams p) {
  extern __shared__ float4 smem_raw[];
  float2* buf = reinterpret_cast<float2*>(smem_raw);
  const int np = p.rc / 2;
  float2* tw = buf + (size_t)p.W * np;
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;  // b * H + h
  const int c0 = blockIdx.y * p.rc;

  make_twiddles(tw, p.W);  // synchronises

  // load x[b][h][:][c0 : c0 + rc] as np complex signals of length W
  constexpr int V = Store<T>::kVec;
  const int vpr = p.rc / V;
  const T* xr = x + row * p.W * p.C + c0;
  for (int it = tid; it < p.W * vpr; it += blockDim.x) {
    const int n = it / vpr, cv = it - n * vpr;
    V16 v;
    v.u = *reinterpret_cast<const uint4*>(xr + (int64_t)n * p.C + cv * V);
#pragma unroll
    for (int q = 0; q < V / 2; ++q) {
      float a, b;
      if constexpr (V == 4) { a = v.f[2 * q]; b = v.f[2 * q + 1]; }
      else { a = (float)v.h[2 * q]; b = (float)v.h[2 * q + 1]; }
      buf[n * np + cv * (V / 2) + q] = make_float2(a, b);
    }
  }
  __syncthreads();

  const int sig = tid % np, sub = tid / np, nsub = blockDim.x / np;
  fft_lds<kRowEmax, false>(buf, np, p.rw, sig, sub, nsub, tw);

  // separate the two real channels of each signal and store kw in [0, KW):
  //   X_c = (Z[k] + conj Z[W-k]) / 2,  X_{c+1} = (Z[k] - conj Z[W-k]) / (2i)
  const float sc = 0.5f * p.inv_sqrt_w;
  T* Sr = S + row * (int64_t)p.KW * p.C * 2;
  for (int it = tid; it < p.KW * np; it += blockDim.x) {
    const int k = it / np, q = it - k * np;
    const float2 z = buf[k * np + q];
    const int km = (k == 0) ? 0 : p.W - k;
    const float2 zm = buf[km * np + q];
    const float ar = (z.x + zm.x) * sc, ai = (z.y - zm.y) * sc;
    const float br = (z.y + zm.y) * sc, bi = (zm.x - z.x) * sc;
    T* o = Sr + ((int64_t)k * p.C + c0 + 2 * q) * 2;
    if constexpr (V == 4) {
      *reinterpret_cast<float4*>(o) = make_float4(ar, ai, br, bi);
    } else {
      union { uint2 u; bf16 h[4]; } w;
      w.h[0] = (bf16)ar; w.h[1] = (bf16)ai; w.h[2] = (bf16)br; w.h[3] = (bf16)bi;
      *reinterpret_cast<uint2*>(o) = w.u;
    }
  }
}

// ------------------------------------------------------------------ kernel 3: W-axis C2R + residual

// grid (B * H, C / rc), block kRowThreads.  mode 0: out = x + y in T; mode 1: dst = y (float).
template <typename T>
__global__ void __launch_bounds__(kRowThreads)
row_c2r_kernel(const T* __restrict__ S, const T* __restrict__ x, T* __restrict__ out,
               float* __restrict__ dst, RowParams p, int mode) {
  extern __shared__ float4 smem_raw[];
  float2* buf = reinterpret_cast<float2*>(smem_raw);
  const int np = p.rc / 2;
  float2* tw = buf + (size_t)p.W * np;
  const int tid = threadIdx.x;
  const int64_t row = blockIdx.x;  // b * H + h
  const int c0 = blockIdx.y * p.rc;
  const int half = p.W / 2;

  make_twiddles(tw, p.W);

  // Z[k] = Y_c[k] + i Y_{c+1}[k] over the full length, with Y[W-k] = conj Y[k] and only
  // the real parts of the k = 0 and k = W/2 bins; columns k >= KW are zero.
  const T* Sr = S + row * (int64_t)p.KW * p.C * 2;
  for (int it = tid; it < (half + 1) * np; it += blockDim.x) {
    const int k = it / np, q = it - k * np;
    float ar = 0.f, ai = 0.f, br = 0.f, bi = 0.f;
    if (k < p.KW) {
      const T* s = Sr + ((int64_t)k * p.C + c0 + 2 * q) * 2;
      if constexpr (Store<T>::kVec == 4) {
        const float4 v = *reinterpret_cast<const float4*>(s);
        ar = v.x; ai = v.y; br = v.z; bi = v.w;
      } else {
        union { uint2 u; bf16 h[4]; } w;
        w.u = *reinterpret_cast<const uint2*>(s);
        ar = (float)w.h[0]; ai = (float)w.h[1]; br = (float)w.h[2]; bi = (float)w.h[3];
      }
    }
    if (k == 0 || k == half) {
      buf[k * np + q] = make_float2(ar, br);
    } else {
      buf[k * np + q] = make_float2(ar - bi, ai + br);
      buf[(p.W - k) * np + q] = make_float2(ar + bi, br - ai);
    }
  }
  __syncthreads();

  const int sig = tid % np, sub = tid / np, nsub = blockDim.x / np;
  fft_lds<kRowEmax, true>(buf, np, p.rw, sig, sub, nsub, tw);

  constexpr int V = Store<T>::kVec;
  const int vpr = p.rc / V;
  const float sc = p.inv_sqrt_w;
  const int64_t base = row * p.W * p.C + c0;
  for (int it = tid; it < p.W * vpr; it += blockDim.x) {
    const int n = it / vpr, cv = it - n * vpr;
    const int64_t off = base + (int64_t)n * p.C + cv * V;
    float y[V];
#pragma unroll
    for (int q = 0; q < V / 2; ++q) {
      const float2 z = buf[n * np + cv * (V / 2) + q];
      y[2 * q] = z.x * sc;
      y[2 * q + 1] = z.y * sc;
    }
    if (mode == 1) {
#pragma unroll
      for (int e = 0; e < V; e += 4)
        *reinterpret_cast<float4*>(dst + off + e) = make_float4(y[e], y[e + 1], y[e + 2], y[e + 3]);
      continue;
    }
    V16 xv, ov;
    xv.u = *reinterpret_cast<const uint4*>(x + off);
#pragma unroll
    for (int e = 0; e < V; ++e) {
      if constexpr (V == 4) ov.f[e] = xv.f[e] + y[e];
      else ov.h[e] = (bf16)((float)xv.h[e] + y[e]);
    }
    *reinterpret_cast<uint4*>(out + off) = ov.u;
  }
}

// ------------------------------------------------------------------ kernel 2: column

// One layer of the block MLP on the LDS tile: acc[m][n] = tile rows x Wexp for the
// wave's two 16-column output tiles, over the live row tiles.
template <typename T>
__device__ __forceinline__ void block_gemm(const T* tile, int ldt, const T* w, int n_out,
                                           int n_in, int mt, uint32_t live, int wave, int lane,
                                           f32x4 (&acc)[kColMaxMTiles][2]) {
  typedef Mma<T> M;
#pragma unroll
  for (int m = 0; m < kColMaxMTiles; ++m)
    for (int n = 0; n < 2; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int jn0 = (32 * wave + (lane & 15)) >> 1;  // complex output column of tile 0
  const int jn1 = jn0 + 8;
  const int sg = lane & 1;
  for (int kb = 0; kb < 2 * n_in; kb += M::kK) {
    const typename M::Frag b0 = M::load_b(w, n_out, kb, jn0, sg, lane);
    const typename M::Frag b1 = M::load_b(w, n_out, kb, jn1, sg, lane);
#pragma unroll
    for (int m = 0; m < kColMaxMTiles; ++m) {
      if (m < mt && ((live >> m) & 1u)) {
        const typename M::Frag a = M::load_a(tile + (16 * m + (lane & 15)) * ldt, kb, lane);
        acc[m][0] = M::mma(a, b0, acc[m][0]);
        acc[m][1] = M::mma(a, b1, acc[m][1]);
      }
    }
  }
}

// grid B * KW * nb, block 64 * min(8, max(max(bs, hs) / 16, 4)).  stage: 0 full, 1 stop after
// the forward transform, 2 stop after the MLP.  hs != bs: the hidden layer (2 hs real entries
// per row) has its own LDS tile after the column tile, and waves take its 32-column groups in
// turn.
template <typename T>
__global__ void __launch_bounds__(kColMaxThreads)
column_kernel(T* __restrict__ S, const T* __restrict__ w1, const T* __restrict__ b1,
              const T* __restrict__ w2, const T* __restrict__ b2, ColParams p, int stage) {
  extern __shared__ float4 smem_raw[];
  T* tile = reinterpret_cast<T*>(smem_raw);                              // H16 x ldt
  T* htile = p.htile_bytes ? reinterpret_cast<T*>(reinterpret_cast<char*>(smem_raw) + p.tile_bytes)
                           : tile;                                       // H16 x ldh
  float2* fbuf = reinterpret_cast<float2*>(reinterpret_cast<char*>(smem_raw) + p.tile_bytes +
                                           p.htile_bytes);
  float2* tw = fbuf + (size_t)p.H * p.chk;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nthr = blockDim.x;
  const int bs = p.bs, hs = p.hs, ldt = p.ldt, H = p.H, H16 = p.H16;
  const int ldh = p.htile_bytes ? p.ldh : ldt;

  const int blk = blockIdx.x % p.nb;  // consecutive workgroups -> different XCDs -> blocks
  const int rest = blockIdx.x / p.nb;
  const int kw = rest % p.KW;
  const int64_t b = rest / p.KW;

  make_twiddles(tw, H);

  // ---- load the column tile: rows h < H of S[b][h][kw][blk*bs : +bs], zero padding rows
  constexpr int V = Store<T>::kVec;
  const int vpr = 2 * bs / V;
  const int64_t row_stride = (int64_t)p.KW * p.C * 2;
  T* col = S + ((b * H) * p.KW + kw) * (int64_t)p.C * 2 + (int64_t)blk * bs * 2;
  for (int it = tid; it < H16 * vpr; it += nthr) {
    const int h = it / vpr, cv = it - h * vpr;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (h < H) v = *reinterpret_cast<const uint4*>(col + h * row_stride + cv * V);
    *reinterpret_cast<uint4*>(tile + h * ldt + cv * V) = v;
  }
  __syncthreads();

  const int chk = p.chk;
  const int sig = tid % chk, sub = tid / chk, nsub = nthr / chk;
  const float sch = p.inv_sqrt_h;

  // ---- forward DFT along H, chk channels at a time through the float32 buffer
  for (int cc = 0; cc < bs; cc += chk) {
    for (int it = tid; it < H * chk; it += nthr) {
      const int h = it / chk, q = it - h * chk;
      const T* e = tile + h * ldt + 2 * (cc + q);
      fbuf[h * chk + q] = make_float2(ld_f(e), ld_f(e + 1));
    }
    __syncthreads();
    fft_lds<kColEmax, false>(fbuf, chk, p.rh, sig, sub, nsub, tw);
    for (int it = tid; it < H * chk; it += nthr) {
      const int h = it / chk, q = it - h * chk;
      const float2 z = fbuf[h * chk + q];
      T* e = tile + h * ldt + 2 * (cc + q);
      e[0] = Store<T>::to(z.x * sch);
      e[1] = Store<T>::to(z.y * sch);
    }
    __syncthreads();
  }

  if (stage != 1) {
    // ---- block MLP.  A wave owns 32 real output columns (16 complex) at a time.
    const int mt = H16 / 16;
    uint32_t live = 0;
    for (int m = 0; m < mt; ++m) {
      bool any = false;
      for (int r = 16 * m; r < 16 * m + 16; ++r) any |= row_kept(r, H, p.kept_h);
      live |= (any ? 1u : 0u) << m;
    }
    const T* W1 = w1 + (int64_t)blk * bs * hs * 2;
    const T* W2 = w2 + (int64_t)blk * hs * bs * 2;
    const T* B1 = b1 + (int64_t)blk * hs * 2;
    const T* B2 = b2 + (int64_t)blk * bs * 2;
    const int nwaves = nthr / 64;
    f32x4 acc[kColMaxMTiles][2];

    // layer 1: hidden groups grp = wave, wave + nwaves, ...; in place (hs = bs: one group per
    // wave at most) the spectrum rows are read by every wave before any is overwritten
    const int ng1 = hs / 16;
    const int rounds = (ng1 + nwaves - 1) / nwaves;
    for (int rd = 0; rd < rounds; ++rd) {
      const int grp = wave + rd * nwaves;
      const bool act = grp < ng1;
      if (act) block_gemm<T>(tile, ldt, W1, hs, bs, mt, live, grp, lane, acc);
      if (htile == tile) __syncthreads();
      if (act) {
        const int nu = 32 * grp + (lane & 15);
        const float bia0 = ld_f(B1 + nu), bia1 = ld_f(B1 + nu + 16);
#pragma unroll
        for (int m = 0; m < kColMaxMTiles; ++m) {
          if (m < mt && ((live >> m) & 1u)) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int row = 16 * m + 4 * (lane >> 4) + r;
              htile[row * ldh + nu] = Store<T>::to(fmaxf(acc[m][0][r] + bia0, 0.f));
              htile[row * ldh + nu + 16] = Store<T>::to(fmaxf(acc[m][1][r] + bia1, 0.f));
            }
          }
        }
      }
    }
    __syncthreads();  // hidden layer complete
    const bool active = wave < bs / 16;
    const int nu0 = 32 * wave + (lane & 15);  // real output column of tile 0 (tile 1: +16)
    if (active) block_gemm<T>(htile, ldh, W2, bs, hs, mt, live, wave, lane, acc);
    __syncthreads();  // every wave has read the hidden rows
    if (active) {
      const float bia0 = ld_f(B2 + nu0), bia1 = ld_f(B2 + nu0 + 16);
      const float lam = p.lam;
#pragma unroll
      for (int m = 0; m < kColMaxMTiles; ++m) {
        if (m < mt) {
          const bool lv = (live >> m) & 1u;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row = 16 * m + 4 * (lane >> 4) + r;
            const bool keep = lv && row_kept(row, H, p.kept_h);
            float o0 = lv ? acc[m][0][r] + bia0 : 0.f;
            float o1 = lv ? acc[m][1][r] + bia1 : 0.f;
            o0 = o0 > lam ? o0 - lam : (o0 < -lam ? o0 + lam : 0.f);
            o1 = o1 > lam ? o1 - lam : (o1 < -lam ? o1 + lam : 0.f);
            tile[row * ldt + nu0] = Store<T>::to(keep ? o0 : 0.f);
            tile[row * ldt + nu0 + 16] = Store<T>::to(keep ? o1 : 0.f);
          }
        }
      }
    }
    __syncthreads();

    if (stage == 0) {
      // ---- inverse DFT along H
      for (int cc = 0; cc < bs; cc += chk) {
        for (int it = tid; it < H * chk; it += nthr) {
          const int h = it / chk, q = it - h * chk;
          const T* e = tile + h * ldt + 2 * (cc + q);
          fbuf[h * chk + q] = make_float2(ld_f(e), ld_f(e + 1));
        }
        __syncthreads();
        fft_lds<kColEmax, true>(fbuf, chk, p.rh, sig, sub, nsub, tw);
        for (int it = tid; it < H * chk; it += nthr) {
          const int h = it / chk, q = it - h * chk;
          const float2 z = fbuf[h * chk + q];
          T* e = tile + h * ldt + 2 * (cc + q);
          e[0] = Store<T>::to(z.x * sch);
          e[1] = Store<T>::to(z.y * sch);
        }
        __syncthreads();
      }
    }
  }

  // ---- store the tile back in place
  for (int it = tid; it < H * vpr; it += nthr) {
    const int h = it / vpr, cv = it - h * vpr;
    *reinterpret_cast<uint4*>(col + h * row_stride + cv * V) =
        *reinterpret_cast<const uint4*>(tile + h * ldt + cv * V);
  }
}

// ------------------------------------------------------------------ diagnostic export

// dst [B][H][Wm][C][2] float from S [B][H][KW][C][2]; columns kw >= KW written as 0.
template <typename T>
__global__ void export_spectrum_kernel(const T* __restrict__ S, float* __restrict__ dst,
                                       int64_t B, int H, int Wm, int KW, int C) {
  const int64_t total = B * H * (int64_t)Wm * C * 2;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t e = i % (2 * C);
    const int64_t r = i / (2 * C);  // (b * H + h) * Wm + kw
    const int kw = (int)(r % Wm);
    const int64_t bh = r / Wm;
    dst[i] = (kw < KW) ? ld_f(S + (bh * KW + kw) * 2 * C + e) : 0.f;
  }
}

}  // namespace afno
