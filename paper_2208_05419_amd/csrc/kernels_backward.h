// kernels_backward.h -- the AFNO filter's backward pass on gfx950.
//
// For an upstream gradient g = dL/dout the filter's transpose runs the forward steps in
// reverse ("Model Innovations", steps 1-3; the paper trains through them, "Implementation
// Details" (a), (e)).  With F the 2-D real DFT (W-axis R2C then H-axis DFT, ortho), G its
// half-spectrum inverse (H-axis inverse DFT then W-axis C2R with weights c_kw = 1 at kw = 0
// and W/2, else 2) and the per-mode block MLP v = X W1 + b1, h = relu(v), o = h W2 + b2,
// z = S_lam(o) (componentwise on re and im, zero outside the cutoff), y = G(z):
//
//   dz  = c_kw F(g)                       (G's transpose: the weighted C2R's is c_kw R2C,
//                                          the unitary inverse H-DFT's the forward H-DFT)
//   do  = dz where |o| > lam and the mode is kept, else 0   (componentwise)
//   dh  = do W2^H,   dv = dh where v > 0, else 0
//   dX  = dv W1^H
//   dx  = g + G(dX / c_kw)                (F's transpose: C2R with unit weights)
//   dW1 = sum over modes conj(X)^T dv,  db1 = sum dv;  dW2 = sum conj(h)^T do,  db2 = sum do
//
// Passes: the forward W-axis kernel on x and on g (spectra Sx, Sg); a backward column kernel
// per (b, kw, block) recomputes X, h and both masks, transforms the gradient column and runs
// the two conjugate-transposed products, writing dX's inverse back into Sg and the per-mode
// factors X, h, do, dv to HBM in 8-mode groups; a weight-product kernel (wgrad_slab for bf16
// with 2 bs in {64, 128, 192}, else wgrad_kernel) forms the weight and bias gradients from the
// factors on the matrix cores as chunk sums, which wgrad_finalize_parts adds in a fixed order
// (no floating-point atomics: repeated calls give the same bits); the forward W-axis inverse kernel
// with g as its residual gives dx.  This header
// holds the size-generic column kernel (any dtype, H <= 192); kernels_backward_mfma.h the bf16
// one for H <= 96 with the H transforms on the matrix cores.
#pragma once
#include "kernels_generic.h"
#include "kernels_mfma.h"

namespace afno {

// wt[k][j][i] = conj(w[k][i][j]) for both layers: x wt = x W^H on the block_gemm path
template <typename T>
__device__ __forceinline__ void conj_transpose_one(int64_t t, const T* __restrict__ w1,
                                                   const T* __restrict__ w2, T* __restrict__ wt1,
                                                   T* __restrict__ wt2, int nb, int bs) {
  const int64_t n = (int64_t)nb * bs * bs;
  const int layer = t >= n ? 1 : 0;
  const int64_t u = t - layer * n;
  const int64_t k = u / ((int64_t)bs * bs);
  const int r = (int)(u - k * bs * bs), i = r / bs, j = r % bs;
  const T* src = (layer ? w2 : w1) + ((k * bs + i) * bs + j) * 2;
  T* dst = (layer ? wt2 : wt1) + ((k * bs + j) * bs + i) * 2;
  dst[0] = src[0];
  dst[1] = Store<T>::to(-ld_f(src + 1));
}

template <typename T>
__global__ void __launch_bounds__(256) conj_transpose_weights(const T* __restrict__ w1,
                                                              const T* __restrict__ w2,
                                                              T* __restrict__ wt1,
                                                              T* __restrict__ wt2, int nb, int bs) {
  const int64_t n = (int64_t)nb * bs * bs;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < 2 * n;
       t += (int64_t)gridDim.x * blockDim.x)
    conj_transpose_one<T>(t, w1, w2, wt1, wt2, nb, bs);
}

template <typename T>
__global__ void __launch_bounds__(256) fill_zero_f32(float* __restrict__ p, int64_t n) {
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < n;
       t += (int64_t)gridDim.x * blockDim.x)
    p[t] = 0.f;
}

// Per-mode factors: four tensors (X, h, do, dv), each [nb][mpad / 8][2 bs][8] in T: modes in
// groups of eight, the group's 2 bs entries consecutive, eight modes per entry contiguous (one
// 16-byte matrix-core operand for bf16).  The column (b, kw) holds modes (b KW + kw) HC ..
// + HC - 1, HC = H16 rounded up to 32 (rows past H hold X = 0, do = dv = 0, so they add
// nothing to the sums); mpad = B KW HC, a multiple of 32 (the slab product reads a chunk's
// ragged last 64-mode step as zeros past its end).
enum { kModeX = 0, kModeH = 1, kModeDo = 2, kModeDv = 3 };

// tile rows 0 .. HC - 1 of the block's 2 bs entries -> dst groups m0 / 8 .., 8 rows per task
// (rows past H16 are zero)
template <typename T>
__device__ __forceinline__ void write_modes(const T* tile, int ldt, int H16, int HC, int bs,
                                            T* dst, int64_t m0) {
  const int tasks = bs * (HC / 8);
  const int nb2 = 2 * bs;
  for (int t = threadIdx.x; t < tasks; t += blockDim.x) {
    const int c = t % bs, r0 = 8 * (t / bs);
    float re[8], im[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float2 z = r0 < H16 ? ld_c(tile + (r0 + i) * ldt + 2 * c) : make_float2(0.f, 0.f);
      re[i] = z.x;
      im[i] = z.y;
    }
    T* pr = dst + (((m0 + r0) / 8) * nb2 + 2 * c) * 8;
    T* pi = pr + 8;
    if constexpr (sizeof(T) == 2) {
      union { uint4 u; bf16 h[8]; } a, b;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        a.h[i] = (bf16)re[i];
        b.h[i] = (bf16)im[i];
      }
      *reinterpret_cast<uint4*>(pr) = a.u;
      *reinterpret_cast<uint4*>(pi) = b.u;
    } else {
#pragma unroll
      for (int i = 0; i < 8; i += 4) {
        *reinterpret_cast<float4*>(pr + i) = make_float4(re[i], re[i + 1], re[i + 2], re[i + 3]);
        *reinterpret_cast<float4*>(pi + i) = make_float4(im[i], im[i + 1], im[i + 2], im[i + 3]);
      }
    }
  }
}

// one column's rows h < H from S into the tile (times scale), padding rows zero
template <typename T>
__device__ __forceinline__ void load_column(T* tile, const T* col, int64_t row_stride, int ldt,
                                            int H, int H16, int bs, float scale) {
  for (int it = threadIdx.x; it < H16 * bs; it += blockDim.x) {
    const int h = it / bs, c = it - h * bs;
    float2 z = make_float2(0.f, 0.f);
    if (h < H) {
      z = ld_c(col + h * row_stride + 2 * c);
      z.x *= scale;
      z.y *= scale;
    }
    st_c(tile + h * ldt + 2 * c, z);
  }
}

// DFT along H of the tile's rows h < H (forward or inverse), chk channels at a time through
// the float buffer, scaled by 1/sqrt(H)
template <typename T, bool INV>
__device__ __forceinline__ void dft_tile(T* tile, float2* fbuf, const float2* tw, const ColParams& p) {
  const int tid = threadIdx.x, nthr = blockDim.x;
  const int chk = p.chk, H = p.H, ldt = p.ldt;
  const int sig = tid % chk, sub = tid / chk, nsub = nthr / chk;
  for (int cc = 0; cc < p.bs; cc += chk) {
    for (int it = tid; it < H * chk; it += nthr) {
      const int h = it / chk, q = it - h * chk;
      fbuf[h * chk + q] = ld_c(tile + h * ldt + 2 * (cc + q));
    }
    __syncthreads();
    fft_lds<kColEmax, INV>(fbuf, chk, p.rh, sig, sub, nsub, tw);
    for (int it = tid; it < H * chk; it += nthr) {
      const int h = it / chk, q = it - h * chk;
      const float2 z = fbuf[h * chk + q];
      st_c(tile + h * ldt + 2 * (cc + q), make_float2(z.x * p.inv_sqrt_h, z.y * p.inv_sqrt_h));
    }
    __syncthreads();
  }
}

// LDS of column_bwd_kernel: the tile, two bit masks [H16][2 bs / 32] words (word w of a row
// holds real columns 32 w .. 32 w + 31, the columns one MFMA wave owns), the float buffer,
// the twiddles
__host__ __device__ inline size_t col_bwd_mask_bytes(const ColParams& p) {
  return ((size_t)p.H16 * (2 * p.bs / 32) * 4 + 15) / 16 * 16;
}
__host__ __device__ inline size_t col_bwd_lds(const ColParams& p) {
  return (size_t)p.tile_bytes + 2 * col_bwd_mask_bytes(p) + (size_t)p.H * p.chk * 8 + (size_t)p.H * 8;
}
__host__ __device__ inline int col_bwd_hc(int H16) { return (H16 + 31) / 32 * 32; }

// the 32 mask bits of a row for the wave's two 16-column tiles: bit l16 from column tile 0,
// bit l16 + 16 from tile 1; lane l16 == 0 of each 16-lane group holds its row's word
__device__ __forceinline__ uint32_t mask_word(bool p0, bool p1, int lane) {
  const unsigned long long b0 = __ballot(p0), b1 = __ballot(p1);
  const int g = lane >> 4;
  return (uint32_t)((b0 >> (16 * g)) & 0xffffull) | ((uint32_t)((b1 >> (16 * g)) & 0xffffull) << 16);
}

// grid B * KW * nb (block index fastest), block 64 * max(bs / 16, 4), dynamic LDS
// col_bwd_lds(p).  Sx: the forward spectrum of x; Sg: that of g, replaced by
// G^-1-side gradient dX' = IDFT_H(dX) / c_kw (so that the forward C2R kernel's c_kw weights
// give the unit-weight transpose); modes: the four per-mode factor tensors (the weight-product
// pass takes the weight and bias gradients from them).
template <typename T>
__global__ void __launch_bounds__(kColMaxThreads)
column_bwd_kernel(const T* __restrict__ Sx, T* __restrict__ Sg, const T* __restrict__ w1,
                  const T* __restrict__ b1, const T* __restrict__ w2, const T* __restrict__ b2,
                  const T* __restrict__ wt1, const T* __restrict__ wt2, ColParams p,
                  T* __restrict__ modes, int64_t mpad, int W) {
  extern __shared__ float4 smem_raw[];
  T* tile = reinterpret_cast<T*>(smem_raw);
  const size_t mk_bytes = col_bwd_mask_bytes(p);
  uint32_t* mk1 = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(smem_raw) + p.tile_bytes);  // v > 0
  uint32_t* mk2 = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(mk1) + mk_bytes);  // |o| > lam, kept
  float2* fbuf = reinterpret_cast<float2*>(reinterpret_cast<char*>(mk2) + mk_bytes);
  float2* tw = fbuf + (size_t)p.H * p.chk;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, l16 = lane & 15;
  const int bs = p.bs, ldt = p.ldt, H = p.H, H16 = p.H16, nb2 = 2 * bs, nw = nb2 / 32;
  const int HC = col_bwd_hc(H16);

  const int blk = blockIdx.x % p.nb;
  const int rest = blockIdx.x / p.nb;
  const int kw = rest % p.KW;
  const int64_t b = rest / p.KW;
  const int64_t row_stride = (int64_t)p.KW * p.C * 2;
  const int64_t coff = ((b * H) * p.KW + kw) * (int64_t)p.C * 2 + (int64_t)blk * bs * 2;
  const int64_t m0 = (b * p.KW + kw) * (int64_t)HC;
  auto mode_tensor = [&](int t) { return modes + ((int64_t)t * p.nb + blk) * nb2 * mpad; };
  const float ckw = (kw == 0 || 2 * kw == W) ? 1.f : 2.f;

  make_twiddles(tw, H);

  const int mt = H16 / 16;
  uint32_t live = 0;
  for (int m = 0; m < mt; ++m) {
    bool any = false;
    for (int r = 16 * m; r < 16 * m + 16; ++r) any |= row_kept(r, H, p.kept_h);
    live |= (any ? 1u : 0u) << m;
  }
  const bool active = wave < bs / 16;
  const int nu0 = 32 * wave + (lane & 15);  // real output column of tile 0 (tile 1: +16)
  f32x4 acc[kColMaxMTiles][2];

  // ---- X = F(x) column; write X
  load_column<T>(tile, Sx + coff, row_stride, ldt, H, H16, bs, 1.f);
  __syncthreads();
  dft_tile<T, false>(tile, fbuf, tw, p);
  write_modes<T>(tile, ldt, H16, HC, bs, mode_tensor(kModeX), m0);

  // ---- layer 1: h = relu(X W1 + b1) -> tile, mask v > 0
  if (active) block_gemm<T>(tile, ldt, w1 + (int64_t)blk * bs * bs * 2, bs, bs, mt, live, wave, lane, acc);
  __syncthreads();  // the tile's X rows are read (products and the X write)
  if (active) {
    const T* B1 = b1 + (int64_t)blk * bs * 2;
    const float bia0 = ld_f(B1 + nu0), bia1 = ld_f(B1 + nu0 + 16);
#pragma unroll
    for (int m = 0; m < kColMaxMTiles; ++m) {
      if (m >= mt) continue;
      const bool lv = (live >> m) & 1u;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * m + 4 * (lane >> 4) + r;
        const float v0 = acc[m][0][r] + bia0, v1 = acc[m][1][r] + bia1;
        if (lv) {
          tile[row * ldt + nu0] = Store<T>::to(fmaxf(v0, 0.f));
          tile[row * ldt + nu0 + 16] = Store<T>::to(fmaxf(v1, 0.f));
        }
        const uint32_t wd = mask_word(lv && v0 > 0.f, lv && v1 > 0.f, lane);
        if (l16 == 0) mk1[row * nw + wave] = wd;
      }
    }
  }
  __syncthreads();
  write_modes<T>(tile, ldt, H16, HC, bs, mode_tensor(kModeH), m0);

  // ---- layer 2: only its mask |o| > lam (and the cutoff) is needed
  if (active) block_gemm<T>(tile, ldt, w2 + (int64_t)blk * bs * bs * 2, bs, bs, mt, live, wave, lane, acc);
  if (active) {
    const T* B2 = b2 + (int64_t)blk * bs * 2;
    const float bia0 = ld_f(B2 + nu0), bia1 = ld_f(B2 + nu0 + 16);
#pragma unroll
    for (int m = 0; m < kColMaxMTiles; ++m) {
      if (m >= mt) continue;
      const bool lv = (live >> m) & 1u;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * m + 4 * (lane >> 4) + r;
        const bool keep = lv && row_kept(row, H, p.kept_h);
        const uint32_t wd = mask_word(keep && fabsf(acc[m][0][r] + bia0) > p.lam,
                                      keep && fabsf(acc[m][1][r] + bia1) > p.lam, lane);
        if (l16 == 0) mk2[row * nw + wave] = wd;
      }
    }
  }
  __syncthreads();  // the h rows are read (products and the h write), masks complete

  // ---- dz = c_kw F(g) column; do = dz masked; write do
  load_column<T>(tile, Sg + coff, row_stride, ldt, H, H16, bs, ckw);
  __syncthreads();
  dft_tile<T, false>(tile, fbuf, tw, p);
  for (int it = tid; it < H16 * nb2; it += blockDim.x) {
    const int row = it / nb2, e = it - row * nb2;
    if (!((mk2[row * nw + (e >> 5)] >> (e & 31)) & 1u)) tile[row * ldt + e] = Store<T>::to(0.f);
  }
  __syncthreads();
  write_modes<T>(tile, ldt, H16, HC, bs, mode_tensor(kModeDo), m0);

  // ---- dv = (do W2^H) masked by v > 0; write dv
  if (active) block_gemm<T>(tile, ldt, wt2 + (int64_t)blk * bs * bs * 2, bs, bs, mt, live, wave, lane, acc);
  __syncthreads();
  if (active) {
#pragma unroll
    for (int m = 0; m < kColMaxMTiles; ++m) {
      if (m >= mt) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * m + 4 * (lane >> 4) + r;
        const uint32_t wd = mk1[row * nw + wave];  // 0 on rows outside the live tiles
        tile[row * ldt + nu0] = Store<T>::to((wd >> l16) & 1u ? acc[m][0][r] : 0.f);
        tile[row * ldt + nu0 + 16] = Store<T>::to((wd >> (l16 + 16)) & 1u ? acc[m][1][r] : 0.f);
      }
    }
  }
  __syncthreads();
  write_modes<T>(tile, ldt, H16, HC, bs, mode_tensor(kModeDv), m0);

  // ---- dX = dv W1^H -> inverse H-DFT -> Sg column / c_kw
  if (active) block_gemm<T>(tile, ldt, wt1 + (int64_t)blk * bs * bs * 2, bs, bs, mt, live, wave, lane, acc);
  __syncthreads();
  if (active) {
#pragma unroll
    for (int m = 0; m < kColMaxMTiles; ++m) {
      if (m >= mt) continue;
      const bool lv = (live >> m) & 1u;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = 16 * m + 4 * (lane >> 4) + r;
        tile[row * ldt + nu0] = Store<T>::to(lv ? acc[m][0][r] : 0.f);
        tile[row * ldt + nu0 + 16] = Store<T>::to(lv ? acc[m][1][r] : 0.f);
      }
    }
  }
  __syncthreads();
  dft_tile<T, true>(tile, fbuf, tw, p);
  T* col = Sg + coff;
  const float inv_c = 1.f / ckw;
  for (int it = tid; it < H * bs; it += blockDim.x) {
    const int h = it / bs, c = it - h * bs;
    const float2 z = ld_c(tile + h * ldt + 2 * c);
    st_c(col + h * row_stride + 2 * c, make_float2(z.x * inv_c, z.y * inv_c));
  }
}

// Weight-gradient products over all modes: for layer 0 (dW1) A = X, B = dv; for layer 1
// (dW2) A = h, B = do; part[chunk][layer][blk][r][s] = sum over the chunk's modes of
// A[r][m] B[s][m] (r, s the 2 bs real entries, (c, rho) interleaved), and
// bpart[chunk][layer][blk][s] = sum of B[s][m] (the bias gradients db1, db2): plain stores,
// one workgroup per output value and chunk, summed over the chunks by wgrad_finalize_parts in
// chunk order, so repeated calls give the same bits.
// grid (2 nb tiles64^2, nchunk = ceil(mpad / kchunk)), 256 threads: four waves with 32 x 32
// each of a 64 x 64 output tile; kchunk a multiple of 32.
template <typename T>
__global__ void __launch_bounds__(256) wgrad_kernel(const T* __restrict__ modes, int64_t mpad,
                                                    int nb, int bs, int kchunk,
                                                    float* __restrict__ part,
                                                    float* __restrict__ bpart) {
  typedef Mma<T> M;
  const int nb2 = 2 * bs;
  const int nt64 = (nb2 + 63) / 64;
  int g = blockIdx.x;
  const int ts = g % nt64; g /= nt64;
  const int tr = g % nt64; g /= nt64;
  const int blk = g % nb; g /= nb;
  const int layer = g;  // 0: dW1, 1: dW2
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r0 = 64 * tr + 32 * (wave >> 1), s0 = 64 * ts + 32 * (wave & 1);
  const T* A = modes + ((int64_t)(layer ? kModeH : kModeX) * nb + blk) * nb2 * mpad;
  const T* Bm = modes + ((int64_t)(layer ? kModeDo : kModeDv) * nb + blk) * nb2 * mpad;
  const int64_t k0 = (int64_t)blockIdx.y * kchunk;
  const int64_t k1 = k0 + kchunk < mpad ? k0 + kchunk : mpad;
  f32x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const bool rv[2] = {r0 < nb2, r0 + 16 < nb2}, sv[2] = {s0 < nb2, s0 + 16 < nb2};
  const int l16 = lane & 15, gq = lane >> 4;
  // the two waves of the first row tile also sum their B fragments: entries s0 + 16 j + l16,
  // this lane's modes of each k-step
  const bool bias_wave = tr == 0 && (wave >> 1) == 0;
  float bsum[2] = {0.f, 0.f};
  for (int64_t k = k0; k < k1; k += M::kK) {
    typename M::Frag a[2], bfr[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = rv[i] ? r0 + 16 * i + l16 : 0;
      const int s = sv[i] ? s0 + 16 * i + l16 : 0;
      if constexpr (sizeof(T) == 2) {  // eight modes k + 8 gq .. + 7: one group
        const int64_t grp = (k >> 3) + gq;
        a[i] = *reinterpret_cast<const bf16x8*>(A + (grp * nb2 + r) * 8);
        bfr[i] = *reinterpret_cast<const bf16x8*>(Bm + (grp * nb2 + s) * 8);
      } else {
        const int64_t md = k + gq;
        a[i] = A[((md >> 3) * nb2 + r) * 8 + (md & 7)];
        bfr[i] = Bm[((md >> 3) * nb2 + s) * 8 + (md & 7)];
      }
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = M::mma(a[i], bfr[j], acc[i][j]);
    if (bias_wave) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if constexpr (sizeof(T) == 2) {
          float s8 = 0.f;
#pragma unroll
          for (int q = 0; q < 8; ++q) s8 += (float)bfr[j][q];
          bsum[j] += s8;
        } else {
          bsum[j] += bfr[j];
        }
      }
    }
  }
  const int64_t slot = ((int64_t)blockIdx.y * 2 + layer) * nb + blk;
  if (bias_wave) {
    // the four lane groups hold different modes of the same entry: a fixed butterfly
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float v = bsum[j];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (gq == 0 && sv[j]) bpart[slot * nb2 + s0 + 16 * j + l16] = v;
    }
  }
  float* out = part + slot * nb2 * nb2;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (!rv[i] || !sv[j]) continue;
      const int s = s0 + 16 * j + l16;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r = r0 + 16 * i + 4 * gq + q;
        out[(int64_t)r * nb2 + s] = acc[i][j][q];
      }
    }
}

// bf16 weight-gradient products for 2 bs = NB2 a multiple of 64: one workgroup per (layer,
// block, mode chunk) computes the chunk's whole NB2 x NB2 product, so each per-mode operand is
// read from HBM once.  Per 64-mode step the two operand slabs (8 mode groups x NB2 entries x
// 16 bytes each) stream through LDS, double buffered; the global loads of the two following
// steps are in flight (in registers) during the current step's products, so that a workgroup
// keeps two steps' bytes on the way from HBM.  16 waves as 4 x 4, each (NB2 / 64)^2 output
// tiles of 16 x 16 (one workgroup per compute unit).  Words beyond the chunk's modes read 0
// (buffer range check).  The chunk's sums go to part[chunk][layer][blk][r][s] (plain stores).
// The same pass sums the second operand over the chunk's modes (do for dW2, dv for dW1: the
// bias gradients db2, db1): each thread adds up the words it moves, in step order, and the
// eight mode groups of an entry are added in a fixed order at the end, to
// bpart[chunk][layer][blk][entry] -- so no atomics, and repeated calls give the same bits.
// grid 2 nb nchunk (layer, block, chunk with block fastest), 1024 threads, dynamic LDS
// 2 * 2 * 8 * NB2 * 16 bytes; kchunk a multiple of 64.
template <int NB2>
__global__ void __launch_bounds__(1024) wgrad_slab(const bf16* __restrict__ modes, int64_t mpad,
                                                   int nb, int kchunk, float* __restrict__ part,
                                                   float* __restrict__ bpart) {
  constexpr int T = NB2 / 64;       // output tiles per wave along each axis
  constexpr int SLAB = 8 * NB2;     // 16-byte words per operand and step
  constexpr int LW = 2 * SLAB / 1024;  // words each thread moves per step
  static_assert(SLAB % 64 == 0 && 2 * SLAB % 1024 == 0, "operand uniform per wave, whole words");
  extern __shared__ uint4 slab_lds[];  // [2 buffers][2 operands][SLAB]
  const int tid = threadIdx.x, lane = tid & 63, l16 = lane & 15, gq = lane >> 4;
  const int wave = tid >> 6, wr = wave >> 2, wc = wave & 3;
  int g = blockIdx.x;
  const int blk = g % nb;
  g /= nb;
  const int layer = g & 1;
  const int chunk = g >> 1;
  const int64_t k0 = (int64_t)chunk * kchunk;
  const int64_t k1 = k0 + kchunk < mpad ? k0 + kchunk : mpad;
  const int steps = (int)((k1 - k0 + 63) / 64);
  // the chunk's words of each operand: groups k0 / 8 .. k1 / 8, NB2 words each
  const uint32_t cbytes = buf_bytes((uint64_t)(k1 - k0) / 8 * NB2 * 16);
  const int64_t cw = (k0 >> 3) * NB2;
  const Buf ra(reinterpret_cast<const uint4*>(
                   modes + ((int64_t)(layer ? kModeH : kModeX) * nb + blk) * NB2 * mpad) + cw,
               cbytes);
  const Buf rb(reinterpret_cast<const uint4*>(
                   modes + ((int64_t)(layer ? kModeDo : kModeDv) * nb + blk) * NB2 * mpad) + cw,
               cbytes);
  // word w = tid + 1024 i of a step: operand w / SLAB (uniform per wave), word w % SLAB of
  // that operand's slab, which starts 8 NB2 words further on each step
  uint32_t voff[LW];
  bool opb[LW];
#pragma unroll
  for (int i = 0; i < LW; ++i) {
    const int w = tid + 1024 * i;
    opb[i] = __builtin_amdgcn_readfirstlane(w / SLAB) != 0;
    voff[i] = (uint32_t)(w % SLAB) * 16u;
  }
  auto load = [&](uint4 (&r)[LW], int s) {
    // the step's offset goes into the per-lane offset, which the range check covers; the factors
  // are read once (non-temporal loads keep them from displacing other data in the caches)
    const uint32_t so = (uint32_t)s * (uint32_t)(SLAB * 16);
#pragma unroll
    for (int i = 0; i < LW; ++i) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(opb[i] ? rb.r : ra.r, voff[i] + so, 0,
                                                            kNonTemporal);
      r[i] = make_uint4(v[0], v[1], v[2], v[3]);
    }
  };
  // per word moved: the sum of its eight modes, over all steps (used for the second operand)
  float bsum[LW];
#pragma unroll
  for (int i = 0; i < LW; ++i) bsum[i] = 0.f;
  auto stash = [&](const uint4 (&r)[LW], int buf) {
#pragma unroll
    for (int i = 0; i < LW; ++i) {
      slab_lds[buf * 2 * SLAB + tid + 1024 * i] = r[i];
      if (opb[i]) {  // wave-uniform
        const uint32_t v[4] = {r[i].x, r[i].y, r[i].z, r[i].w};
        float s8 = 0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          s8 += __uint_as_float(v[q] << 16) + __uint_as_float(v[q] & 0xffff0000u);
        bsum[i] += s8;
      }
    }
  };
  f32x4 acc[T][T];
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int j = 0; j < T; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](int buf) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      const uint4* LA = slab_lds + buf * 2 * SLAB + (4 * kk + gq) * NB2 + l16;
      const uint4* LB = LA + SLAB;
      uint4 a[T], b[T];
#pragma unroll
      for (int i = 0; i < T; ++i) a[i] = LA[16 * (wr * T + i)];
#pragma unroll
      for (int j = 0; j < T; ++j) b[j] = LB[16 * (wc * T + j)];
#pragma unroll
      for (int i = 0; i < T; ++i)
#pragma unroll
        for (int j = 0; j < T; ++j) acc[i][j] = mma_bf16(a[i], b[j], acc[i][j]);
    }
  };
  if (steps > 0) {
    // two register sets take turns, so that no step's words are copied between registers;
    // the steps run in pairs (a step past the chunk reads zeros and adds nothing).  The
    // scheduling barriers keep each step's loads issued before the products they overlap.
    uint4 r0[LW], r1[LW];
    load(r0, 0);
    load(r1, 1);
    stash(r0, 0);
    __syncthreads();
    for (int s = 0; s < steps; s += 2) {
      load(r0, s + 2);  // buffer 0 was read last in step s
      __builtin_amdgcn_sched_barrier(0);
      compute(0);
      stash(r1, 1);
      __syncthreads();
      load(r1, s + 3);
      __builtin_amdgcn_sched_barrier(0);
      compute(1);
      stash(r0, 0);
      __syncthreads();
    }
  }
  // bias sums: word (group, entry) of the second operand's slab -> LDS, then per entry the
  // eight groups in order (the slabs are no longer read: every product is behind a barrier)
  __syncthreads();
  float* red = reinterpret_cast<float*>(slab_lds);
#pragma unroll
  for (int i = 0; i < LW; ++i)
    if (opb[i]) red[(tid + 1024 * i) % SLAB] = bsum[i];
  __syncthreads();
  if (tid < NB2) {
    float sb = 0.f;
#pragma unroll
    for (int q = 0; q < 8; ++q) sb += red[q * NB2 + tid];
    bpart[(((int64_t)chunk * 2 + layer) * nb + blk) * NB2 + tid] = sb;
  }
  float* out = part + (((int64_t)chunk * 2 + layer) * nb + blk) * NB2 * NB2;
#pragma unroll
  for (int i = 0; i < T; ++i)
#pragma unroll
    for (int j = 0; j < T; ++j) {
      const int col = 16 * (wc * T + j) + l16;
#pragma unroll
      for (int q = 0; q < 4; ++q) out[(16 * (wr * T + i) + 4 * gq + q) * NB2 + col] = acc[i][j][q];
    }
}

// dW (re, im) from the weight-product kernels' chunk sums part[chunk][2][nb][2 bs][2 bs]: for
// entries r = (i, rho), s = (j, sigma), dW[i][j] = (P[(i,0)][(j,0)] + P[(i,1)][(j,1)],
// P[(i,0)][(j,1)] - P[(i,1)][(j,0)]) (conj(a) b summed); db1, db2 from the chunk bias sums
// bpart[chunk][2][nb][2 bs]; each summed over the chunks here in chunk order.  Grid over
// 2 nb bs^2.
__global__ void __launch_bounds__(256) wgrad_finalize_parts(const float* __restrict__ part,
                                                            int nchunk, const float* __restrict__ bpart,
                                                            int nb, int bs, float* __restrict__ dw1,
                                                            float* __restrict__ dw2,
                                                            float* __restrict__ db1,
                                                            float* __restrict__ db2) {
  const int nb2 = 2 * bs;
  const int64_t n = (int64_t)nb * bs * bs;
  const int64_t nbias = (int64_t)nb * nb2;
  const int64_t cstride = (int64_t)2 * nb * nb2 * nb2;
  for (int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; t < 2 * n;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int layer = t >= n ? 1 : 0;
    const int64_t u = t - layer * n;
    const int64_t k = u / ((int64_t)bs * bs);
    const int r = (int)(u - k * bs * bs), i = r / bs, j = r % bs;
    const float* P = part + ((int64_t)layer * nb + k) * nb2 * nb2;
    float rr = 0.f, ii = 0.f, ri = 0.f, ir = 0.f;
    for (int c = 0; c < nchunk; ++c, P += cstride) {
      rr += P[(2 * i) * nb2 + 2 * j];
      ii += P[(2 * i + 1) * nb2 + 2 * j + 1];
      ri += P[(2 * i) * nb2 + 2 * j + 1];
      ir += P[(2 * i + 1) * nb2 + 2 * j];
    }
    float* d = (layer ? dw2 : dw1) + ((k * bs + i) * bs + j) * 2;
    d[0] = rr + ii;
    d[1] = ri - ir;
    if (t < 2 * nbias) {
      float sb = 0.f;
      for (int c = 0; c < nchunk; ++c) sb += bpart[(int64_t)c * 2 * nbias + t];
      (t < nbias ? db1 : db2)[t < nbias ? t : t - nbias] = sb;
    }
  }
}

}  // namespace afno
