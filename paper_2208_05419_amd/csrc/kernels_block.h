// kernels_block.h -- the rest of one AFNO transformer block around the spectral filter:
// per-token LayerNorm, the channel-mixing MLP (C -> 4C -> C, shared by all tokens, "Model
// Innovations" and "Implementation Details" (c)) as two bf16 matrix-core GEMMs with fused
// epilogues, and the residual adds.  Tokens are the rows of x [B H W][C] (row-major).
//
//   t   = LN1(x)                         layer_norm_kernel
//   u   = filter(t)  (= t + y(t))         the filter's kernels
//   v   = u + x,  w = LN2(v)              add_layer_norm_kernel
//   h   = GELU(w Wa + ba)                 gemm_bf16<kEpiGelu>
//   out = v + h Wb + bb                   gemm_bf16<kEpiResidual>
#pragma once
#include "kernel_common.h"
#include "kernels_mfma.h"

namespace afno {

constexpr int kLnMaxPerLane = 32;  // values a lane holds: C <= 64 * 32
constexpr float kLnEps = 1e-6f;

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// LayerNorm of one token's C channels held as vals[0 .. n) by this lane (channels
// 8 (lane + 64 i) .. + 7 for chunk i), two passes over registers; writes bf16.
template <int NCH>
__device__ __forceinline__ void ln_token(float (&vals)[NCH][8], int nchunk, int C, int lane,
                                         const bf16* __restrict__ gamma,
                                         const bf16* __restrict__ beta, bf16* __restrict__ y) {
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NCH; ++i)
    if (lane + 64 * i < nchunk) {
#pragma unroll
      for (int e = 0; e < 8; ++e) s += vals[i][e];
    }
  const float mean = wave_sum(s) / (float)C;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < NCH; ++i)
    if (lane + 64 * i < nchunk) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float d = vals[i][e] - mean;
        q += d * d;
      }
    }
  const float rstd = rsqrtf(wave_sum(q) / (float)C + kLnEps);
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    const int ch = lane + 64 * i;
    if (ch < nchunk) {
      const uint4 gw = *reinterpret_cast<const uint4*>(gamma + 8 * ch);
      const uint4 bw = *reinterpret_cast<const uint4*>(beta + 8 * ch);
      const uint32_t* gu = reinterpret_cast<const uint32_t*>(&gw);
      const uint32_t* bu = reinterpret_cast<const uint32_t*>(&bw);
      uint32_t o[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const float g0 = __uint_as_float(gu[p] << 16), g1 = __uint_as_float(gu[p] & 0xffff0000u);
        const float b0 = __uint_as_float(bu[p] << 16), b1 = __uint_as_float(bu[p] & 0xffff0000u);
        o[p] = cvt_pk((vals[i][2 * p] - mean) * rstd * g0 + b0,
                      (vals[i][2 * p + 1] - mean) * rstd * g1 + b1);
      }
      *reinterpret_cast<uint4*>(y + 8 * ch) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

__device__ __forceinline__ void unpack8(uint4 w, float (&v)[8]) {
  const uint32_t* u = reinterpret_cast<const uint32_t*>(&w);
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    v[2 * p] = __uint_as_float(u[p] << 16);
    v[2 * p + 1] = __uint_as_float(u[p] & 0xffff0000u);
  }
}

// y = LN(x) per token; one wave per token, 4 tokens per 256-thread workgroup.  C a multiple
// of 8, at most 64 * kLnMaxPerLane.
__global__ void __launch_bounds__(256) layer_norm_kernel(const bf16* __restrict__ x,
                                                         const bf16* __restrict__ gamma,
                                                         const bf16* __restrict__ beta,
                                                         bf16* __restrict__ y, int64_t M, int C) {
  constexpr int NCH = kLnMaxPerLane / 8;
  const int lane = threadIdx.x & 63;
  const int64_t tok = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= M) return;
  const int nchunk = C / 8;
  const bf16* xr = x + tok * C;
  float vals[NCH][8];
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    const int ch = lane + 64 * i;
    if (ch < nchunk) unpack8(*reinterpret_cast<const uint4*>(xr + 8 * ch), vals[i]);
  }
  ln_token<NCH>(vals, nchunk, C, lane, gamma, beta, y + tok * C);
}

// v = u + x (rounded to bf16 and stored), w = LN(v) of the stored v; as layer_norm_kernel.
__global__ void __launch_bounds__(256) add_layer_norm_kernel(const bf16* __restrict__ u,
                                                             const bf16* __restrict__ x,
                                                             const bf16* __restrict__ gamma,
                                                             const bf16* __restrict__ beta,
                                                             bf16* __restrict__ v,
                                                             bf16* __restrict__ w, int64_t M, int C) {
  constexpr int NCH = kLnMaxPerLane / 8;
  const int lane = threadIdx.x & 63;
  const int64_t tok = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= M) return;
  const int nchunk = C / 8;
  float vals[NCH][8];
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    const int ch = lane + 64 * i;
    if (ch < nchunk) {
      float a[8], b[8];
      unpack8(*reinterpret_cast<const uint4*>(u + tok * C + 8 * ch), a);
      unpack8(*reinterpret_cast<const uint4*>(x + tok * C + 8 * ch), b);
      uint32_t o[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) o[p] = cvt_pk(a[2 * p] + b[2 * p], a[2 * p + 1] + b[2 * p + 1]);
      const uint4 ow = make_uint4(o[0], o[1], o[2], o[3]);
      *reinterpret_cast<uint4*>(v + tok * C + 8 * ch) = ow;
      unpack8(ow, vals[i]);  // LN of the stored (rounded) v
    }
  }
  ln_token<NCH>(vals, nchunk, C, lane, gamma, beta, w + tok * C);
}

// dst[c][r] = src[r][c] for a rows x cols bf16 matrix (weights to the GEMM's [N][K] form)
__global__ void __launch_bounds__(256) transpose_bf16(const bf16* __restrict__ src,
                                                      bf16* __restrict__ dst, int rows, int cols) {
  __shared__ uint16_t t[32][33];
  const int c0 = blockIdx.x * 32, r0 = blockIdx.y * 32;
  const uint16_t* s = reinterpret_cast<const uint16_t*>(src);
  uint16_t* d = reinterpret_cast<uint16_t*>(dst);
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 32 x 8
  for (int i = ty; i < 32; i += 8) {
    const int r = r0 + i, c = c0 + tx;
    t[i][tx] = (r < rows && c < cols) ? s[(int64_t)r * cols + c] : (uint16_t)0;
  }
  __syncthreads();
  for (int i = ty; i < 32; i += 8) {
    const int c = c0 + i, r = r0 + tx;
    if (c < cols && r < rows) d[(int64_t)c * rows + r] = t[tx][i];
  }
}

enum { kEpiGelu = 0, kEpiResidual = 1 };

// GEMM geometry of the register-staged kernel (column counts N that are not a multiple of
// 256): workgroup tile 256 x BN (rows x columns of D), k-stage 64 (two MFMA k-steps per
// barrier); 4 x (BN / 64) waves, each 64 x 64 (4 x 4 MFMA tiles of 16 x 16).  LDS: two stages
// of the A (256 x 64) and B (BN x 64) slabs, rows padded to 72 elements; the epilogue reuses
// it for 64 rows of fp32 at a time.
template <int BN>
struct GemmGeo {
  static constexpr int BM = 256, BK = 64, LDK = BK + 8;
  static constexpr int NWN = BN / 64, NT = 64 * 4 * NWN;    // threads
  static constexpr int ASLAB = BM * LDK, BSLAB = BN * LDK;
  static constexpr int STAGE = ASLAB + BSLAB;               // elements
  static constexpr int LDC = BN + 4;                         // epilogue stride, floats
  static constexpr int kLA = BM * (BK / 8) / NT, kLB = BN * (BK / 8) / NT;  // words per thread
  static constexpr int kBytes = 2 * STAGE * 2 > 64 * LDC * 4 ? 2 * STAGE * 2 : 64 * LDC * 4;
  static_assert(BM * (BK / 8) % NT == 0 && BN * (BK / 8) % NT == 0, "whole words per thread");
};

// D[M][N] = epi(A[M][K] Bt[N][K]^T + bias[N]) in bf16, fp32 accumulation on the matrix cores.
// The next k-stage's global loads are in flight during the current stage's products.
// Epilogue: + bias staged through LDS in fp32 (64 rows at a time), then, on the way out to
// row-contiguous stores, GELU (kEpiGelu) or + R[M][N] (kEpiResidual).  Rows of A past M are read clamped and never
// stored.  Tiles go XCD-aware: workgroup g runs on XCD g % 8 and the workgroups of one XCD
// take all column tiles of a row tile in turn, so that row tile's A stays in that XCD's L2.
// N a multiple of BN, K a multiple of 64; grid 8 ceil(MB / 8) (N / BN) with MB = ceil(M / 256);
// GemmGeo<BN>::NT threads; dynamic LDS GemmGeo<BN>::kBytes.
template <int EPI, int BN>
__global__ void __launch_bounds__(GemmGeo<BN>::NT) gemm_bf16(const bf16* __restrict__ A,
                                                             const bf16* __restrict__ Bt,
                                                             const bf16* __restrict__ bias,
                                                             const bf16* __restrict__ R,
                                                             bf16* __restrict__ D, int M, int N,
                                                             int K) {
  typedef GemmGeo<BN> G;
  extern __shared__ uint4 gemm_smem[];
  bf16* S = reinterpret_cast<bf16*>(gemm_smem);           // [2][STAGE]: A slab, then B slab
  float* sC = reinterpret_cast<float*>(gemm_smem);        // [64][LDC] in the epilogue

  const int nbn = N / BN;
  const int g = blockIdx.x, xcd = g & 7, i = g >> 3;
  const int mb = (i / nbn) * 8 + xcd, nbk = i - (i / nbn) * nbn;
  const int m0 = mb * G::BM, n0 = nbk * BN;
  if (m0 >= M) return;  // padding workgroups: the whole group leaves before any barrier

  const int tid = threadIdx.x, lane = tid & 63, l16 = lane & 15, gq = lane >> 4;
  const int wave = tid >> 6, wm = wave / G::NWN, wn = wave % G::NWN;
  // global -> LDS: thread tid moves k-word tid % 8 of rows tid / 8 + RS j (A: kLA rows, B: kLB)
  constexpr int WPR = G::BK / 8, RS = G::NT / WPR;
  const int r4 = tid / WPR, kc = 8 * (tid % WPR);
  const bf16* srcB = Bt + (int64_t)(n0 + r4) * K + kc;
  int64_t aoff[G::kLA];
#pragma unroll
  for (int j = 0; j < G::kLA; ++j) aoff[j] = (int64_t)min(m0 + r4 + RS * j, M - 1) * K + kc;
  const int dA = r4 * G::LDK + kc, dB = G::ASLAB + r4 * G::LDK + kc;
  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int stages = K / G::BK;
  {
    uint4 ra[G::kLA], rb[G::kLB];
#pragma unroll
    for (int j = 0; j < G::kLA; ++j) ra[j] = *reinterpret_cast<const uint4*>(A + aoff[j]);
#pragma unroll
    for (int j = 0; j < G::kLB; ++j)
      rb[j] = *reinterpret_cast<const uint4*>(srcB + (int64_t)RS * j * K);
#pragma unroll
    for (int j = 0; j < G::kLA; ++j) *reinterpret_cast<uint4*>(S + dA + RS * j * G::LDK) = ra[j];
#pragma unroll
    for (int j = 0; j < G::kLB; ++j) *reinterpret_cast<uint4*>(S + dB + RS * j * G::LDK) = rb[j];
  }
  __syncthreads();
  for (int s = 0; s < stages; ++s) {
    const int buf = s & 1;
    // the next stage's words (the last stage reloads its own: loads and stores unconditional)
    const int kn = (s + 1 < stages ? s + 1 : s) * G::BK;
    uint4 na[G::kLA], nb_[G::kLB];
#pragma unroll
    for (int j = 0; j < G::kLA; ++j) na[j] = *reinterpret_cast<const uint4*>(A + aoff[j] + kn);
#pragma unroll
    for (int j = 0; j < G::kLB; ++j)
      nb_[j] = *reinterpret_cast<const uint4*>(srcB + (int64_t)RS * j * K + kn);
    const bf16* cA = S + buf * G::STAGE + (64 * wm + l16) * G::LDK + 8 * gq;
    const bf16* cB = S + buf * G::STAGE + G::ASLAB + (64 * wn + l16) * G::LDK + 8 * gq;
#pragma unroll
    for (int kk = 0; kk < G::BK; kk += 32) {
      uint4 fa[4], fb[4];
#pragma unroll
      for (int a = 0; a < 4; ++a)
        fa[a] = *reinterpret_cast<const uint4*>(cA + 16 * a * G::LDK + kk);
#pragma unroll
      for (int b = 0; b < 4; ++b)
        fb[b] = *reinterpret_cast<const uint4*>(cB + 16 * b * G::LDK + kk);
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = mma_bf16(fa[a], fb[b], acc[a][b]);
    }
    bf16* nS = S + (buf ^ 1) * G::STAGE;
#pragma unroll
    for (int j = 0; j < G::kLA; ++j) *reinterpret_cast<uint4*>(nS + dA + RS * j * G::LDK) = na[j];
#pragma unroll
    for (int j = 0; j < G::kLB; ++j) *reinterpret_cast<uint4*>(nS + dB + RS * j * G::LDK) = nb_[j];
    __syncthreads();
  }

  // ---- epilogue, one wave row (64 rows) at a time
  float bv[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) bv[b] = (float)bias[n0 + 64 * wn + 16 * b + l16];
  constexpr int C4 = BN / 4;              // groups of 4 columns per row
  constexpr int PER = 64 * C4 / G::NT;    // groups per thread
#pragma unroll 1
  for (int part = 0; part < 4; ++part) {
    if (wm == part) {
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            sC[(16 * a + 4 * gq + q) * G::LDC + 64 * wn + 16 * b + l16] = acc[a][b][q] + bv[b];
          }
    }
    __syncthreads();
#pragma unroll 1
    for (int j = 0; j < PER; ++j) {
      const int c = tid + G::NT * j;
      const int r = c / C4, c4 = 4 * (c - (c / C4) * C4);
      const int row = m0 + 64 * part + r;
      if (row < M) {
        const float4 z = *reinterpret_cast<const float4*>(sC + r * G::LDC + c4);
        float o0 = z.x, o1 = z.y, o2 = z.z, o3 = z.w;
        if constexpr (EPI == kEpiGelu) {  // GELU(z) = z Phi(z) = 0.5 z (1 + erf(z / sqrt 2))
          o0 = 0.5f * o0 * (1.f + erff(o0 * 0.70710678118654752f));
          o1 = 0.5f * o1 * (1.f + erff(o1 * 0.70710678118654752f));
          o2 = 0.5f * o2 * (1.f + erff(o2 * 0.70710678118654752f));
          o3 = 0.5f * o3 * (1.f + erff(o3 * 0.70710678118654752f));
        }
        const int64_t off = (int64_t)row * N + n0 + c4;
        if constexpr (EPI == kEpiResidual) {
          const uint2 rw = *reinterpret_cast<const uint2*>(R + off);
          o0 += __uint_as_float(rw.x << 16);
          o1 += __uint_as_float(rw.x & 0xffff0000u);
          o2 += __uint_as_float(rw.y << 16);
          o3 += __uint_as_float(rw.y & 0xffff0000u);
        }
        *reinterpret_cast<uint2*>(D + off) = make_uint2(cvt_pk(o0, o1), cvt_pk(o2, o3));
      }
    }
    __syncthreads();
  }
}

// The same product with the k-stages moved by the direct-to-LDS loads (global_load_lds_dwordx4:
// each lane's 16 bytes go straight into the LDS, no registers or LDS store instructions in
// between), so that three stages can be in flight during the current one's products.
// Workgroup tile 256 x 256, 32-deep k-stages in a ring of four LDS stages (A slab 256 x 32,
// then B slab 256 x 32, 32 KB each), 16 waves as 4 x 4 of 64 x 64.  Slab rows are 64 bytes
// (four 16-byte chunks) without padding; chunk c of row r sits at position c ^ 2((r / 8) % 2),
// so that the 32 lanes of each ds_read_b128 pass (rows 0-15, two chunks each) cover the 64
// banks once.  A wave's load moves 16 consecutive rows (lane i: row i / 4, position i % 4).
// The four stages are separate arrays: the compiler then sees that a stage being read is not
// one whose loads are still in flight, and the loop waits on exactly the current stage's loads
// (per wave: two loads per stage, in issue order).  The loads of the last stages' successors
// re-read the last stage into a buffer nobody reads, so every wait counts the same.  Epilogue
// as gemm_bf16's, 64 rows at a time, each 16-row tile row staged in its own array.
// N a multiple of 256, K a multiple of 128; grid 8 ceil(MB / 8) (N / 256), 1024 threads, no
// dynamic LDS.
__shared__ uint4 gd_stage0[2048];
__shared__ uint4 gd_stage1[2048];
__shared__ uint4 gd_stage2[2048];
__shared__ uint4 gd_stage3[2048];

template <int EPI>
__global__ void __launch_bounds__(1024) gemm_dma(const bf16* __restrict__ A,
                                                 const bf16* __restrict__ Bt,
                                                 const bf16* __restrict__ bias,
                                                 const bf16* __restrict__ R,
                                                 bf16* __restrict__ D, int M, int N, int K) {
  constexpr int BM = 256, BN = 256, BK = 32, LDC = BN + 4;
  const int nbn = N / BN;
  const int g = blockIdx.x, xcd = g & 7, i = g >> 3;
  const int mb = (i / nbn) * 8 + xcd, nbk = i - (i / nbn) * nbn;
  const int m0 = mb * BM, n0 = nbk * BN;
  if (m0 >= M) return;  // padding workgroups: the whole group leaves before any barrier

  const int tid = threadIdx.x, lane = tid & 63, l16 = lane & 15, gq = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), wm = wave >> 2, wn = wave & 3;
  const int S = K / BK;
  // this lane's load: row 16 wave + lane / 4 of both slabs, chunk (lane % 4) ^ swizzle
  const int lr = lane >> 2, lc = (lane & 3) ^ (2 * ((lr >> 3) & 1));
  const bf16* ga = A + (int64_t)min(m0 + 16 * wave + lr, M - 1) * K + 8 * lc;
  const bf16* gb = Bt + (int64_t)(n0 + 16 * wave + lr) * K + 8 * lc;
  // this lane's operand slot in a 16-row group: row l16, chunk gq
  const int fs = 4 * l16 + (gq ^ (2 * ((l16 >> 3) & 1)));

  auto issue = [&](uint4* st, int s) {
    const int64_t kk = (int64_t)(s < S ? s : S - 1) * BK;
    __builtin_amdgcn_global_load_lds(ga + kk, st + 64 * wave, 16, 0, 0);
    __builtin_amdgcn_global_load_lds(gb + kk, st + 1024 + 64 * wave, 16, 0, 0);
  };
  f32x4 acc[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const uint4* st) {
    uint4 fa[4], fb[4];
#pragma unroll
    for (int a = 0; a < 4; ++a) fa[a] = st[(4 * wm + a) * 64 + fs];
#pragma unroll
    for (int b = 0; b < 4; ++b) fb[b] = st[1024 + (4 * wn + b) * 64 + fs];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < 4; ++b) acc[a][b] = mma_bf16(fa[a], fb[b], acc[a][b]);
  };
  // this wave's loads of the current stage done (the two later stages' four loads may still
  // be in flight), then every wave's: the barrier also tells that the stage read last is free
  auto sync = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0x0f74);  // vmcnt(4), no wait on the other counters
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  issue(gd_stage0, 0);
  issue(gd_stage1, 1);
  issue(gd_stage2, 2);
  for (int s = 0; s < S; s += 4) {
    sync();
    issue(gd_stage3, s + 3);
    compute(gd_stage0);
    sync();
    issue(gd_stage0, s + 4);
    compute(gd_stage1);
    sync();
    issue(gd_stage1, s + 5);
    compute(gd_stage2);
    sync();
    issue(gd_stage2, s + 6);
    compute(gd_stage3);
  }
  // the three surplus loads land before the stages are reused below
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");

  // ---- epilogue, one wave row (64 rows) at a time; tile row a in stage array a
  float* sc[4] = {reinterpret_cast<float*>(gd_stage0), reinterpret_cast<float*>(gd_stage1),
                  reinterpret_cast<float*>(gd_stage2), reinterpret_cast<float*>(gd_stage3)};
  float bv[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) bv[b] = (float)bias[n0 + 64 * wn + 16 * b + l16];
  constexpr int C4 = BN / 4;         // groups of 4 columns per row
  constexpr int PER = 64 * C4 / 1024;  // groups per thread
#pragma unroll 1
  for (int part = 0; part < 4; ++part) {
    if (wm == part) {
#pragma unroll
      for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            sc[a][(4 * gq + q) * LDC + 64 * wn + 16 * b + l16] = acc[a][b][q] + bv[b];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int c = tid + 1024 * j;
      const int r = c / C4, c4 = 4 * (c - (c / C4) * C4);
      const int row = m0 + 64 * part + r;
      const float* src = r < 16 ? sc[0] : r < 32 ? sc[1] : r < 48 ? sc[2] : sc[3];
      const float4 z = *reinterpret_cast<const float4*>(src + (r & 15) * LDC + c4);
      if (row < M) {
        float o0 = z.x, o1 = z.y, o2 = z.z, o3 = z.w;
        if constexpr (EPI == kEpiGelu) {  // GELU(z) = z Phi(z) = 0.5 z (1 + erf(z / sqrt 2))
          o0 = 0.5f * o0 * (1.f + erff(o0 * 0.70710678118654752f));
          o1 = 0.5f * o1 * (1.f + erff(o1 * 0.70710678118654752f));
          o2 = 0.5f * o2 * (1.f + erff(o2 * 0.70710678118654752f));
          o3 = 0.5f * o3 * (1.f + erff(o3 * 0.70710678118654752f));
        }
        const int64_t off = (int64_t)row * N + n0 + c4;
        if constexpr (EPI == kEpiResidual) {
          // streamed once: non-temporal, so that the output and residual streams do not
          // push the operands' k-slices out of the caches
          const unsigned long long rq =
              __builtin_nontemporal_load(reinterpret_cast<const unsigned long long*>(R + off));
          const uint2 rw = make_uint2((uint32_t)rq, (uint32_t)(rq >> 32));
          o0 += __uint_as_float(rw.x << 16);
          o1 += __uint_as_float(rw.x & 0xffff0000u);
          o2 += __uint_as_float(rw.y << 16);
          o3 += __uint_as_float(rw.y & 0xffff0000u);
        }
        __builtin_nontemporal_store(
            (unsigned long long)cvt_pk(o0, o1) | ((unsigned long long)cvt_pk(o2, o3) << 32),
            reinterpret_cast<unsigned long long*>(D + off));
      }
    }
    __syncthreads();
  }
}

}  // namespace afno
