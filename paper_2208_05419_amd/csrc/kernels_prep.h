// kernels_prep.h -- the column kernels' prepared operands: the block weights re-laid in MFMA
// fragment order, and the bf16 H-axis DFT table.  Written once per call into the workspace,
// either by their own launch or by extra workgroups appended to the W-axis forward launch.
#pragma once
#include "kernel_common.h"

namespace afno {

// Transform table in fragment order: word (s * KT + t) * 64 + lane holds the B fragment of
// k-step s and column tile t (lane: column 16 t + lane % 16, K rows 32 s + 8 (lane / 16) ...
// + 7) of T[(sigma, i)][j] = Re (sigma 0) / Im (sigma 1) of exp(-2 pi i i j / H) / sqrt(H),
// zero for i >= H or j >= H.  Entries rounded to bf16 from single precision.
__device__ __forceinline__ uint4 dft_table_word(int64_t i, int H, int HP) {
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
      const int m = (r * j) % H;  // the argument reduced exactly: 2 m / H in [0, 2)
      float sn, cs;
      sincospif(2.0f * (float)m / (float)H, &sn, &cs);
      v = sigma == 0 ? cs * sc : -sn * sc;
    }
    w.h[e] = (bf16)v;  // float is accurate far below the bf16 rounding step
  }
  return w.u;
}

// What to prepare: both layers of every block in fragment order (frag_words_per_block words
// per block, word ((layer * KSTEPS + s) * NT16 + t) * 64 + lane), then, if tout is set, the
// DFT table for height H padded to HP.
template <typename T>
struct PrepJob {
  const T* w1;
  const T* w2;
  typename FragWord<T>::type* wout;
  uint4* tout;
  int nb, bs, H, HP;
  int nmain;  // workgroups of the host launch's own work (the prepared words come after)
};

template <typename T>
__device__ __forceinline__ int64_t prep_words(const PrepJob<T>& pj) {
  return (int64_t)pj.nb * frag_words_per_block<T>(pj.bs) +
         (pj.tout ? (int64_t)(2 * pj.HP / 32) * (pj.HP / 16) * 64 : 0);
}

// Words i, i + stride, ... of the job.
template <typename T>
__device__ void prep_operands(int64_t i, int64_t stride, const PrepJob<T>& pj) {
  const int nt16 = 2 * pj.bs / 16, ksteps = 2 * pj.bs / Mma<T>::kK;
  const int64_t nw = (int64_t)pj.nb * frag_words_per_block<T>(pj.bs);
  const int64_t total = prep_words(pj);
  for (; i < total; i += stride) {
    if (i >= nw) {
      pj.tout[i - nw] = dft_table_word(i - nw, pj.H, pj.HP);
      continue;
    }
    const int lane = (int)(i & 63);
    int64_t f = i >> 6;
    const int t = (int)(f % nt16);
    f /= nt16;
    const int s = (int)(f % ksteps);
    f /= ksteps;
    const int layer = (int)(f & 1);
    const int64_t blk = f >> 1;
    const T* w = (layer ? pj.w2 : pj.w1) + blk * pj.bs * pj.bs * 2;
    const int j = (16 * t + (lane & 15)) >> 1;
    pj.wout[i] = FragWord<T>::make(w, pj.bs, s * Mma<T>::kK, j, lane & 1, lane);
  }
}

// The job as its own launch (grid-stride over the words).
template <typename T>
__global__ void __launch_bounds__(256) prep_operands_kernel(PrepJob<T> pj) {
  prep_operands<T>(blockIdx.x * (int64_t)blockDim.x + threadIdx.x, (int64_t)gridDim.x * blockDim.x, pj);
}

}  // namespace afno
