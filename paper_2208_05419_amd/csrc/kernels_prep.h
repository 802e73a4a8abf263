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

// The H-th roots of unity the transform table is made of: roots[m] = (cos, sin)(2 pi m / H),
// m < H, computed by the workgroup's threads (the same single-precision sincospif values
// dft_table_word takes).  Ends with a barrier: every thread of the workgroup must call it.
__device__ __forceinline__ void dft_roots(float2* roots, int H) {
  for (int m = threadIdx.x; m < H; m += blockDim.x) {
    float sn, cs;
    sincospif(2.0f * (float)m / (float)H, &sn, &cs);
    roots[m] = make_float2(cs, sn);
  }
  __syncthreads();
}

// One column (sigma, j) of the transform table: T[(sigma, r)][j] for every r < HP, stored as
// the HP / 8 fragment words of dft_table_word's order that hold it, from the roots of
// dft_roots.  The matrix-core column kernels apply this one table in both directions, and the
// inverse's sum over the kept rows k of T[(sigma, k)][h] O[k] meets a component of O that is
// the same at every kept row (the biases put one there, tens of times the rest): with each
// entry rounded to the nearest bf16 on its own, that component carries the column's summed
// rounding error (about sqrt(H) half-ulps) onto every output row h instead of row 0 alone.  So
// the entries of the kept rows (|signed r| < kept_h, every row when kept_h > H / 2) are
// rounded in turn with the error carried forward: entry r takes the bf16 nearest to v_r - e,
// e the sum of the earlier entries' errors, which keeps every partial column sum within half
// an ulp of its exact value while each entry stays within about one ulp of v_r.
__device__ __forceinline__ void dft_table_column(int task, int H, int HP, int kept_h,
                                                 const float2* roots, uint4* tout) {
  const int sigma = task / HP, j = task - sigma * HP;
  const int KT = HP / 16;
  const float sc = 1.0f / sqrtf((float)H);
  const bool all_rows = kept_h > H / 2;
  const int jm = j < H ? j : 0;
  float err = 0.f;
  int m = 0;  // (r j) mod H, stepped
  for (int r0 = 0; r0 < HP; r0 += 8) {
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int r = r0 + e;
      v[e] = 0.f;
      if (r < H && j < H) {
        const float2 z = roots[m];
        v[e] = sigma == 0 ? z.x * sc : -z.y * sc;
      }
      m += jm;
      m = m >= H ? m - H : m;
    }
    union { uint4 u; bf16 h[8]; } w;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int r = r0 + e;
      const bool carry = r < H && (all_rows || row_kept(r, H, kept_h));
      const bf16 b = (bf16)(carry ? v[e] - err : v[e]);
      if (carry) err += (float)b - v[e];
      w.h[e] = b;
    }
    // the 8 entries of K rows sigma HP + r0 .. + 7 make one fragment word of column j
    const int kap = sigma * HP + r0;
    tout[((int64_t)(kap >> 5) * KT + (j >> 4)) * 64 + (j & 15) + 16 * ((kap >> 3) & 3)] = w.u;
  }
}

// The two tables of the kept-row column kernel (kernels_kept_mfma.h) for height H padded to
// HP and KP kept rows (kept_row): the forward table Tf[(sigma, h)][k'] = T[(sigma, h)][kept_row(k')]
// (K = 2 HP, N = KP; zero for h >= H or k' >= 2 kept_h - 1), fragment word by word with every
// entry rounded to nearest, then the inverse table Ti[(sigma, k')][h] = T[(sigma, kept_row(k'))][h]
// (K = 2 KP, N = HP), one column (sigma, h) per task with dft_table_column's error carry over
// the kept rows.  Tasks: DKS KT 64 words, then 2 HP columns.  roots: dft_roots.
__host__ __device__ inline int64_t kept_table_tasks(int HP, int KP) {
  return (int64_t)(2 * HP / 32) * (KP / 16) * 64 + 2 * HP;
}
__device__ __forceinline__ void kept_table_task(int64_t i, int H, int HP, int KP, int kept_h,
                                                const float2* roots, uint4* tout) {
  const int KT = KP / 16, HT = HP / 16;
  const int64_t ntf = (int64_t)(2 * HP / 32) * KT * 64;
  const float sc = 1.0f / sqrtf((float)H);
  const int nkept = 2 * kept_h - 1;
  if (i < ntf) {
    const int lane = (int)(i & 63);
    const int f = (int)(i >> 6);
    const int t = f % KT, s = f / KT;
    const int kp = 16 * t + (lane & 15);
    union { uint4 u; bf16 h[8]; } w;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int kap = 32 * s + 8 * (lane >> 4) + e;
      const int sigma = kap / HP, h = kap % HP;
      float v = 0.f;
      if (h < H && kp < nkept) {
        const float2 z = roots[(h * kept_row(kp, H, kept_h)) % H];
        v = sigma == 0 ? z.x * sc : -z.y * sc;
      }
      w.h[e] = (bf16)v;
    }
    tout[i] = w.u;
    return;
  }
  const int task = (int)(i - ntf);  // column (sigma, h) of Ti
  const int sigma = task / HP, h = task - sigma * HP;
  uint4* ti = tout + ntf;
  float err = 0.f;
  for (int kp0 = 0; kp0 < KP; kp0 += 8) {
    union { uint4 u; bf16 h[8]; } w;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int kp = kp0 + e;
      float v = 0.f;
      if (h < H && kp < nkept) {
        const float2 z = roots[(kept_row(kp, H, kept_h) * h) % H];
        v = sigma == 0 ? z.x * sc : -z.y * sc;
      }
      const bool carry = kp < nkept;
      const bf16 b = (bf16)(carry ? v - err : v);
      if (carry) err += (float)b - v;
      w.h[e] = b;
    }
    const int kap = sigma * KP + kp0;  // 8 K rows: one fragment word of column h
    ti[((int64_t)(kap >> 5) * HT + (h >> 4)) * 64 + (h & 15) + 16 * ((kap >> 3) & 3)] = w.u;
  }
}

// fragment words of the hidden-size block weights (bf16, hidden size hs: per block layer 1,
// (2 bs / 32) k-steps x (2 hs / 16) n-tiles, then layer 2, (2 hs / 32) x (2 bs / 16)), after
// the DFT table's 2 HP column tasks (dft_table_column), tasks i, i + stride, ...
__device__ __forceinline__ void prep_hidden_words(int64_t i, int64_t stride, const bf16* w1,
                                                  const bf16* w2, uint4* wout, uint4* tout,
                                                  int nb, int bs, int hs, int H, int HP,
                                                  int kept_h, const float2* roots) {
  const int mh = 2 * hs / 16, mt = 2 * bs / 16;
  const int64_t l1 = (int64_t)(2 * bs / 32) * mh * 64;
  const int64_t per_block = 2 * l1;
  const int64_t nw = (int64_t)nb * per_block;
  // the table's column tasks first: each is a sequential pass over a column, so they start
  // in the launch's first workgroup
  const int64_t ntab = tout ? (int64_t)2 * HP : 0;
  const int64_t total = nw + ntab;
  for (; i < total; i += stride) {
    if (i < ntab) {
      dft_table_column((int)i, H, HP, kept_h, roots, tout);
      continue;
    }
    const int64_t q = i - ntab;  // weight word q
    const int64_t blk = q / per_block;
    int64_t u = q - blk * per_block;
    const int layer = u >= l1 ? 1 : 0;
    u -= layer * l1;
    const int lane = (int)(u & 63);
    const int64_t f = u >> 6;
    const int nt = layer ? mt : mh;                 // output tiles of the layer
    const int t = (int)(f % nt), s = (int)(f / nt);
    const bf16* w = layer ? w2 + blk * (int64_t)hs * bs * 2 : w1 + blk * (int64_t)bs * hs * 2;
    const int n_out = layer ? bs : hs;
    const int j = (16 * t + (lane & 15)) >> 1;
    wout[q] = FragWord<bf16>::make(w, n_out, s * 32, j, lane & 1, lane);
  }
}

// What to prepare: both layers of every block in fragment order (frag_words_per_block words
// per block, word ((layer * KSTEPS + s) * NT16 + t) * 64 + lane), then, if tout is set, the
// DFT table for height H padded to HP: kept_h >= 0, 2 HP column tasks (dft_table_column, the
// rounding that carries its error over the kept rows; needs dft_roots); kept_h < 0, one task
// per fragment word (dft_table_word, every entry rounded to nearest).
template <typename T>
struct PrepJob {
  const T* w1;
  const T* w2;
  typename FragWord<T>::type* wout;
  uint4* tout;
  int nb, bs, H, HP;
  int nprep;   // workgroups the host launch gives the job (placed before its own work)
  int kept_h;  // the table's rounding, as above
  int kp;      // > 0: the kept-row kernel's two tables for kp kept rows (kept_table_task)
  int hs;      // > 0 and != bs (bf16): the hidden-size kernel's fragments (prep_hidden_words)
};

__host__ __device__ inline int64_t dft_table_tasks(int HP, int kept_h) {
  return kept_h >= 0 ? (int64_t)2 * HP : (int64_t)(2 * HP / 32) * (HP / 16) * 64;
}

template <typename T>
__device__ __forceinline__ int64_t prep_words(const PrepJob<T>& pj) {
  if (sizeof(T) == 2 && pj.hs > 0 && pj.hs != pj.bs)
    return (int64_t)pj.nb * 2 * (2 * pj.bs / 32) * (2 * pj.hs / 16) * 64 + (pj.tout ? 2 * pj.HP : 0);
  return (int64_t)pj.nb * frag_words_per_block<T>(pj.bs) +
         (pj.tout ? (pj.kp > 0 ? kept_table_tasks(pj.HP, pj.kp) : dft_table_tasks(pj.HP, pj.kept_h))
                  : 0);
}

// Tasks i, i + stride, ... of the job: one fragment word of the weights each, then the table
// tasks.  roots: dft_roots' values (needed when pj.tout is set and pj.kept_h >= 0).
template <typename T>
__device__ void prep_operands(int64_t i, int64_t stride, const PrepJob<T>& pj,
                              const float2* roots) {
  if constexpr (sizeof(T) == 2) {
    if (pj.hs > 0 && pj.hs != pj.bs) {
      prep_hidden_words(i, stride, pj.w1, pj.w2, pj.wout, pj.tout, pj.nb, pj.bs, pj.hs, pj.H,
                        pj.HP, pj.kept_h, roots);
      return;
    }
  }
  const int nt16 = 2 * pj.bs / 16, ksteps = 2 * pj.bs / Mma<T>::kK;
  const int64_t nw = (int64_t)pj.nb * frag_words_per_block<T>(pj.bs);
  const int64_t total = prep_words(pj);
  for (; i < total; i += stride) {
    if (i >= nw) {
      if (pj.kp > 0)
        kept_table_task(i - nw, pj.H, pj.HP, pj.kp, pj.kept_h, roots, pj.tout);
      else if (pj.kept_h >= 0)
        dft_table_column((int)(i - nw), pj.H, pj.HP, pj.kept_h, roots, pj.tout);
      else
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

// The job as its own launch (grid-stride over the tasks).  H <= 96 when the table is made.
template <typename T>
__global__ void __launch_bounds__(256) prep_operands_kernel(PrepJob<T> pj) {
  __shared__ float2 roots[96];
  if (pj.tout && pj.kept_h >= 0) dft_roots(roots, pj.H);
  prep_operands<T>(blockIdx.x * (int64_t)blockDim.x + threadIdx.x, (int64_t)gridDim.x * blockDim.x,
                   pj, roots);
}

}  // namespace afno
