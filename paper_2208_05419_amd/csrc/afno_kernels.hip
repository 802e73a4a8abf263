// afno_kernels.hip -- launch sequence of the AFNO spectral filter on gfx950: picks the
// size-specialised kernels of kernels_fast.h where one exists for the grid, else the
// size-generic kernels of kernels_generic.h.
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
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <type_traits>

#include "afno_internal.h"
#include "kernels_fast.h"
#include "kernels_generic.h"
#include "kernels_mfma.h"
#include "kernels_hidden_mfma.h"
#include "kernels_kept_mfma.h"
#include "kernels_backward.h"
#include "kernels_backward_mfma.h"
#include "kernels_block.h"

namespace afno {

// ------------------------------------------------------------------ size-specialised dispatch
//
// W-axis kernels: W = N1 N2, NP complex signals (2 NP channels) per workgroup.
//   W = 32: 8 x 4, NP 32;  W = 180: 12 x 15, NP 32;  W = 360: 24 x 15, NP 16.
// Column kernel, bf16 with H <= 96 and BS in {32, 64, 96}: H transforms as MFMA products
//   against a transform table (kernels_mfma.h), H padded to HP in {32, 64, 96}.
// Column kernel, vector-ALU transforms: H = N1 N2 with block size BS.
//   H = 16, BS = 16: 4 x 4;  H = 90, BS = 96: 9 x 10;  H = 180, BS = 32: 12 x 15;
//   H = 180, BS = 64 and 128: 12 x 15 (bf16 only, with a bf16 transform intermediate: a
//   float one would not fit the LDS).
int mfma_col_hp(int64_t H) { return H <= 32 ? 32 : (H <= 64 ? 64 : 96); }

size_t hidden_frag_bytes(const Plan& pl);

// tasks of the preparation job: the fragment-ordered weights' words (hidden = true: the
// hidden-size kernel's), and the DFT table's columns if with_tab
static int64_t prep_words_host(const Plan& pl, bool with_tab, int kept_h, int kp = 0,
                               bool hidden = false) {
  const int hp = mfma_col_hp(pl.H);
  if (hidden) return (int64_t)hidden_frag_bytes(pl) / 16 + (with_tab ? 2 * hp : 0);
  return pl.nb * (pl.dtype == 0 ? frag_words_per_block<float>((int)pl.bs)
                                : frag_words_per_block<bf16>((int)pl.bs)) +
         (with_tab ? (kp > 0 ? kept_table_tasks(hp, kp) : dft_table_tasks(hp, kept_h)) : 0);
}

// Size-specialised W-axis kernels: (W, N1, N2, NP), W = N1 N2 split into an N2-point register
// stage and an N1-point stage after the LDS exchange, NP complex signals (2 NP channels) per
// workgroup.  Splits and slice widths are the measured fastest per direction (W = 180: forward
// 12 x 15 on 32 channels, inverse 15 x 12 on 64; W = 360: 15 x 24 on 32 channels both ways).
#define AFNO_ROW_FAST_LIST(X) X(32, 8, 4, 32) X(180, 12, 15, 16) X(360, 15, 24, 16)
#define AFNO_ROW_INV_LIST(X) X(32, 8, 4, 32) X(180, 15, 12, 32) X(360, 15, 24, 16)
// both directions specialised for W, and C a whole number of slices in each
bool fast_row_available(int64_t W, int64_t C) {
  bool fwd = false, inv = false;
#define AFNO_CASE(w, n1, n2, np) if (W == w) fwd = C % (2 * np) == 0;
  AFNO_ROW_FAST_LIST(AFNO_CASE)
#undef AFNO_CASE
#define AFNO_CASE(w, n1, n2, np) if (W == w) inv = C % (2 * np) == 0;
  AFNO_ROW_INV_LIST(AFNO_CASE)
#undef AFNO_CASE
  return fwd && inv;
}

bool fast_col_available(int dtype, int64_t H, int64_t bs) {
  if ((H == 16 && bs == 16) || (H == 90 && bs == 96) || (H == 180 && bs == 32)) return true;
  return dtype == 1 && H == 180 && (bs == 64 || bs == 128);
}

// pj.tout / pj.wout null: no preparation job; else its words go to extra workgroups
template <typename T>
static void launch_row_fwd_fast(const Plan& pl, const T* x, T* S, PrepJob<T> pj, hipStream_t st) {
  const unsigned gx = (unsigned)(pl.B * pl.H);
  const float sc = 0.5f * pl.row.inv_sqrt_w;
#define AFNO_CASE(w, n1, n2, np)                                                          \
  if (pl.W == w) {                                                                        \
    const unsigned nmain = (unsigned)row_grid<np, (int)sizeof(T)>(gx, (int)(pl.C / (2 * np))); \
    const unsigned nprep = pj.wout ? (unsigned)(std::min<int64_t>(                        \
        (prep_words_host(pl, pj.tout != nullptr, pj.kept_h, pj.kp, pj.hs > 0) + np * n1 - 1) / (np * n1), 1024) \
        + 7) / 8 * 8 : 0;                                                                 \
    pj.nprep = (int)nprep;                                                                \
    hipLaunchKernelGGL((row_r2c_fast<T, w, n1, n2, np>), dim3(nprep + nmain),              \
                       dim3(np * n1), 0, st, x, S, (int)pl.C, (int)pl.KW, sc, (int64_t)gx, pj); \
    return;                                                                               \
  }
  AFNO_ROW_FAST_LIST(AFNO_CASE)
#undef AFNO_CASE
}

template <typename T>
static void launch_row_inv_fast(const Plan& pl, const T* S, const T* x, T* out, float* dst,
                                int mode, hipStream_t st) {
  const unsigned gx = (unsigned)(pl.B * pl.H);
  const float sc = pl.row.inv_sqrt_w;
#define AFNO_CASE(w, n1, n2, np)                                                          \
  if (pl.W == w) {                                                                        \
    const unsigned ng = (unsigned)row_grid<np, (int)sizeof(T)>(gx, (int)(pl.C / (2 * np))); \
    hipLaunchKernelGGL((row_c2r_fast<T, w, n1, n2, np>), dim3(ng), dim3(np * n1), 0, st,  \
                       S, x, out, dst, (int)pl.C, (int)pl.KW, sc, mode, (int64_t)gx);     \
    return;                                                                               \
  }
  AFNO_ROW_INV_LIST(AFNO_CASE)
#undef AFNO_CASE
}

template <typename T, typename FT, int H, int N1, int N2, int BS, int WPE,
          int NT = ColShape<BS>::kThreads>
static void launch_col_fast_one(const Plan& pl, T* S, const typename FragWord<T>::type* wf,
                                const T* b1, const T* b2, int stage, hipStream_t st) {
  constexpr int lds = ColLds<T, FT, H, BS>::kBytes;
  constexpr int nthr = NT;
  hipLaunchKernelGGL((column_fast<T, FT, H, N1, N2, BS, WPE, NT>), dim3((unsigned)(pl.B * pl.KW * pl.nb)),
                     dim3(nthr), lds, st, S, wf, b1, b2, (int)pl.C, (int)pl.KW, (int)pl.nb,
                     (int)pl.kept_h, pl.col.lam, pl.col.inv_sqrt_h, stage);
}

template <typename T>
static void launch_col_fast(const Plan& pl, T* S, const T* b1, const T* b2, int stage,
                            hipStream_t st) {
  typedef typename FragWord<T>::type Word;
  const Word* wf = reinterpret_cast<const Word*>(reinterpret_cast<const char*>(S) + pl.frag_offset);
  if (pl.H == 16 && pl.bs == 16)
    launch_col_fast_one<T, float, 16, 4, 4, 16, 4>(pl, S, wf, b1, b2, stage, st);
  else if (pl.H == 90 && pl.bs == 96)
    launch_col_fast_one<T, float, 90, 9, 10, 96, 4, 512>(pl, S, wf, b1, b2, stage, st);
  else if (pl.H == 180 && pl.bs == 32)
    launch_col_fast_one<T, float, 180, 12, 15, 32, 6, 512>(pl, S, wf, b1, b2, stage, st);
  else if constexpr (sizeof(T) == 2) {
    if (pl.bs == 64)
      launch_col_fast_one<T, bf16, 180, 12, 15, 64, 3, 256>(pl, S, wf, b1, b2, stage, st);
    else
      launch_col_fast_one<T, bf16, 180, 12, 15, 128, 4, 1024>(pl, S, wf, b1, b2, stage, st);
  }
}

#define AFNO_MFMA_COL_LIST(X) \
  X(32, 32) X(32, 64) X(32, 96) X(64, 32) X(64, 64) X(64, 96) X(96, 32) X(96, 64) X(96, 96)

bool mfma_col_available(int dtype, int64_t H, int64_t bs) {
  return dtype == 1 && H <= 96 && (bs == 32 || bs == 64 || bs == 96);
}

size_t mfma_tab_bytes(const Plan& pl) {
  const int hp = mfma_col_hp(pl.H);
  return (size_t)(2 * hp / 32) * (hp / 16) * 64 * 16;
}

// the kept-row column kernel (kernels_kept_mfma.h): bf16, block size 96, 64 < H <= 96, and a
// cutoff that keeps at most 48 rows (2 kept_h - 1 <= 48); 0 elsewhere, else the padded count
int mfma_kept_rows(const Plan& pl) {
  if (pl.path != 0 || pl.dtype != 1 || pl.col.hs != pl.bs || pl.bs != 96 || pl.H <= 64 ||
      pl.H > 96 || pl.kept_h < 1 || pl.kept_h > pl.H / 2)
    return 0;
  const int64_t nkept = 2 * pl.kept_h - 1;
  return nkept <= 48 ? (int)((nkept + 15) / 16 * 16) : 0;
}

#define AFNO_KEPT_LIST(X) X(16) X(32) X(48)

size_t kept_tab_bytes(int kp) {
  switch (kp) {
#define AFNO_CASE(KP_) case KP_: return (size_t)KeptCol<96, 96, KP_>::kTabBytes;
    AFNO_KEPT_LIST(AFNO_CASE)
#undef AFNO_CASE
  }
  return 0;
}

// the forward's transform tables: the kept-row kernel's where it runs, and the full table (for
// the diagnostic spectrum stage, which needs every row)
size_t fwd_tab_bytes(const Plan& pl) {
  return std::max(mfma_tab_bytes(pl), kept_tab_bytes(mfma_kept_rows(pl)));
}

static void launch_col_mfma(const Plan& pl, bf16* S, const bf16* b1, const bf16* b2, int stage,
                            hipStream_t st) {
  const uint4* wf = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(S) + pl.frag_offset);
  const uint4* tab = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(S) + pl.tab_offset);
  const int hp = mfma_col_hp(pl.H);
  const dim3 grid((unsigned)(pl.B * pl.KW * pl.nb));
  const int kp = stage == 1 ? 0 : mfma_kept_rows(pl);
#define AFNO_CASE(KP_)                                                                      \
  if (kp == KP_) {                                                                          \
    hipLaunchKernelGGL((column_mfma_kept<96, 96, KP_>), grid, dim3(384),                   \
                       (KeptCol<96, 96, KP_>::kBytes), st, S, wf, tab, b1, b2, (int)pl.H,   \
                       (int)pl.C, (int)pl.KW, (int)pl.nb, (int)pl.kept_h, pl.col.lam, stage); \
    return;                                                                                 \
  }
  AFNO_KEPT_LIST(AFNO_CASE)
#undef AFNO_CASE
#define AFNO_CASE(HP_, BS_)                                                                 \
  if (hp == HP_ && pl.bs == BS_) {                                                          \
    constexpr int lds = MfmaCol<HP_, BS_>::kBytes;                                          \
    hipLaunchKernelGGL((column_mfma<HP_, BS_>), grid, dim3(512), lds, st,                  \
                       S, wf, tab, b1, b2, (int)pl.H, (int)pl.C, (int)pl.KW, (int)pl.nb,   \
                       (int)pl.kept_h, pl.col.lam, stage);                                  \
    return;                                                                                 \
  }
  AFNO_MFMA_COL_LIST(AFNO_CASE)
#undef AFNO_CASE
}

#define AFNO_MFMA_HID_LIST(X)                                                               \
  X(32, 32, 64) X(32, 64, 128) X(32, 96, 192) X(64, 32, 64) X(64, 64, 128) X(64, 96, 192)   \
  X(96, 32, 64) X(96, 64, 128) X(96, 96, 192)

// the matrix-core column kernel for hidden = 2 bs (bf16, H <= 96, bs 32 / 64 / 96)
static bool mfma_hidden_available(int dtype, int64_t H, int64_t bs, int64_t hs) {
  return dtype == 1 && H <= 96 && (bs == 32 || bs == 64 || bs == 96) && hs == 2 * bs;
}

size_t hidden_frag_bytes(const Plan& pl) {
  return (size_t)pl.nb * 2 * (size_t)(2 * pl.bs / 32) * (size_t)(2 * pl.col.hs / 16) * 64 * 16;
}

static void launch_col_mfma_hidden(const Plan& pl, bf16* S, const bf16* b1, const bf16* b2,
                                   hipStream_t st) {
  const uint4* wf = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(S) + pl.frag_offset);
  const uint4* tab = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(S) + pl.tab_offset);
  const int hp = mfma_col_hp(pl.H);
  const dim3 grid((unsigned)(pl.B * pl.KW * pl.nb));
#define AFNO_CASE(HP_, BS_, HS_)                                                            \
  if (hp == HP_ && pl.bs == BS_ && pl.col.hs == HS_) {                                      \
    hipLaunchKernelGGL((column_mfma_hidden<HP_, BS_, HS_>), grid, dim3(512),                \
                       (MfmaHid<HP_, BS_, HS_>::kBytes), st, S, wf, tab, b1, b2, (int)pl.H, \
                       (int)pl.C, (int)pl.KW, (int)pl.nb, (int)pl.kept_h, pl.col.lam);       \
    return;                                                                                 \
  }
  AFNO_MFMA_HID_LIST(AFNO_CASE)
#undef AFNO_CASE
}

// ------------------------------------------------------------------ launchers

// 0: MFMA-transform column kernel, else size-specialised, else generic; 1: generic only;
// 2: as 0 without the MFMA-transform column kernel.  A plan takes the value once (make_plan),
// so a call's workspace sizing and its launches agree even if another thread switches it.
static std::atomic<int> g_kernel_path{0};

void set_kernel_path(int path) { g_kernel_path.store(path); }
int kernel_path() { return g_kernel_path.load(); }

bool use_mfma_col(const Plan& pl) {
  return pl.path == 0 && pl.col.hs == pl.bs && mfma_col_available(pl.dtype, pl.H, pl.bs);
}

bool use_mfma_hidden(const Plan& pl) {
  return pl.path == 0 && pl.col.hs != pl.bs &&
         mfma_hidden_available(pl.dtype, pl.H, pl.bs, pl.col.hs);
}

bool use_fast_col(const Plan& pl) {
  return pl.path != 1 && pl.col.hs == pl.bs && !use_mfma_col(pl) &&
         fast_col_available(pl.dtype, pl.H, pl.bs);
}

size_t frag_bytes(const Plan& pl) {
  return (size_t)pl.nb * (size_t)(pl.dtype == 0 ? frag_words_per_block<float>((int)pl.bs) * 4
                                                 : frag_words_per_block<bf16>((int)pl.bs) * 16);
}

template <typename T>
static hipError_t launch_all(const Plan& pl, const void* x, const void* w1, const void* b1,
                             const void* w2, const void* b2, void* S, void* out, float* dst,
                             int stage, hipStream_t st, hipEvent_t* ev) {
  const T* xt = static_cast<const T*>(x);
  T* St = static_cast<T*>(S);
  const bool generic = pl.path == 1;
  const bool row_fast = !generic && fast_row_available(pl.W, pl.C);
  const bool col_mfma = use_mfma_col(pl);
  const bool col_fast = use_fast_col(pl);
  const bool col_hid = use_mfma_hidden(pl);
  dim3 rgrid((unsigned)(pl.B * pl.H), (unsigned)(pl.C / pl.row.rc));
  // prepared column-kernel operands (after the spectrum in the workspace; independent of x):
  // extra workgroups of the size-specialised W-axis forward launch, else a launch of their own
  PrepJob<T> pj{static_cast<const T*>(w1), static_cast<const T*>(w2), nullptr, nullptr,
                (int)pl.nb, (int)pl.bs, (int)pl.H, mfma_col_hp(pl.H), 0, (int)pl.kept_h,
                stage == kStageSpectrum ? 0 : mfma_kept_rows(pl)};
  if (col_mfma || col_fast || (sizeof(T) == 2 && col_hid))
    pj.wout = reinterpret_cast<typename FragWord<T>::type*>(static_cast<char*>(S) + pl.frag_offset);
  if (col_mfma || (sizeof(T) == 2 && col_hid))
    pj.tout = reinterpret_cast<uint4*>(static_cast<char*>(S) + pl.tab_offset);
  if (sizeof(T) == 2 && col_hid) pj.hs = (int)pl.col.hs;  // the hidden-size kernel's fragments
  // ev[0]: recorded only before a preparation launch of its own (a preparation inside the W-axis
  // forward launch belongs to that phase; the profile counts an unrecorded ev[0] as zero)
  const bool prep_launch = pj.wout && !row_fast;
  if (ev && prep_launch) (void)hipEventRecord(ev[0], st);
  if (prep_launch) {
    const unsigned g = (unsigned)std::min<int64_t>(
        (prep_words_host(pl, pj.tout != nullptr, pj.kept_h, pj.kp, pj.hs > 0) + 255) / 256, 4096);
    hipLaunchKernelGGL(prep_operands_kernel<T>, dim3(g), dim3(256), 0, st, pj);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[1], st);
  if (row_fast)
    launch_row_fwd_fast<T>(pl, xt, St, pj, st);
  else
    hipLaunchKernelGGL(row_r2c_kernel<T>, rgrid, dim3(kRowThreads), pl.row_lds, st, xt, St, pl.row);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[2], st);
  const int col_stage = (stage == kStageSpectrum) ? 1 : (stage == kStageMixed ? 2 : 0);
  if (col_mfma) {
    if constexpr (sizeof(T) == 2)
      launch_col_mfma(pl, St, static_cast<const bf16*>(b1), static_cast<const bf16*>(b2),
                      col_stage, st);
  } else if (col_hid && col_stage == 0) {
    if constexpr (sizeof(T) == 2)
      launch_col_mfma_hidden(pl, St, static_cast<const bf16*>(b1), static_cast<const bf16*>(b2), st);
  } else if (col_fast)
    launch_col_fast<T>(pl, St, static_cast<const T*>(b1), static_cast<const T*>(b2), col_stage, st);
  else
    hipLaunchKernelGGL(column_kernel<T>, dim3((unsigned)(pl.B * pl.KW * pl.nb)),
                       dim3(pl.col_threads), pl.col_lds, st, St, static_cast<const T*>(w1),
                       static_cast<const T*>(b1), static_cast<const T*>(w2),
                       static_cast<const T*>(b2), pl.col, col_stage);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (ev) (void)hipEventRecord(ev[3], st);
  if (stage == kStageSpectrum || stage == kStageMixed) {
    const int64_t total = pl.B * pl.H * (pl.W / 2 + 1) * pl.C * 2;
    const unsigned g = (unsigned)std::min<int64_t>((total + 255) / 256, 65536);
    hipLaunchKernelGGL(export_spectrum_kernel<T>, dim3(g), dim3(256), 0, st, St, dst, pl.B,
                       (int)pl.H, (int)(pl.W / 2 + 1), (int)pl.KW, (int)pl.C);
    return hipGetLastError();
  }
  const int mode = stage == kStageDelta ? 1 : 0;
  if (row_fast)
    launch_row_inv_fast<T>(pl, St, xt, static_cast<T*>(out), dst, mode, st);
  else
    hipLaunchKernelGGL(row_c2r_kernel<T>, rgrid, dim3(kRowThreads), pl.row_lds, st, St, xt,
                       static_cast<T*>(out), dst, pl.row, mode);
  e = hipGetLastError();
  if (ev && e == hipSuccess) (void)hipEventRecord(ev[4], st);
  return e;
}

// ------------------------------------------------------------------ backward pass

// the backward column pass runs the bf16 matrix-core kernel where the forward would (auto
// path), else the size-generic one
bool use_mfma_bwd(const Plan& pl) { return use_mfma_col(pl); }

int64_t bwd_mpad(const Plan& pl) { return pl.B * pl.KW * (int64_t)col_bwd_hc((int)pl.col.H16); }

size_t bwd_lds(const Plan& pl) {
  if (use_mfma_bwd(pl)) {
    const int hp = mfma_col_hp(pl.H);
#define AFNO_CASE(HP_, BS_) \
    if (hp == HP_ && pl.bs == BS_) return (size_t)MfmaBwd<HP_, BS_>::kBytes;
    AFNO_MFMA_COL_LIST(AFNO_CASE)
#undef AFNO_CASE
  }
  return col_bwd_lds(pl.col);
}

// workspace bytes of the prepared operands of the matrix-core backward column kernel: the
// forward and the backward weight fragments, the DFT table and its rounding remainders
size_t bwd_prep_bytes(const Plan& pl) {
  if (!use_mfma_bwd(pl)) return 0;
  return 2 * frag_bytes(pl) + 2 * mfma_tab_bytes(pl);
}

// chunks of the slab weight-gradient kernel (bf16, 2 bs = 64, 128 or 192), 0 where the
// tiled kernel runs instead; *kchunk: modes per chunk (a multiple of 64).  About one
// workgroup per compute unit; a chunk's byte offsets stay 32-bit.
int wgrad_slab_chunks(const Plan& pl, int* kchunk) {
  const int64_t nb2 = 2 * pl.bs;
  if (pl.dtype != 1 || (nb2 != 64 && nb2 != 128 && nb2 != 192)) return 0;
  const int64_t mpad = bwd_mpad(pl);
  const int64_t want = std::max<int64_t>(1, std::min<int64_t>(64, 256 / (2 * pl.nb)));
  const int64_t kc = std::max<int64_t>(64, ((mpad + want - 1) / want + 63) / 64 * 64);
  if ((kc / 8 + 3 * 8) * nb2 * 16 > (int64_t)0xffffffffll) return 0;
  *kchunk = (int)kc;
  return (int)((mpad + kc - 1) / kc);
}

// mode chunks of the size-generic weight-product kernel: whole 32-mode steps, at most 32
static int wgrad_generic_chunks(const Plan& pl, int* kchunk) {
  const int64_t mpad = bwd_mpad(pl);
  const int64_t nk = std::max<int64_t>(1, std::min<int64_t>(32, (mpad + 4095) / 4096));
  const int64_t kc = ((mpad + nk - 1) / nk + 31) / 32 * 32;
  *kchunk = (int)kc;
  return (int)((mpad + kc - 1) / kc);
}

// the weight-product pass's mode chunks (and their length); *slab: the slab kernel runs
static int wgrad_chunks(const Plan& pl, int* kchunk, bool* slab) {
  const int ns = wgrad_slab_chunks(pl, kchunk);
  *slab = ns > 0;
  return ns > 0 ? ns : wgrad_generic_chunks(pl, kchunk);
}

// floats of the backward's fp32 chunk sums: per mode chunk, the weight products
// [2][nb][2 bs][2 bs], then per chunk the bias sums [2][nb][2 bs]
size_t bwd_acc_floats(const Plan& pl) {
  int kc = 0;
  bool slab = false;
  const int nchunk = wgrad_chunks(pl, &kc, &slab);
  const size_t nb2 = 2 * (size_t)pl.bs;
  return (size_t)nchunk * 2 * pl.nb * nb2 * (nb2 + 1);
}

// The W-axis forward transform of x into S (no operand preparation).
template <typename T>
static hipError_t launch_row_forward(const Plan& pl, const T* x, T* S, hipStream_t st) {
  if (pl.path != 1 && fast_row_available(pl.W, pl.C)) {
    PrepJob<T> pj{nullptr, nullptr, nullptr, nullptr, (int)pl.nb, (int)pl.bs, (int)pl.H, 0, 0, -1, 0};
    launch_row_fwd_fast<T>(pl, x, S, pj, st);
  } else {
    dim3 rgrid((unsigned)(pl.B * pl.H), (unsigned)(pl.C / pl.row.rc));
    hipLaunchKernelGGL(row_r2c_kernel<T>, rgrid, dim3(kRowThreads), pl.row_lds, st, x, S, pl.row);
  }
  return hipGetLastError();
}

static void launch_col_bwd_mfma(const Plan& pl, const bf16* Sx, bf16* Sg, const uint4* wfwd,
                                const uint4* wbwd, const uint4* tab, const uint4* tab_lo,
                                const bf16* b1,
                                const bf16* b2, bf16* modes, int64_t mpad, hipStream_t st) {
  const int hp = mfma_col_hp(pl.H);
  const dim3 grid((unsigned)(pl.B * pl.KW * pl.nb));
#define AFNO_CASE(HP_, BS_)                                                                   \
  if (hp == HP_ && pl.bs == BS_) {                                                            \
    hipLaunchKernelGGL((column_bwd_mfma<HP_, BS_>), grid, dim3(512), (MfmaBwd<HP_, BS_>::kBytes), \
                       st, Sx, Sg, wfwd, wbwd, tab, tab_lo, b1, b2, (int)pl.H, (int)pl.C, (int)pl.KW,   \
                       (int)pl.nb, (int)pl.kept_h, pl.col.lam, (int)pl.W, modes, mpad);      \
    return;                                                                                   \
  }
  AFNO_MFMA_COL_LIST(AFNO_CASE)
#undef AFNO_CASE
}

template <typename T>
static hipError_t launch_bwd(const Plan& pl, const BwdPtrs& a, hipStream_t st) {
  const T* x = static_cast<const T*>(a.x);
  const T* g = static_cast<const T*>(a.gout);
  char* ws = static_cast<char*>(a.ws);
  T* Sx = reinterpret_cast<T*>(ws + pl.bwd.sx_offset);
  T* Sg = reinterpret_cast<T*>(ws + pl.bwd.sg_offset);
  T* wt1 = reinterpret_cast<T*>(ws + pl.bwd.wt_offset);
  T* wt2 = wt1 + pl.nb * pl.bs * pl.bs * 2;
  T* modes = reinterpret_cast<T*>(ws + pl.bwd.modes_offset);
  float* acc = reinterpret_cast<float*>(ws + pl.bwd.acc_offset);
  const int nb = (int)pl.nb, bs = (int)pl.bs, nb2 = 2 * bs;
  int kchunk = 0;
  bool slab = false;
  const int nchunk = wgrad_chunks(pl, &kchunk, &slab);
  // the chunk sums of the weight products [nchunk][2][nb][2 bs][2 bs], then of the bias sums
  // [nchunk][2][nb][2 bs]: stored, not accumulated, so nothing is cleared
  float* bsums = acc + (int64_t)nchunk * 2 * nb * nb2 * nb2;
  const int64_t mpad = bwd_mpad(pl);
  const bool mfma = use_mfma_bwd(pl);
  hipError_t e = launch_row_forward<T>(pl, x, Sx, st);
  if (e == hipSuccess) e = launch_row_forward<T>(pl, g, Sg, st);
  if (e != hipSuccess) return e;
  const int64_t nw = (int64_t)2 * nb * bs * bs;
  if (!mfma)
    hipLaunchKernelGGL(conj_transpose_weights<T>, dim3((unsigned)std::min<int64_t>((nw + 255) / 256, 4096)),
                       dim3(256), 0, st, static_cast<const T*>(a.w1), static_cast<const T*>(a.w2),
                       wt1, wt2, nb, bs);
  if constexpr (sizeof(T) == 2) {
    if (mfma) {
      typedef typename FragWord<T>::type Word;
      Word* wfwd = reinterpret_cast<Word*>(ws + pl.bwd.prep_offset);
      Word* wbwd = reinterpret_cast<Word*>(ws + pl.bwd.prep_offset + frag_bytes(pl));
      uint4* tab = reinterpret_cast<uint4*>(ws + pl.bwd.prep_offset + 2 * frag_bytes(pl));
      uint4* tab_lo = reinterpret_cast<uint4*>(ws + pl.bwd.prep_offset + 2 * frag_bytes(pl) +
                                               mfma_tab_bytes(pl));
      const int hp = mfma_col_hp(pl.H);
      const int64_t ntab = (int64_t)mfma_tab_bytes(pl) / 16;
      // the table rounded entry by entry (kept_h -1): tab_lo holds its remainders
      PrepJob<T> pf{static_cast<const T*>(a.w1), static_cast<const T*>(a.w2), wfwd, tab, nb, bs,
                    (int)pl.H, hp, 0, -1, 0};
      PrepJob<T> pb{wt2, wt1, wbwd, nullptr, nb, bs, (int)pl.H, hp, 0, -1, 0};
      // everything that does not read wt1 / wt2 in one launch, then their fragments
      BwdPrep bp{pf, static_cast<const bf16*>(a.w1), static_cast<const bf16*>(a.w2), wt1, wt2,
                 tab_lo, nb, bs, (int)pl.H, hp, prep_words_host(pl, true, -1), ntab, nw};
      const int64_t nall = bp.n_pf + bp.n_lo + bp.n_ct;
      hipLaunchKernelGGL(bwd_prep_kernel, dim3((unsigned)std::min<int64_t>((nall + 255) / 256, 4096)),
                         dim3(256), 0, st, bp);
      const unsigned gb = (unsigned)std::min<int64_t>((prep_words_host(pl, false, -1) + 255) / 256, 4096);
      hipLaunchKernelGGL(prep_operands_kernel<T>, dim3(gb), dim3(256), 0, st, pb);
      launch_col_bwd_mfma(pl, Sx, Sg, reinterpret_cast<const uint4*>(wfwd),
                          reinterpret_cast<const uint4*>(wbwd), tab, tab_lo,
                          static_cast<const T*>(a.b1),
                          static_cast<const T*>(a.b2), modes, mpad, st);
    }
  }
  if (!mfma)
    hipLaunchKernelGGL(column_bwd_kernel<T>, dim3((unsigned)(pl.B * pl.KW * pl.nb)),
                       dim3(pl.col_threads), bwd_lds(pl), st, Sx, Sg, static_cast<const T*>(a.w1),
                       static_cast<const T*>(a.b1), static_cast<const T*>(a.w2),
                       static_cast<const T*>(a.b2), wt1, wt2, pl.col, modes, mpad, (int)pl.W);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // dx = g + C2R(Sg): the W-axis inverse with g as the residual, first, while the gradient
  // spectrum the column pass has just written may still sit in the last-level cache
  T* dx = static_cast<T*>(a.dx);
  if (pl.path != 1 && fast_row_available(pl.W, pl.C))
    launch_row_inv_fast<T>(pl, Sg, g, dx, nullptr, 0, st);
  else {
    dim3 rgrid((unsigned)(pl.B * pl.H), (unsigned)(pl.C / pl.row.rc));
    hipLaunchKernelGGL(row_c2r_kernel<T>, rgrid, dim3(kRowThreads), pl.row_lds, st, Sg, g, dx,
                       nullptr, pl.row, 0);
  }
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // weight and bias gradients over all modes: chunk sums, then their sum in chunk order
  if (slab) {
    const dim3 sgrid((unsigned)(2 * nb * nchunk));
    if (nb2 == 64)
      hipLaunchKernelGGL(wgrad_slab<64>, sgrid, dim3(1024), 512 * 64, st,
                         reinterpret_cast<const bf16*>(modes), mpad, nb, kchunk, acc, bsums);
    else if (nb2 == 128)
      hipLaunchKernelGGL(wgrad_slab<128>, sgrid, dim3(1024), 512 * 128, st,
                         reinterpret_cast<const bf16*>(modes), mpad, nb, kchunk, acc, bsums);
    else
      hipLaunchKernelGGL(wgrad_slab<192>, sgrid, dim3(1024), 512 * 192, st,
                         reinterpret_cast<const bf16*>(modes), mpad, nb, kchunk, acc, bsums);
  } else {
    // 64 x 64 output tiles, chunks of whole 32-mode steps
    const int nt64 = (nb2 + 63) / 64;
    const dim3 wgrid((unsigned)(2 * nb * nt64 * nt64), (unsigned)nchunk);
    hipLaunchKernelGGL(wgrad_kernel<T>, wgrid, dim3(256), 0, st, modes, mpad, nb, bs, kchunk, acc,
                       bsums);
  }
  hipLaunchKernelGGL(wgrad_finalize_parts, dim3((unsigned)std::min<int64_t>((nw + 255) / 256, 4096)),
                     dim3(256), 0, st, acc, nchunk, bsums, nb, bs, a.dw1, a.dw2, a.db1, a.db2);
  return hipGetLastError();
}

hipError_t launch_backward(const Plan& pl, const BwdPtrs& a, hipStream_t st) {
  if (pl.dtype == 0) return launch_bwd<float>(pl, a, st);
  return launch_bwd<bf16>(pl, a, st);
}

// zero weight and bias gradients (a call whose modes are all cut off)
hipError_t launch_zero_grads(const Plan& pl, const BwdPtrs& a, hipStream_t st) {
  const int64_t nw = pl.nb * pl.bs * pl.bs * 2, nbias = pl.nb * pl.bs * 2;
  const unsigned g = (unsigned)std::min<int64_t>((nw + 255) / 256, 4096);
  hipLaunchKernelGGL(fill_zero_f32<float>, dim3(g), dim3(256), 0, st, a.dw1, nw);
  hipLaunchKernelGGL(fill_zero_f32<float>, dim3(g), dim3(256), 0, st, a.dw2, nw);
  hipLaunchKernelGGL(fill_zero_f32<float>, dim3(1), dim3(256), 0, st, a.db1, nbias);
  hipLaunchKernelGGL(fill_zero_f32<float>, dim3(1), dim3(256), 0, st, a.db2, nbias);
  return hipGetLastError();
}

// ------------------------------------------------------------------ AFNO block

hipError_t launch_block(const Plan& pl, const BlockPtrs& a, hipStream_t st) {
  const int64_t M = pl.B * pl.H * pl.W;
  const int C = (int)pl.C, N1 = 4 * C;
  char* ws = a.ws;
  bf16* t = reinterpret_cast<bf16*>(ws + a.t_off);
  bf16* u = reinterpret_cast<bf16*>(ws + a.u_off);
  bf16* v = reinterpret_cast<bf16*>(ws + a.v_off);
  bf16* w = reinterpret_cast<bf16*>(ws + a.w_off);
  bf16* h = reinterpret_cast<bf16*>(ws + a.h_off);
  bf16* wat = reinterpret_cast<bf16*>(ws + a.wat_off);
  bf16* wbt = reinterpret_cast<bf16*>(ws + a.wbt_off);
  const bf16* x = static_cast<const bf16*>(a.x);
  // the MLP weights in the GEMM's [N][K] form
  hipLaunchKernelGGL(transpose_bf16, dim3((unsigned)((N1 + 31) / 32), (unsigned)((C + 31) / 32)),
                     dim3(256), 0, st, static_cast<const bf16*>(a.wa), wat, C, N1);
  hipLaunchKernelGGL(transpose_bf16, dim3((unsigned)((C + 31) / 32), (unsigned)((N1 + 31) / 32)),
                     dim3(256), 0, st, static_cast<const bf16*>(a.wb), wbt, N1, C);
  const unsigned lng = (unsigned)((M + 3) / 4);
  hipLaunchKernelGGL(layer_norm_kernel, dim3(lng), dim3(256), 0, st, x,
                     static_cast<const bf16*>(a.ln1_g), static_cast<const bf16*>(a.ln1_b), t, M, C);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_filter(pl, t, a.w1, a.b1, a.w2, a.b2, ws + a.s_off, u, nullptr, kStageFull, st,
                    nullptr);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(add_layer_norm_kernel, dim3(lng), dim3(256), 0, st, u, x,
                     static_cast<const bf16*>(a.ln2_g), static_cast<const bf16*>(a.ln2_b), v, w, M, C);
  // row tiles of 256, padded to whole XCD rounds; column tiles of 256 (direct-to-LDS kernel)
  // where N allows, else 128 (C a multiple of 128 makes K = C or 4 C a multiple of 128)
  const int64_t mbp = ((M + 255) / 256 + 7) / 8 * 8;
  auto gemm = [&](auto epi, const bf16* Am, const bf16* Bm, const bf16* bias, const bf16* Rm,
                  bf16* Dm, int N, int K) {
    constexpr int E = decltype(epi)::value;
    if (N % 256 == 0 && K % 128 == 0)
      hipLaunchKernelGGL((gemm_dma<E>), dim3((unsigned)(mbp * (N / 256))), dim3(1024), 0, st, Am,
                         Bm, bias, Rm, Dm, (int)M, N, K);
    else
      hipLaunchKernelGGL((gemm_bf16<E, 128>), dim3((unsigned)(mbp * (N / 128))),
                         dim3(GemmGeo<128>::NT), GemmGeo<128>::kBytes, st, Am, Bm, bias, Rm, Dm,
                         (int)M, N, K);
  };
  gemm(std::integral_constant<int, kEpiGelu>(), w, wat, static_cast<const bf16*>(a.ba), nullptr, h,
       N1, C);
  gemm(std::integral_constant<int, kEpiResidual>(), h, wbt, static_cast<const bf16*>(a.bb), v,
       static_cast<bf16*>(a.out), C, N1);
  return hipGetLastError();
}

hipError_t set_kernel_attributes() {
  const int lds_max = kLdsBytes;
  hipError_t e, first = hipSuccess;
#define AFNO_ATTR(K)                                                                         \
  e = hipFuncSetAttribute(reinterpret_cast<const void*>(K),                                \
                          hipFuncAttributeMaxDynamicSharedMemorySize, lds_max);            \
  if (e != hipSuccess && first == hipSuccess) first = e;
  AFNO_ATTR(row_r2c_kernel<float>)
  AFNO_ATTR(row_r2c_kernel<bf16>)
  AFNO_ATTR(row_c2r_kernel<float>)
  AFNO_ATTR(row_c2r_kernel<bf16>)
  AFNO_ATTR(column_kernel<float>)
  AFNO_ATTR(column_kernel<bf16>)
  AFNO_ATTR(column_bwd_kernel<float>)
  AFNO_ATTR(column_bwd_kernel<bf16>)
  AFNO_ATTR((gemm_bf16<kEpiGelu, 128>))
  AFNO_ATTR((gemm_bf16<kEpiResidual, 128>))
  AFNO_ATTR(wgrad_slab<64>)
  AFNO_ATTR(wgrad_slab<128>)
  AFNO_ATTR(wgrad_slab<192>)
#define AFNO_CASE(HP_, BS_) AFNO_ATTR((column_bwd_mfma<HP_, BS_>))
  AFNO_MFMA_COL_LIST(AFNO_CASE)
#undef AFNO_CASE
  AFNO_ATTR((column_fast<float, float, 90, 9, 10, 96, 4, 512>))
  AFNO_ATTR((column_fast<bf16, float, 90, 9, 10, 96, 4, 512>))
  AFNO_ATTR((column_fast<bf16, bf16, 180, 12, 15, 128, 4, 1024>))
  AFNO_ATTR((column_fast<float, float, 180, 12, 15, 32, 6, 512>))
  AFNO_ATTR((column_fast<bf16, float, 180, 12, 15, 32, 6, 512>))
  AFNO_ATTR((column_fast<bf16, bf16, 180, 12, 15, 64, 3, 256>))
#define AFNO_CASE(HP_, BS_) AFNO_ATTR((column_mfma<HP_, BS_>))
  AFNO_MFMA_COL_LIST(AFNO_CASE)
#undef AFNO_CASE
#define AFNO_CASE(HP_, BS_, HS_) AFNO_ATTR((column_mfma_hidden<HP_, BS_, HS_>))
  AFNO_MFMA_HID_LIST(AFNO_CASE)
#undef AFNO_CASE
#define AFNO_CASE(KP_) AFNO_ATTR((column_mfma_kept<96, 96, KP_>))
  AFNO_KEPT_LIST(AFNO_CASE)
#undef AFNO_CASE
#undef AFNO_ATTR
  return first;
}

hipError_t launch_filter(const Plan& pl, const void* x, const void* w1, const void* b1,
                         const void* w2, const void* b2, void* S, void* out, float* dst,
                         int stage, hipStream_t st, hipEvent_t* ev) {
  if (pl.dtype == 0)
    return launch_all<float>(pl, x, w1, b1, w2, b2, S, out, dst, stage, st, ev);
  return launch_all<bf16>(pl, x, w1, b1, w2, b2, S, out, dst, stage, st, ev);
}

}  // namespace afno
