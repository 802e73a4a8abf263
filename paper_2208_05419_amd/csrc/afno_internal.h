// afno_internal.h -- launch plan shared by the C ABI (afno_api.cpp) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "fft_lds.h"

namespace afno {

constexpr int kRowThreads = 256;      // threads of a W-axis workgroup
constexpr int kRowEmax = 32;          // complex values a thread holds in a W pass
constexpr int kRowLdsMax = 160 * 1024; // LDS budget of a W-axis workgroup
constexpr int kColEmax = 24;          // complex values a thread holds in an H pass
constexpr int kColMaxMTiles = 12;     // 16-row MFMA tiles per column: H <= 192
constexpr int kColMaxThreads = 512;   // 8 waves: bs <= 128
constexpr int kLdsBytes = 160 * 1024; // LDS of one gfx950 CU

// profile events per timed call: before the first kernel and after each of the four
// phases (operand preparation, W forward, column, W inverse)
constexpr int kProfEvents = 5;

constexpr int kStageFull = 0;
constexpr int kStageSpectrum = 1;
constexpr int kStageMixed = 2;
constexpr int kStageDelta = 3;

struct RowParams {
  int W, C, KW, rc;   // rc channels (rc/2 complex signals) per workgroup
  float inv_sqrt_w;
  Radices rw;
};

struct ColParams {
  int H, H16, bs, nb, C, KW;
  int hs;             // hidden units per block (hs = bs: the hidden layer reuses the tile)
  int ldt;            // LDS row stride of the column tile, elements
  int ldh;            // LDS row stride of the hidden tile (hs != bs), elements
  int htile_bytes;    // the hidden tile (0 when hs = bs)
  int chk;            // channels per pass of the H transform
  int kept_h;
  int tile_bytes;
  float lam, inv_sqrt_h;
  Radices rh;
};

struct Plan {
  int64_t B, H, W, C, nb, bs;
  int dtype;          // 0 fp32, 1 bf16
  int path;           // kernel path (set_kernel_path) when the plan was made
  int64_t KW;         // kept_w: W columns that carry kept modes
  int64_t kept_h;
  RowParams row;
  ColParams col;
  size_t row_lds, col_lds;
  int col_threads;
  size_t spec_bytes;  // spectrum: B * H * KW * C complex values
  size_t frag_offset; // fragment-ordered weights (size-specialised column kernels), after S
  size_t tab_offset;  // transform table (MFMA-transform column kernel), after the weights
  size_t ws_bytes;    // whole workspace
  struct {            // backward-pass workspace offsets (afno_filter_backward)
    size_t sx_offset, sg_offset, wt_offset, prep_offset, modes_offset, acc_offset, bytes;
  } bwd;
};

// pointers of one backward call (dw*, db* float32)
struct BwdPtrs {
  const void *x, *w1, *b1, *w2, *b2, *gout;
  void* dx;
  float *dw1, *db1, *dw2, *db2;
  void* ws;
};

// pointers of one AFNO-block call (all bf16) and its workspace offsets
struct BlockPtrs {
  const void *x, *ln1_g, *ln1_b, *w1, *b1, *w2, *b2, *ln2_g, *ln2_b, *wa, *ba, *wb, *bb;
  void* out;
  char* ws;
  size_t t_off, u_off, v_off, w_off, h_off, wat_off, wbt_off, s_off;
};

hipError_t set_kernel_attributes();
// 0: specialised kernels where available, 1: generic only, 2: as 0 without the
// MFMA-transform column kernel
void set_kernel_path(int path);
int kernel_path();
bool fast_row_available(int64_t W, int64_t C);
bool fast_col_available(int dtype, int64_t H, int64_t bs);
bool mfma_col_available(int dtype, int64_t H, int64_t bs);
bool use_mfma_col(const Plan& pl);  // under the current kernel path
bool use_fast_col(const Plan& pl);  // under the current kernel path
bool use_mfma_hidden(const Plan& pl);  // matrix-core column kernel for hidden = 2 bs
size_t hidden_frag_bytes(const Plan& pl);
size_t frag_bytes(const Plan& pl);
size_t mfma_tab_bytes(const Plan& pl);
size_t fwd_tab_bytes(const Plan& pl);   // the forward's tables (kept-row kernel included)
// ev: NULL, or kProfEvents events recorded before the first kernel and after each phase
// backward pass: modes per block of the per-mode factor tensors, and the column kernel's LDS
int64_t bwd_mpad(const Plan& pl);
size_t bwd_lds(const Plan& pl);
size_t bwd_prep_bytes(const Plan& pl);  // prepared operands of the matrix-core backward
size_t bwd_acc_floats(const Plan& pl);  // fp32 sums of the weight and bias gradients
int wgrad_slab_chunks(const Plan& pl, int* kchunk);
hipError_t launch_backward(const Plan& pl, const BwdPtrs& a, hipStream_t st);
hipError_t launch_zero_grads(const Plan& pl, const BwdPtrs& a, hipStream_t st);
// one AFNO block (LayerNorm, filter, LayerNorm, channel MLP, residuals); pl: the filter's
// plan for the block's shape
hipError_t launch_block(const Plan& pl, const BlockPtrs& a, hipStream_t st);
hipError_t launch_filter(const Plan& pl, const void* x, const void* w1, const void* b1,
                         const void* w2, const void* b2, void* S, void* out, float* dst,
                         int stage, hipStream_t st, hipEvent_t* ev);

}  // namespace afno
