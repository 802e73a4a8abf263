// afno_api.cpp -- the C ABI declared in include/afno.h: argument validation, the launch
// plan (transform factorisation, cutoff counts, LDS budgets) and the stream-ordered
// spectrum workspace.  Every step of the filter runs in the kernels of afno_kernels.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "afno.h"
#include "afno_internal.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}

// n = 4^a 2^b 3^c 5^d -> one pass per factor; false if another prime divides n.
bool factorize(int64_t n, afno::Radices& r) {
  r.n = (int)n;
  r.count = 0;
  const int order[4] = {4, 2, 3, 5};
  for (int f : order) {
    while (n % f == 0 && (f != 2 || n % 4 != 0)) {
      if (r.count >= afno::kMaxPasses) return false;
      r.r[r.count++] = f;
      n /= f;
    }
  }
  return n == 1;
}

// every pass of `r` fits the per-thread register budget with nsub butterfly slots
bool passes_fit(const afno::Radices& r, int nsub, int emax) {
  for (int p = 0; p < r.count; ++p) {
    const int R = r.r[p];
    const int per_thread = (r.n / R + nsub - 1) / nsub;
    if (per_thread > (emax + R - 1) / R) return false;
  }
  return true;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

struct Args {
  const void *x, *w1, *b1, *w2, *b2;
  int64_t B, H, W, C, nb;
  float lam, keep;
  int dtype;
  void* out;
  size_t out_bytes;  // 0: the size of x
  int64_t hs;        // hidden units per block; 0: the block size
};

// Validation (no HIP call) and plan construction.  Returns AFNO_OK, or an error code
// with g_last_error set.
int make_plan(const Args& a, afno::Plan& pl) {
  pl.path = afno::kernel_path();
  if (a.dtype != AFNO_DTYPE_FP32 && a.dtype != AFNO_DTYPE_BF16)
    return fail(AFNO_ERR_INVALID_ARG, "dtype must be AFNO_DTYPE_FP32 (0) or AFNO_DTYPE_BF16 (1)");
  if (a.B < 0 || a.H <= 0 || a.W <= 0 || a.C <= 0 || a.nb <= 0)
    return fail(AFNO_ERR_INVALID_ARG, "B must be >= 0 and H, W, C, num_blocks > 0");
  if (a.C % a.nb != 0)
    return fail(AFNO_ERR_INVALID_ARG, "C must be a multiple of num_blocks");
  if (!std::isfinite(a.lam) || a.lam < 0.f)
    return fail(AFNO_ERR_INVALID_ARG, "lambda must be finite and >= 0");
  if (!(a.keep > 0.f && a.keep <= 1.f))
    return fail(AFNO_ERR_INVALID_ARG, "keep_fraction must be in (0, 1]");

  pl.B = a.B; pl.H = a.H; pl.W = a.W; pl.C = a.C; pl.nb = a.nb;
  pl.bs = a.C / a.nb;
  const int64_t hs = a.hs ? a.hs : pl.bs;
  if (hs <= 0) return fail(AFNO_ERR_INVALID_ARG, "hidden must be > 0");
  pl.dtype = a.dtype;
  // hard mode cutoff, products in double
  const int64_t Kh = a.H / 2 + 1, Wm = a.W / 2 + 1;
  pl.kept_h = (int64_t)std::floor((double)Kh * (double)a.keep);
  pl.KW = (int64_t)std::floor((double)Wm * (double)a.keep);
  if (pl.kept_h == 0) pl.KW = 0;  // no row passes: no mode is kept
  if (a.B == 0) return AFNO_OK;

  if (!a.x || !a.w1 || !a.b1 || !a.w2 || !a.b2 || !a.out)
    return fail(AFNO_ERR_INVALID_ARG, "null pointer argument");

  const size_t es = a.dtype == AFNO_DTYPE_FP32 ? 4 : 2;
  if (!aligned(a.x, 16) || !aligned(a.out, 16))
    return fail(AFNO_ERR_UNSUPPORTED, "x and out must be 16-byte aligned");
  if (!aligned(a.w1, 4) || !aligned(a.b1, 4) || !aligned(a.w2, 4) || !aligned(a.b2, 4))
    return fail(AFNO_ERR_UNSUPPORTED, "weights and biases must be 4-byte aligned");
  if (a.W % 2 != 0) return fail(AFNO_ERR_UNSUPPORTED, "W must be even");
  if (!factorize(a.W, pl.row.rw) || !factorize(a.H, pl.col.rh))
    return fail(AFNO_ERR_UNSUPPORTED, "H and W must be of the form 2^a 3^b 5^c");
  if (pl.bs % 16 != 0 || pl.bs > 128)
    return fail(AFNO_ERR_UNSUPPORTED, "block size C/num_blocks must be a multiple of 16 and <= 128");
  if (hs % 16 != 0 || hs > 256)
    return fail(AFNO_ERR_UNSUPPORTED, "hidden size must be a multiple of 16 and <= 256");
  if (a.W > 1024) return fail(AFNO_ERR_UNSUPPORTED, "W must be <= 1024");
  if (a.H > 16 * afno::kColMaxMTiles)
    return fail(AFNO_ERR_UNSUPPORTED, "H must be <= 192");
  const double elems = (double)a.B * a.H * a.W * a.C;
  if (elems > 4.0e15 || (double)a.B * a.H * (a.C / 16) > 2.0e9 || (double)a.B * Wm * a.nb > 2.0e9)
    return fail(AFNO_ERR_UNSUPPORTED, "tensor too large");
  // the kernels address one column of the spectrum (H rows of kept_w * C complex values) and
  // one row of the grid (W * C values, float32 for the diagnostic stage output) through
  // 32-bit byte offsets from a per-workgroup base
  {
    const double col_span = (double)a.H * (double)pl.KW * (double)a.C * 2.0 * (double)es;
    const double row_span = (double)a.W * (double)a.C * 4.0;
    if (col_span > 4294967295.0 || row_span > 4294967295.0)
      return fail(AFNO_ERR_UNSUPPORTED,
                  "a spectrum column (H * kept_w * C complex values) or a grid row (W * C "
                  "values) spans more than 4 GiB");
  }

  // W-axis workgroups: rc channels, rc/2 complex signals
  pl.row.W = (int)a.W; pl.row.C = (int)a.C; pl.row.KW = (int)pl.KW;
  pl.row.inv_sqrt_w = (float)(1.0 / std::sqrt((double)a.W));
  pl.row.rc = 0;
  for (int rc : {64, 32, 16}) {
    if (a.C % rc != 0) continue;
    const int np = rc / 2;
    const size_t lds = (size_t)a.W * np * 8 + (size_t)a.W * 8;
    if (lds > (size_t)afno::kRowLdsMax) continue;
    if (!passes_fit(pl.row.rw, afno::kRowThreads / np, afno::kRowEmax)) continue;
    pl.row.rc = rc;
    pl.row_lds = lds;
    break;
  }
  if (pl.row.rc == 0) return fail(AFNO_ERR_UNSUPPORTED, "W too large for the W-axis kernel");

  // column workgroups
  afno::ColParams& c = pl.col;
  c.H = (int)a.H; c.H16 = (int)((a.H + 15) / 16 * 16); c.bs = (int)pl.bs; c.nb = (int)a.nb;
  c.C = (int)a.C; c.KW = (int)pl.KW; c.kept_h = (int)pl.kept_h;
  c.lam = a.lam;
  c.inv_sqrt_h = (float)(1.0 / std::sqrt((double)a.H));
  c.hs = (int)hs;
  c.ldt = 2 * c.bs + (a.dtype == AFNO_DTYPE_BF16 ? 8 : 4);
  c.ldh = 2 * c.hs + (a.dtype == AFNO_DTYPE_BF16 ? 8 : 4);
  c.chk = (c.bs % 32 == 0) ? 32 : 16;  // must divide bs
  {  // waves: one per 32 real output columns of the wider layer, 4 to 8
    const int64_t wmax = std::max<int64_t>(c.bs, c.hs) / 16;
    pl.col_threads = 64 * (int)std::min<int64_t>(8, std::max<int64_t>(4, wmax));
  }
  c.tile_bytes = (int)(((size_t)c.H16 * c.ldt * es + 15) / 16 * 16);
  c.htile_bytes = c.hs == c.bs ? 0 : (int)(((size_t)c.H16 * c.ldh * es + 15) / 16 * 16);
  pl.col_lds = (size_t)c.tile_bytes + (size_t)c.htile_bytes + (size_t)a.H * c.chk * 8 +
               (size_t)a.H * 8;
  if (pl.col_lds > (size_t)afno::kLdsBytes)
    return fail(AFNO_ERR_UNSUPPORTED, "column tile (H x block size) does not fit in LDS");
  if (!passes_fit(c.rh, pl.col_threads / c.chk, afno::kColEmax))
    return fail(AFNO_ERR_UNSUPPORTED, "H transform exceeds the per-thread register budget");

  pl.spec_bytes = (size_t)a.B * a.H * pl.KW * a.C * 2 * es;
  pl.frag_offset = (pl.spec_bytes + 255) / 256 * 256;
  const bool mfma = afno::use_mfma_col(pl);
  const bool hid = afno::use_mfma_hidden(pl);
  const size_t fb = hid ? afno::hidden_frag_bytes(pl)
                        : ((mfma || afno::use_fast_col(pl)) ? afno::frag_bytes(pl) : 0);
  pl.tab_offset = (pl.frag_offset + fb + 255) / 256 * 256;
  pl.ws_bytes = (mfma || hid) ? pl.tab_offset + afno::fwd_tab_bytes(pl) : pl.frag_offset + fb;

  // out must not overlap any input
  const size_t xb = (size_t)a.B * a.H * a.W * a.C * es;
  const size_t ob = a.out_bytes ? a.out_bytes : xb;
  const size_t wb = (size_t)a.nb * pl.bs * hs * 2 * es, bb = (size_t)a.nb * pl.bs * 2 * es;
  const size_t hb = (size_t)a.nb * hs * 2 * es;
  if (overlaps(a.out, ob, a.x, xb) || overlaps(a.out, ob, a.w1, wb) ||
      overlaps(a.out, ob, a.w2, wb) || overlaps(a.out, ob, a.b1, hb) ||
      overlaps(a.out, ob, a.b2, bb))
    return fail(AFNO_ERR_ALIAS, "out overlaps an input");
  return AFNO_OK;
}

std::once_flag g_attr_once;

// The workspace of afno_filter_forward_noalloc: a file-scope device array, one copy on every
// GPU the library runs on, held until the process ends.  Its name in host code is only a
// handle: scratch_address() resolves the current device's copy once and host code passes that
// address on, never the name.
constexpr size_t kScratchBytes = (size_t)AFNO_NOALLOC_MAX_WORKSPACE;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of scratch (hipGetSymbolAddress on the first call per device).
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(AFNO_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  }
  if (dev < 0 || dev >= kMaxDevices)
    return fail(AFNO_ERR_UNSUPPORTED, "device index beyond the library's table of devices");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return fail(AFNO_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return AFNO_OK;
}

// Per-call workspaces come from a stream-ordered memory pool of the library's own, one per
// device, that keeps freed memory for the next call instead of returning it to the device
// (release threshold: unbounded), so that a call's allocation and free cost only the pool's
// bookkeeping (measured: the 90 x 180 x 768 bf16 call takes 2.5 us less than from the
// device's default pool).  The pool holds the largest workspaces in use at once until the
// process ends.
std::mutex g_pool_mu;
hipMemPool_t g_pool[kMaxDevices] = {};

hipError_t ws_alloc(void** p, size_t bytes, hipStream_t stream) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipMallocAsync(p, bytes, stream);
  hipMemPool_t pool = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_pool_mu);
    if (!g_pool[dev]) {
      hipMemPoolProps props = {};
      props.allocType = hipMemAllocationTypePinned;
      props.location.type = hipMemLocationTypeDevice;
      props.location.id = dev;
      e = hipMemPoolCreate(&pool, &props);
      if (e != hipSuccess) return e;
      uint64_t keep = UINT64_MAX;
      e = hipMemPoolSetAttribute(pool, hipMemPoolAttrReleaseThreshold, &keep);
      if (e != hipSuccess) {
        (void)hipMemPoolDestroy(pool);
        return e;
      }
      g_pool[dev] = pool;
    }
    pool = g_pool[dev];
  }
  return hipMallocFromPoolAsync(p, bytes, pool, stream);
}

// diagnostic per-kernel timing (afno_profile_begin / afno_profile_end)
struct Profile {
  std::mutex mu;
  bool on = false;
  int cap = 0, used = 0;
  std::vector<hipEvent_t> ev;  // afno::kProfEvents per timed call
};
Profile g_prof;

hipEvent_t* profile_slot() {
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on || g_prof.used >= g_prof.cap) return nullptr;
  return &g_prof.ev[afno::kProfEvents * (size_t)g_prof.used++];
}

// noalloc: the workspace is the current device's scratch array (no allocation); a plan
// whose workspace exceeds it is rejected before any HIP call.
int run(const Args& a, int stage, float* dst, hipStream_t stream, bool noalloc = false) {
  afno::Plan pl;
  int rc = make_plan(a, pl);
  if (rc != AFNO_OK || a.B == 0) return rc;
  if (noalloc && pl.KW > 0 && pl.ws_bytes > kScratchBytes)
    return fail(AFNO_ERR_UNSUPPORTED, "the workspace of " + std::to_string(pl.ws_bytes) +
                                          " bytes exceeds the " + std::to_string(kScratchBytes) +
                                          " bytes of afno_filter_forward_noalloc");

  std::call_once(g_attr_once, [] {
    (void)afno::set_kernel_attributes();
    (void)hipGetLastError();
  });

  const size_t xb = (size_t)a.B * a.H * a.W * a.C * (a.dtype == AFNO_DTYPE_FP32 ? 4 : 2);
  hipError_t e;
  if (pl.KW == 0) {  // nothing kept: the filter is zero
    if (stage == afno::kStageFull)
      e = hipMemcpyAsync(a.out, a.x, xb, hipMemcpyDeviceToDevice, stream);
    else {
      const size_t n = stage == afno::kStageDelta ? (size_t)a.B * a.H * a.W * a.C
                                                  : (size_t)a.B * a.H * (a.W / 2 + 1) * a.C * 2;
      e = hipMemsetAsync(dst, 0, n * sizeof(float), stream);
    }
    if (e != hipSuccess) return fail(AFNO_ERR_HIP, std::string("copy: ") + hipGetErrorString(e));
    return AFNO_OK;
  }

  void* S = nullptr;
  if (noalloc) {
    rc = scratch_address(&S);
    if (rc != AFNO_OK) return rc;
    hipEvent_t* ev = stage == afno::kStageFull ? profile_slot() : nullptr;
    e = afno::launch_filter(pl, a.x, a.w1, a.b1, a.w2, a.b2, S, a.out, dst, stage, stream, ev);
    if (e != hipSuccess) return fail(AFNO_ERR_HIP, std::string("launch: ") + hipGetErrorString(e));
    return AFNO_OK;
  }
  e = ws_alloc(&S, pl.ws_bytes, stream);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(AFNO_ERR_HIP, std::string("workspace allocation of ") +
                                  std::to_string(pl.ws_bytes) + " bytes: " + hipGetErrorString(e));
  }
  hipEvent_t* ev = stage == afno::kStageFull ? profile_slot() : nullptr;
  e = afno::launch_filter(pl, a.x, a.w1, a.b1, a.w2, a.b2, S, a.out, dst, stage, stream, ev);
  hipError_t ef = hipFreeAsync(S, stream);
  if (e != hipSuccess) return fail(AFNO_ERR_HIP, std::string("launch: ") + hipGetErrorString(e));
  if (ef != hipSuccess) return fail(AFNO_ERR_HIP, std::string("workspace free: ") + hipGetErrorString(ef));
  return AFNO_OK;
}

// the backward pass: validation beyond the forward's, workspace layout, launches
int run_backward(const Args& a, const void* gout, float* dw1, float* db1, float* dw2, float* db2,
                 hipStream_t stream) {
  afno::Plan pl;
  int rc = make_plan(a, pl);
  if (rc != AFNO_OK) return rc;
  if (a.B > 0 && !gout) return fail(AFNO_ERR_INVALID_ARG, "null pointer argument");
  if (!dw1 || !db1 || !dw2 || !db2) return fail(AFNO_ERR_INVALID_ARG, "null pointer argument");
  const size_t es = a.dtype == AFNO_DTYPE_FP32 ? 4 : 2;
  const size_t xb = (size_t)a.B * a.H * a.W * a.C * es;
  if (a.B > 0 && !aligned(gout, 16)) return fail(AFNO_ERR_UNSUPPORTED, "gout must be 16-byte aligned");
  if (!aligned(dw1, 4) || !aligned(db1, 4) || !aligned(dw2, 4) || !aligned(db2, 4))
    return fail(AFNO_ERR_UNSUPPORTED, "weight and bias gradients must be 4-byte aligned");
  const size_t wgb = (size_t)a.nb * pl.bs * pl.bs * 2 * 4, bgb = (size_t)a.nb * pl.bs * 2 * 4;
  const size_t wb = (size_t)a.nb * pl.bs * pl.bs * 2 * es, bb = (size_t)a.nb * pl.bs * 2 * es;
  struct R { const void* p; size_t n; };
  const R ins[] = {{a.x, xb}, {gout, xb}, {a.w1, wb}, {a.b1, bb}, {a.w2, wb}, {a.b2, bb}};
  const R outs[] = {{a.out, xb}, {dw1, wgb}, {db1, bgb}, {dw2, wgb}, {db2, bgb}};
  for (const R& o : outs) {
    if (!o.p || o.n == 0) continue;
    for (const R& i : ins)
      if (i.p && i.n && overlaps(o.p, o.n, i.p, i.n))
        return fail(AFNO_ERR_ALIAS, "an output overlaps an input");
    for (const R& q : outs)
      if (&q != &o && q.p && q.n && overlaps(o.p, o.n, q.p, q.n))
        return fail(AFNO_ERR_ALIAS, "two outputs overlap");
  }
  if (a.B > 0 && afno::bwd_lds(pl) > (size_t)afno::kLdsBytes)
    return fail(AFNO_ERR_UNSUPPORTED, "backward column tile (H x block size) does not fit in LDS");

  std::call_once(g_attr_once, [] {
    (void)afno::set_kernel_attributes();
    (void)hipGetLastError();
  });
  afno::BwdPtrs bp{a.x, a.w1, a.b1, a.w2, a.b2, gout, a.out, dw1, db1, dw2, db2, nullptr};
  hipError_t e;
  if (a.B == 0 || pl.KW == 0) {  // no mode passes the filter: dx = g, zero gradients
    e = afno::launch_zero_grads(pl, bp, stream);
    if (e == hipSuccess && a.B > 0) e = hipMemcpyAsync(a.out, gout, xb, hipMemcpyDeviceToDevice, stream);
    if (e != hipSuccess) return fail(AFNO_ERR_HIP, std::string("launch: ") + hipGetErrorString(e));
    return AFNO_OK;
  }
  // workspace: Sx, Sg, conjugate-transposed weights, the matrix-core kernel's prepared
  // operands, per-mode factors, fp32 product and bias sums
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  pl.bwd.sx_offset = 0;
  pl.bwd.sg_offset = up(pl.spec_bytes);
  pl.bwd.wt_offset = pl.bwd.sg_offset + up(pl.spec_bytes);
  pl.bwd.prep_offset = pl.bwd.wt_offset + up(2 * wb);
  pl.bwd.modes_offset = pl.bwd.prep_offset + up(afno::bwd_prep_bytes(pl));
  const size_t modes_bytes = (size_t)4 * a.nb * 2 * pl.bs * (size_t)afno::bwd_mpad(pl) * es;
  pl.bwd.acc_offset = pl.bwd.modes_offset + up(modes_bytes);
  pl.bwd.bytes = pl.bwd.acc_offset + afno::bwd_acc_floats(pl) * 4;
  void* ws = nullptr;
  e = ws_alloc(&ws, pl.bwd.bytes, stream);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(AFNO_ERR_HIP, std::string("workspace allocation of ") + std::to_string(pl.bwd.bytes) +
                                  " bytes: " + hipGetErrorString(e));
  }
  bp.ws = ws;
  e = afno::launch_backward(pl, bp, stream);
  hipError_t ef = hipFreeAsync(ws, stream);
  if (e != hipSuccess) return fail(AFNO_ERR_HIP, std::string("launch: ") + hipGetErrorString(e));
  if (ef != hipSuccess) return fail(AFNO_ERR_HIP, std::string("workspace free: ") + hipGetErrorString(ef));
  return AFNO_OK;
}

// One AFNO block: validation, the filter's plan for the block's shape, one workspace.
int run_block(const Args& a, const void* ln1_g, const void* ln1_b, const void* ln2_g,
              const void* ln2_b, const void* wa, const void* ba, const void* wb, const void* bb,
              hipStream_t stream) {
  if (a.dtype != AFNO_DTYPE_BF16 && a.dtype != AFNO_DTYPE_FP32)
    return fail(AFNO_ERR_INVALID_ARG, "dtype must be AFNO_DTYPE_FP32 (0) or AFNO_DTYPE_BF16 (1)");
  afno::Plan pl;
  int rc = make_plan(a, pl);
  if (rc != AFNO_OK) return rc;
  if (a.dtype != AFNO_DTYPE_BF16)
    return fail(AFNO_ERR_UNSUPPORTED, "the AFNO block runs in bf16 storage only");
  if (a.C % 128 != 0 || a.C > 2048)
    return fail(AFNO_ERR_UNSUPPORTED, "the AFNO block needs C a multiple of 128 and <= 2048");
  if (a.B == 0) return AFNO_OK;
  const void* vecs[] = {ln1_g, ln1_b, ln2_g, ln2_b};
  for (const void* p : vecs)
    if (!p) return fail(AFNO_ERR_INVALID_ARG, "null pointer argument");
  if (!wa || !ba || !wb || !bb) return fail(AFNO_ERR_INVALID_ARG, "null pointer argument");
  for (const void* p : vecs)
    if (!aligned(p, 16)) return fail(AFNO_ERR_UNSUPPORTED, "LayerNorm weights must be 16-byte aligned");
  if (!aligned(wa, 2) || !aligned(ba, 2) || !aligned(wb, 2) || !aligned(bb, 2))
    return fail(AFNO_ERR_UNSUPPORTED, "MLP weights must be 2-byte aligned");
  const size_t xb = (size_t)a.B * a.H * a.W * a.C * 2;
  const size_t cb = (size_t)a.C * 2, mb = (size_t)a.C * 4 * a.C * 2;
  struct R { const void* p; size_t n; };
  const R ins[] = {{ln1_g, cb}, {ln1_b, cb}, {ln2_g, cb}, {ln2_b, cb}, {wa, mb}, {ba, 4 * cb},
                   {wb, mb}, {bb, cb}};
  for (const R& i : ins)
    if (overlaps(a.out, xb, i.p, i.n)) return fail(AFNO_ERR_ALIAS, "out overlaps an input");

  std::call_once(g_attr_once, [] {
    (void)afno::set_kernel_attributes();
    (void)hipGetLastError();
  });
  auto up = [](size_t v) { return (v + 255) / 256 * 256; };
  const size_t M = (size_t)a.B * a.H * a.W;
  afno::BlockPtrs bp{a.x, ln1_g, ln1_b, a.w1, a.b1, a.w2, a.b2, ln2_g, ln2_b, wa, ba, wb, bb,
                     a.out, nullptr, 0, 0, 0, 0, 0, 0, 0, 0};
  bp.t_off = 0;
  bp.u_off = up(xb);
  bp.v_off = bp.u_off + up(xb);
  bp.w_off = bp.v_off + up(xb);
  bp.h_off = bp.w_off + up(xb);
  bp.wat_off = bp.h_off + up(M * 4 * a.C * 2);
  bp.wbt_off = bp.wat_off + up(mb);
  bp.s_off = bp.wbt_off + up(mb);
  const size_t bytes = bp.s_off + pl.ws_bytes;
  void* ws = nullptr;
  hipError_t e = ws_alloc(&ws, bytes, stream);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return fail(AFNO_ERR_HIP, std::string("workspace allocation of ") + std::to_string(bytes) +
                                  " bytes: " + hipGetErrorString(e));
  }
  bp.ws = static_cast<char*>(ws);
  e = afno::launch_block(pl, bp, stream);
  hipError_t ef = hipFreeAsync(ws, stream);
  if (e != hipSuccess) return fail(AFNO_ERR_HIP, std::string("launch: ") + hipGetErrorString(e));
  if (ef != hipSuccess) return fail(AFNO_ERR_HIP, std::string("workspace free: ") + hipGetErrorString(ef));
  return AFNO_OK;
}

}  // namespace

extern "C" {

int afno_filter_forward(const void* x, const void* w1, const void* b1, const void* w2,
                        const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                        int64_t num_blocks, float lambda, float keep_fraction, int dtype,
                        void* out, hipStream_t stream) {
  g_last_error.clear();
  Args a{x, w1, b1, w2, b2, B, H, W, C, num_blocks, lambda, keep_fraction, dtype, out, 0};
  return run(a, afno::kStageFull, nullptr, stream);
}

int afno_filter_forward_noalloc(const void* x, const void* w1, const void* b1, const void* w2,
                                const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                                int64_t num_blocks, float lambda, float keep_fraction, int dtype,
                                void* out, hipStream_t stream) {
  g_last_error.clear();
  Args a{x, w1, b1, w2, b2, B, H, W, C, num_blocks, lambda, keep_fraction, dtype, out, 0};
  return run(a, afno::kStageFull, nullptr, stream, true);
}

int afno_filter_forward_hidden(const void* x, const void* w1, const void* b1, const void* w2,
                               const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                               int64_t num_blocks, int64_t hidden, float lambda,
                               float keep_fraction, int dtype, void* out, hipStream_t stream) {
  g_last_error.clear();
  if (hidden <= 0) return fail(AFNO_ERR_INVALID_ARG, "hidden must be > 0");
  Args a{x, w1, b1, w2, b2, B, H, W, C, num_blocks, lambda, keep_fraction, dtype, out, 0, hidden};
  return run(a, afno::kStageFull, nullptr, stream);
}

int afno_block_forward(const void* x, const void* ln1_g, const void* ln1_b, const void* w1,
                       const void* b1, const void* w2, const void* b2, const void* ln2_g,
                       const void* ln2_b, const void* wa, const void* ba, const void* wb,
                       const void* bb, int64_t B, int64_t H, int64_t W, int64_t C,
                       int64_t num_blocks, float lambda, float keep_fraction, int dtype,
                       void* out, hipStream_t stream) {
  g_last_error.clear();
  Args a{x, w1, b1, w2, b2, B, H, W, C, num_blocks, lambda, keep_fraction, dtype, out, 0, 0};
  return run_block(a, ln1_g, ln1_b, ln2_g, ln2_b, wa, ba, wb, bb, stream);
}

int afno_filter_stage(const void* x, const void* w1, const void* b1, const void* w2,
                      const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                      int64_t num_blocks, float lambda, float keep_fraction, int dtype, int stage,
                      float* dst, hipStream_t stream) {
  g_last_error.clear();
  if (stage != AFNO_STAGE_SPECTRUM && stage != AFNO_STAGE_MIXED && stage != AFNO_STAGE_DELTA)
    return fail(AFNO_ERR_INVALID_ARG, "stage must be AFNO_STAGE_SPECTRUM, _MIXED or _DELTA");
  if (B > 0 && dst && !aligned(dst, 16))
    return fail(AFNO_ERR_UNSUPPORTED, "dst must be 16-byte aligned");
  // dst plays the part of out: it must not overlap an input either
  const size_t nd = stage == AFNO_STAGE_DELTA ? (size_t)B * H * W * C
                                              : (size_t)B * H * (W / 2 + 1) * C * 2;
  Args a{x, w1, b1, w2, b2, B, H, W, C, num_blocks, lambda, keep_fraction, dtype, dst,
         B > 0 && H > 0 && W > 0 && C > 0 ? nd * sizeof(float) : 0};
  return run(a, stage, dst, stream);
}

int afno_filter_stage_hidden(const void* x, const void* w1, const void* b1, const void* w2,
                             const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                             int64_t num_blocks, int64_t hidden, float lambda,
                             float keep_fraction, int dtype, int stage, float* dst,
                             hipStream_t stream) {
  g_last_error.clear();
  if (hidden <= 0) return fail(AFNO_ERR_INVALID_ARG, "hidden must be > 0");
  if (stage != AFNO_STAGE_SPECTRUM && stage != AFNO_STAGE_MIXED && stage != AFNO_STAGE_DELTA)
    return fail(AFNO_ERR_INVALID_ARG, "stage must be AFNO_STAGE_SPECTRUM, _MIXED or _DELTA");
  if (B > 0 && dst && !aligned(dst, 16))
    return fail(AFNO_ERR_UNSUPPORTED, "dst must be 16-byte aligned");
  const size_t nd = stage == AFNO_STAGE_DELTA ? (size_t)B * H * W * C
                                              : (size_t)B * H * (W / 2 + 1) * C * 2;
  Args a{x, w1, b1, w2, b2, B, H, W, C, num_blocks, lambda, keep_fraction, dtype, dst,
         B > 0 && H > 0 && W > 0 && C > 0 ? nd * sizeof(float) : 0, hidden};
  return run(a, stage, dst, stream);
}

int afno_filter_backward(const void* x, const void* w1, const void* b1, const void* w2,
                         const void* b2, const void* gout, int64_t B, int64_t H, int64_t W,
                         int64_t C, int64_t num_blocks, float lambda, float keep_fraction,
                         int dtype, void* dx, float* dw1, float* db1, float* dw2, float* db2,
                         hipStream_t stream) {
  g_last_error.clear();
  Args a{x, w1, b1, w2, b2, B, H, W, C, num_blocks, lambda, keep_fraction, dtype, dx, 0};
  return run_backward(a, gout, dw1, db1, dw2, db2, stream);
}

int afno_profile_begin(int max_calls) {
  g_last_error.clear();
  if (max_calls <= 0) return fail(AFNO_ERR_INVALID_ARG, "max_calls must be > 0");
  std::lock_guard<std::mutex> lk(g_prof.mu);
  for (hipEvent_t e : g_prof.ev) (void)hipEventDestroy(e);
  g_prof.ev.assign(afno::kProfEvents * (size_t)max_calls, nullptr);
  for (hipEvent_t& e : g_prof.ev) {
    hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) {
      for (hipEvent_t f : g_prof.ev)
        if (f) (void)hipEventDestroy(f);
      g_prof.ev.clear();
      g_prof.on = false;
      return fail(AFNO_ERR_HIP, std::string("hipEventCreate: ") + hipGetErrorString(r));
    }
  }
  g_prof.cap = max_calls;
  g_prof.used = 0;
  g_prof.on = true;
  return AFNO_OK;
}

int afno_profile_end(double* kernel_ms, int64_t* calls) {
  g_last_error.clear();
  if (!kernel_ms || !calls) return fail(AFNO_ERR_INVALID_ARG, "null output pointer");
  std::lock_guard<std::mutex> lk(g_prof.mu);
  if (!g_prof.on) return fail(AFNO_ERR_INVALID_ARG, "afno_profile_end without afno_profile_begin");
  int rc = AFNO_OK;
  double sum[afno::kProfEvents - 1] = {0.0, 0.0, 0.0, 0.0};
  for (int c = 0; c < g_prof.used && rc == AFNO_OK; ++c) {
    hipEvent_t* ev = &g_prof.ev[afno::kProfEvents * (size_t)c];
    hipError_t r = hipEventSynchronize(ev[afno::kProfEvents - 1]);
    for (int k = 0; k < afno::kProfEvents - 1 && r == hipSuccess; ++k) {
      float ms = 0.f;
      r = hipEventElapsedTime(&ms, ev[k], ev[k + 1]);
      if (k == 0 && r != hipSuccess) {  // no preparation launch of its own: ev[0] unrecorded
        (void)hipGetLastError();
        r = hipSuccess;
        ms = 0.f;
      }
      sum[k] += ms;
    }
    if (r != hipSuccess) rc = fail(AFNO_ERR_HIP, std::string("profile events: ") + hipGetErrorString(r));
  }
  for (int k = 0; k < afno::kProfEvents - 1; ++k) kernel_ms[k] = sum[k];
  *calls = g_prof.used;
  for (hipEvent_t e : g_prof.ev) (void)hipEventDestroy(e);
  g_prof.ev.clear();
  g_prof.on = false;
  g_prof.cap = g_prof.used = 0;
  return rc;
}

int afno_set_kernel_path(int path) {
  g_last_error.clear();
  if (path != AFNO_PATH_AUTO && path != AFNO_PATH_GENERIC && path != AFNO_PATH_VALU_DFT)
    return fail(AFNO_ERR_INVALID_ARG,
                "path must be AFNO_PATH_AUTO, AFNO_PATH_GENERIC or AFNO_PATH_VALU_DFT");
  afno::set_kernel_path(path);
  return AFNO_OK;
}

const char* afno_last_error(void) { return g_last_error.c_str(); }

int afno_version(void) { return 100; }

}  // extern "C"
