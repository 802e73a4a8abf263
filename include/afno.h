/*
 * afno.h -- C ABI of the MI355X (gfx950) AFNO spectral token-mixing filter.
 *
 * The filter is the spatial-mixing step of the FourCastNet AFNO transformer
 * (section "Model Innovations", the three steps: a 2-D FFT of the token grid, a
 * block-diagonal MLP applied to every token in Fourier space with weights shared by
 * all tokens, an inverse FFT), implemented with real-to-complex / complex-to-real
 * transforms batched over batch and channels, complex weights stored as real arrays
 * with (re, im) as the fastest index and activations acting on the real and
 * imaginary parts independently (section "Implementation Details" (b), "Spectral
 * convolution").  Softshrink, the hard mode cutoff and the residual come from the
 * AFNO layer the paper builds on.  Every step runs in hand-written HIP kernels.
 *
 * For one sample, with Wm = W/2 + 1, nb blocks of bs = C/nb channels, hs = bs:
 *   X[kh][kw][c] = (1/sqrt(HW)) sum_{h,w} x[h][w][c] exp(-2 pi i (kh h/H + kw w/W)),  kw <= W/2
 *   for every mode kept by the cutoff and every block k (true complex products):
 *     v[j] = b1[k][j] + sum_i X[k bs + i] w1[k][i][j];  h[j] = ReLU(Re v[j]) + i ReLU(Im v[j])
 *     o[i] = b2[k][i] + sum_j h[j] w2[k][j][i]
 *     Y[k bs + i] = S(Re o[i]) + i S(Im o[i]),  S(v) = v - lambda (v > lambda),
 *                                              v + lambda (v < -lambda), 0 otherwise
 *   modes outside the cutoff: Y = 0
 *   y[h][w][c] = (1/sqrt(HW)) sum_{kh, kw<=W/2} c_kw Re(Y[kh][kw][c] exp(+2 pi i (kh h/H + kw w/W))),
 *                c_kw = 1 for kw = 0 and kw = W/2, 2 otherwise
 *   out = x + y, rounded once to the storage dtype.
 * Hard mode cutoff (keep_fraction f): kept_h = floor((H/2+1) f) and
 * kept_w = floor((W/2+1) f), both evaluated in double; a mode (kh, kw) is kept when
 * |kh'| < kept_h, kh' = kh for kh <= H/2 and kh - H above, and kw < kept_w.
 * f = 1 keeps every mode; when either count is 0 nothing is kept and out = x.
 */
#ifndef AFNO_H_
#define AFNO_H_

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Storage dtype of x, the weights, the biases and out. */
typedef enum { AFNO_DTYPE_FP32 = 0, AFNO_DTYPE_BF16 = 1 } afno_dtype_t;

/* Return codes. */
enum {
  AFNO_OK = 0,
  AFNO_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, C % nb != 0, bad lambda/keep/dtype */
  AFNO_ERR_UNSUPPORTED = -2, /* valid filter this library does not run: see afno_filter_forward */
  AFNO_ERR_ALIAS = -3,       /* out overlaps an input */
  AFNO_ERR_HIP = -4          /* a HIP allocation or launch failed; see afno_last_error() */
};

/*
 * afno_filter_forward -- out = x + filter(x) (the filter defined above).
 *
 *   x    [B][H][W][C]        dtype, row-major (channels fastest), device memory
 *   w1   [nb][bs][hs][2]     dtype, complex (re, im) fastest, input-major: x @ w1
 *   b1   [nb][hs][2]         dtype
 *   w2   [nb][hs][bs][2]     dtype
 *   b2   [nb][bs][2]         dtype
 *   B >= 0; H, W, C, num_blocks > 0; C % num_blocks == 0; hs = bs = C / num_blocks
 *   lambda         softshrink threshold, finite and >= 0
 *   keep_fraction  hard mode cutoff f, 0 < f <= 1
 *   dtype          an afno_dtype_t
 *   out  [B][H][W][C]        dtype, device memory, must not overlap any input
 *   stream         HIP stream the work is enqueued on (0 = the null stream)
 *
 * Ownership: the caller owns every array; all are contiguous device memory on the
 * current device and must stay valid until the stream has finished the work.  The
 * library allocates a spectrum workspace of B*H*kept_w*C complex values (8 bytes each
 * for fp32, 4 for bf16) stream-ordered on `stream` and frees it stream-ordered, from a
 * memory pool of its own per device that keeps freed memory for later calls (so the
 * largest workspaces in use at once stay allocated until the process ends).
 * The call is asynchronous: it enqueues on `stream` and returns.
 * B == 0 returns AFNO_OK without touching the GPU (x and out may then be NULL).
 * Errors: arguments are validated before any HIP call; on a non-OK return nothing
 * has been enqueued, except for AFNO_ERR_HIP from a launch, after which out is
 * undefined.  AFNO_ERR_UNSUPPORTED: H or W not of the form 2^a 3^b 5^c, W odd,
 * bs not a multiple of 16 or above 128, or a grid too large for on-chip storage
 * (a column of H complex values x bs channels must fit the 160 KiB LDS of one CU,
 * H <= 192 for bs = 128, and W <= 1024), or a spectrum column (H * kept_w * C complex
 * values) or a grid row (W * C float32 values) larger than 4 GiB: the kernels address
 * them with 32-bit byte offsets.
 * Thread safety: calls from several host threads are safe; calls whose streams
 * overlap in time only share read-only inputs.
 */
int afno_filter_forward(const void* x, const void* w1, const void* b1, const void* w2,
                        const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                        int64_t num_blocks, float lambda, float keep_fraction, int dtype,
                        void* out, hipStream_t stream);

/*
 * afno_filter_forward_noalloc -- afno_filter_forward for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Same arguments, kernels and result (bitwise) as afno_filter_forward; the call allocates
 * nothing.  Its workspace (the spectrum, B*H*kept_w*C complex values of 4 bytes (bf16) or 8
 * (fp32), then the prepared block weights and the DFT table, about 1.2 MB for 8 blocks of 96)
 * is an array of AFNO_NOALLOC_MAX_WORKSPACE bytes in device memory that the library holds on
 * every GPU it runs on until the process ends (the 90 x 180 x 768 bf16 filter fits up to
 * B = 5).  AFNO_ERR_UNSUPPORTED, before any HIP call, when the workspace would be larger.
 * Every call on a GPU uses that GPU's one array, which keeps the last call's contents (each
 * call writes all it reads): calls whose work overlaps in time on one GPU (different streams
 * or host threads without ordering between them) race and leave out undefined; calls on one
 * stream are ordered and safe.  The first call on a device also resolves the array's address
 * there (hipGetSymbolAddress; AFNO_ERR_HIP if that fails).  Other errors as
 * afno_filter_forward.
 */
#define AFNO_NOALLOC_MAX_WORKSPACE (128u << 20)
int afno_filter_forward_noalloc(const void* x, const void* w1, const void* b1, const void* w2,
                                const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                                int64_t num_blocks, float lambda, float keep_fraction, int dtype,
                                void* out, hipStream_t stream);

/*
 * afno_filter_forward_hidden -- the same filter with `hidden` hidden units per block in
 * the block MLP (the AFNO layer's hidden-size factor: hidden = factor * bs; the paper's
 * filter, "Model Innovations", uses hidden = bs, which afno_filter_forward assumes).
 *   w1 [nb][bs][hidden][2], b1 [nb][hidden][2], w2 [nb][hidden][bs][2], b2 [nb][bs][2]
 *   hidden > 0 (AFNO_ERR_INVALID_ARG otherwise); a multiple of 16 and <= 256, and the
 *   column's hidden layer (H x hidden complex values) must fit in LDS beside the column
 *   tile (AFNO_ERR_UNSUPPORTED otherwise).  hidden == bs runs exactly afno_filter_forward.
 * Other arguments, ownership and errors as afno_filter_forward.  hidden == 2 * bs with bf16
 * storage, H <= 96 and bs 32, 64 or 96 runs a matrix-core column kernel (the workspace holds
 * its weight fragments and the DFT table besides the spectrum); other hidden sizes run the
 * size-generic column kernel.
 */
int afno_filter_forward_hidden(const void* x, const void* w1, const void* b1, const void* w2,
                               const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                               int64_t num_blocks, int64_t hidden, float lambda,
                               float keep_fraction, int dtype, void* out, hipStream_t stream);

/*
 * afno_block_forward -- one AFNO transformer block around the filter: the paper's layer
 * mixes tokens with the spectral filter and channels with a single-hidden-layer MLP of four
 * times the embedding width shared by all tokens ("Model Innovations"; "Implementation
 * Details" (c)).  With per-token LayerNorms (the paper states none; the AFNO layer's pre-norm
 * arrangement is taken) and the exact GELU:
 *   t = LN1(x);  v = x + filter(t)  (the filter includes its own residual: filter(t) = t + y);
 *   w = LN2(v);  out = v + GELU(w wa + ba) wb + bb
 *   LN(z) = (z - mean) / sqrt(var + 1e-6) * gamma + beta over the C channels of a token,
 *   biased variance.
 *   x, out       [B][H][W][C] bf16; tokens are the rows of x viewed as [B*H*W][C]
 *   ln1_g, ln1_b, ln2_g, ln2_b  [C] bf16, 16-byte aligned
 *   w1, b1, w2, b2              the filter's weights, as afno_filter_forward
 *   wa [C][4C], ba [4C], wb [4C][C], bb [C]   bf16, input-major (z wa)
 * dtype must be AFNO_DTYPE_BF16 (fp32: AFNO_ERR_UNSUPPORTED); C a multiple of 128 and
 * <= 2048; the filter's limits as afno_filter_forward.  out must not overlap any input
 * (AFNO_ERR_ALIAS).  The library allocates one stream-ordered workspace (four token grids,
 * the B*H*W x 4C hidden layer in bf16, the transposed MLP weights and the filter's spectrum)
 * and frees it stream-ordered.  Intermediates (t, the filter output, v, w, the hidden layer)
 * are rounded to bf16; products accumulate in fp32.  Other arguments, ownership, errors and
 * asynchrony as afno_filter_forward.
 */
int afno_block_forward(const void* x, const void* ln1_g, const void* ln1_b, const void* w1,
                       const void* b1, const void* w2, const void* b2, const void* ln2_g,
                       const void* ln2_b, const void* wa, const void* ba, const void* wb,
                       const void* bb, int64_t B, int64_t H, int64_t W, int64_t C,
                       int64_t num_blocks, float lambda, float keep_fraction, int dtype,
                       void* out, hipStream_t stream);

/*
 * afno_filter_stage -- diagnostic entry point: runs the filter's kernels up to a stage
 * and writes that stage's result in float32, for per-stage parity checks.
 *   stage AFNO_STAGE_SPECTRUM  dst [B][H][Wm][C][2] float32: the forward spectrum X
 *                              (both axes, ortho-normalised); columns kw >= kept_w
 *                              are not computed and are written as 0.
 *   stage AFNO_STAGE_MIXED     dst [B][H][Wm][C][2] float32: Y after the block MLP,
 *                              softshrink and the cutoff.
 *   stage AFNO_STAGE_DELTA     dst [B][H][W][C] float32: y = filter(x) before the
 *                              residual add and before rounding to dtype.
 * Other arguments, ownership and errors as afno_filter_forward, with dst in place of
 * out.  The values are what the kernels hold at that point (for bf16 storage the
 * spectra are bf16-rounded).
 */
enum { AFNO_STAGE_SPECTRUM = 1, AFNO_STAGE_MIXED = 2, AFNO_STAGE_DELTA = 3 };
int afno_filter_stage(const void* x, const void* w1, const void* b1, const void* w2,
                      const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                      int64_t num_blocks, float lambda, float keep_fraction, int dtype,
                      int stage, float* dst, hipStream_t stream);

/*
 * afno_filter_stage_hidden -- afno_filter_stage for the block MLP with `hidden` units per
 * block (weights as afno_filter_forward_hidden).  AFNO_STAGE_DELTA runs the same kernels as
 * afno_filter_forward_hidden up to the inverse W-axis transform; AFNO_STAGE_SPECTRUM and
 * AFNO_STAGE_MIXED stop inside the column pass, which for hidden != bs is the size-generic
 * column kernel.  Arguments, ownership and errors as afno_filter_stage and
 * afno_filter_forward_hidden (hidden <= 0: AFNO_ERR_INVALID_ARG).
 */
int afno_filter_stage_hidden(const void* x, const void* w1, const void* b1, const void* w2,
                             const void* b2, int64_t B, int64_t H, int64_t W, int64_t C,
                             int64_t num_blocks, int64_t hidden, float lambda,
                             float keep_fraction, int dtype, int stage, float* dst,
                             hipStream_t stream);

/*
 * afno_filter_backward -- gradients of a loss L through out = x + filter(x), given
 * gout = dL/dout: the transpose of the filter's forward map (the paper trains through it:
 * "Implementation Details" (a), (e)), step by step in reverse order.  With X the forward
 * spectrum, v = X w1 + b1, h = relu(v), o = h w2 + b2 per kept mode and block as above:
 *   dz  = c_kw F(gout)            (F the forward 2-D transform, c_kw its inverse's weights)
 *   do  = dz where |o| > lambda on that component and the mode is kept, else 0
 *   dh  = do w2^H (conjugate transpose),  dv = dh where v > 0 on that component, else 0
 *   dx  = gout + F^T(dv w1^H)     (F^T: the inverse with unit weights c_kw = 1)
 *   dw1 = sum over kept modes of conj(X)^T dv,  db1 = sum of dv
 *   dw2 = sum over kept modes of conj(h)^T do,  db2 = sum of do
 * (re, im pairs hold d/d re and d/d im; relu'(0) = 0 and the softshrink slope is 0 on
 * [-lambda, lambda]).
 *   x, w1, b1, w2, b2, sizes, lambda, keep_fraction, dtype   as afno_filter_forward
 *   gout [B][H][W][C]        dtype, device memory
 *   dx   [B][H][W][C]        dtype, device memory
 *   dw1, dw2 [nb][bs][bs][2]  float32, device memory, overwritten (not accumulated)
 *   db1, db2 [nb][bs][2]      float32, device memory, overwritten
 * No output may overlap an input or another output (AFNO_ERR_ALIAS).  The library
 * allocates stream-ordered workspace on `stream`: two spectra, the conjugate-transposed
 * weights, four per-mode factor tensors of nb * 2 bs * B * kept_w * ceil32(ceil16(H)) values
 * in dtype, and float32 chunk sums (2 nb 2 bs (2 bs + 1) per chunk of modes, at most 64
 * chunks).  B == 0 or nothing kept: dx = gout and zero weight and bias gradients.  Errors as
 * afno_filter_forward; AFNO_ERR_UNSUPPORTED also when a column of the backward kernel (one
 * tile of H x bs complex values plus two bit masks) does not fit the LDS.  Reproducibility:
 * no atomics; the weight and bias gradients are chunk sums stored by the weight-product
 * kernels and added in a fixed order, so repeated calls give the same bits.
 */
int afno_filter_backward(const void* x, const void* w1, const void* b1, const void* w2,
                         const void* b2, const void* gout, int64_t B, int64_t H, int64_t W,
                         int64_t C, int64_t num_blocks, float lambda, float keep_fraction,
                         int dtype, void* dx, float* dw1, float* db1, float* dw2, float* db2,
                         hipStream_t stream);

/*
 * Diagnostic per-kernel timing.  afno_profile_begin(max_calls) creates HIP events for
 * up to max_calls filter calls (process-wide); each later afno_filter_forward call
 * records an event before its first kernel and after each of its four phases, on the
 * call's stream.  afno_profile_end waits for those events, writes the summed
 * milliseconds of each phase to kernel_ms[0..3] (0: operand preparation as a launch of its
 * own -- the block weights in MFMA fragment order and the H-axis DFT table; exactly 0 where
 * there is no such launch, the column kernel taking none or the preparation running as extra
 * workgroups of the size-specialised W-axis forward launch; 1: W-axis forward transform; 2: column kernel,
 * H transforms + block MLP; 3: W-axis inverse transform + residual) and the number of timed calls to *calls, and
 * frees the events.  Calls beyond max_calls are not timed.
 * Returns AFNO_OK, AFNO_ERR_INVALID_ARG (max_calls <= 0, null output, or end without
 * begin) or AFNO_ERR_HIP.  Not for concurrent use with calls on other streams.
 */
int afno_profile_begin(int max_calls);
int afno_profile_end(double* kernel_ms, int64_t* calls);

/*
 * Diagnostic kernel selection, process-wide.  AFNO_PATH_AUTO (the default) runs the
 * specialised kernels where the library has them and the size-generic kernels elsewhere:
 * W-axis kernels for W in {32, 180, 360}; for bf16 with H <= 96 and bs in {32, 64, 96}
 * the column kernel that computes the H-axis DFTs as bf16 matrix-core products against a
 * DFT table (and its hidden-size variant for hidden = 2 bs); else column kernels with
 * vector-ALU FFTs for H x bs in {16 x 16, 90 x 96, 180 x 32, and for bf16 180 x 64 and
 * 180 x 128}.  AFNO_PATH_VALU_DFT is AUTO without the matrix-core DFT column kernels;
 * AFNO_PATH_GENERIC runs the size-generic kernels for every shape.  All compute the same
 * filter (the matrix-core DFT rounds its table to bf16: one more bf16-sized error per H
 * transform).  Returns AFNO_OK or AFNO_ERR_INVALID_ARG.  Safe while other threads enqueue
 * calls: a call reads the setting once, when it sizes its workspace, and runs that path
 * throughout.
 */
enum { AFNO_PATH_AUTO = 0, AFNO_PATH_GENERIC = 1, AFNO_PATH_VALU_DFT = 2 };
int afno_set_kernel_path(int path);

/* Message of the calling thread's last non-OK return ("" if none).  The pointer
 * stays valid until the thread's next call into the library. */
const char* afno_last_error(void);

/* Library version as major*10000 + minor*100 + patch. */
int afno_version(void);

#ifdef __cplusplus
}
#endif
#endif /* AFNO_H_ */
