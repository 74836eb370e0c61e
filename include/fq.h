/*
 * fq.h -- C ABI of libfq, FrameQuant's per-layer quantization pass on AMD Instinct MI355X
 * (gfx950).
 *
 * FrameQuant (Adepu, Zeng, Zhang, Singh, ICML 2024) quantizes one linear layer Theta
 * (d_out x d_in) in the representation of two tight fusion frames: P_l (d_out x K_out)
 * on the output side and P_prev (d_in x K_in) on the input side (Sec. 3, Alg. 1).  The
 * pass has four calls, made in this order:
 *
 *   fq_hessian_accumulate  H   = X^T X over calibration tokens (Sec. 3, proxy loss)
 *   fq_frame_analysis      D   = P_l^T Theta P_prev,  H~ = P_prev^T H P_prev (Alg. 1 step 1)
 *   fq_quantize_frames     2-bit (or 3/4-bit) codes of D with OPTQ-style Hessian-aware rounding and
 *                          Cholesky error feedback after a mu +/- c*sigma clip
 *                          (Alg. 1 steps 2-5)
 *   fq_frame_synthesis     Theta^ = P_l D^ P_prev^T (Alg. 1 return value; appendix
 *                          "Computational Complexity during Inference")
 *
 * fq_quantize_frames is also available as its two phases, fq_quantize_prepare (the part
 * that reads H~ only: damping and the Cholesky factor) and fq_quantize_apply (the part
 * that reads D), so that the factorization can run on one stream while D is still being
 * formed on another; apply in turn splits into fq_quantize_grid (D only: clip and grid,
 * which can also run beside the factorization) and fq_quantize_round (the rounding).
 *
 * Conventions shared by every call
 *  - Matrices are row-major.  Every array argument is a DEVICE pointer owned by the
 *    caller; the library never allocates device memory.  Each call that needs scratch
 *    space takes a caller-provided workspace `ws` of at least the size returned by its
 *    *_workspace_bytes query (16-byte aligned).
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls are stream-ordered and
 *    asynchronous, except fq_quantize_frames, fq_quantize_apply, fq_quantize_round and
 *    fq_quantize_status, which synchronize `stream` once at their end to report the
 *    positive-definiteness and finiteness checks.
 *  - Arguments are validated before anything is launched; on failure the call returns
 *    FQ_ERR_INVALID_ARG (or FQ_ERR_UNSUPPORTED / FQ_ERR_WORKSPACE_TOO_SMALL) and
 *    fq_last_error() describes the problem.  No exception crosses the boundary.
 *  - Calls are thread-safe for distinct buffers and streams; fq_last_error is per thread.
 *  - Sizes may be zero (the call then does nothing, except that fq_hessian_accumulate
 *    with accumulate = 0 still writes H = 0).
 */
#ifndef FQ_H
#define FQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FQ_OK = 0,
  FQ_ERR_INVALID_ARG = 1,           /* bad shape, leading dimension, pointer or scalar */
  FQ_ERR_UNSUPPORTED = 2,           /* valid request the library does not implement */
  FQ_ERR_NOT_POSITIVE_DEFINITE = 3, /* damped H~ has a non-positive Cholesky pivot */
  FQ_ERR_NONFINITE = 4,             /* NaN or Inf in D or H~ */
  FQ_ERR_WORKSPACE_TOO_SMALL = 5,
  FQ_ERR_HIP = 6                    /* a HIP runtime call failed */
} fq_status;

typedef enum { FQ_F32 = 0, FQ_F16 = 1, FQ_BF16 = 2 } fq_dtype;

/*
 * H (+)= X^T X  -- the calibration Hessian (Sec. 3: the FF-space Hessian H~ = C C^T with
 * C = P_prev^T A_prev equals P_prev^T (X^T X) P_prev; A_prev = X^T).
 *   X        device, n_tokens x d_in, element type xt, row stride ldx >= d_in (elements).
 *            f16/bf16 products are exact in fp32; f32 X is split into two bf16 terms
 *            (relative error about 2^-17 per product).
 *   H        device fp32, d_in x d_in, row-major, written in full (exactly symmetric).
 *   accumulate  0: H = X^T X;  1: H += X^T X (chunked calibration sets).
 *   Cross-chunk sums are reduced in fp64 and rounded once to fp32.
 */
fq_status fq_hessian_accumulate(void* stream, const void* X, int xt, int64_t n_tokens,
                                int64_t d_in, int64_t ldx, float* H, int accumulate,
                                void* ws, size_t ws_bytes);
size_t fq_hessian_workspace_bytes(int xt, int64_t n_tokens, int64_t d_in);

/*
 * FF-space weights and Hessian (Alg. 1 step 1; Sec. 3 "What are analogous calculations
 * in FF space?"):
 *   D  = P_out^T W P_in      (K_out x K_in, fp32)      -- skipped when D  == NULL
 *   Ht = P_in^T  H P_in      (K_in x K_in, fp32, exactly symmetric) -- skipped when Ht == NULL
 *   W      device, d_out x d_in, type wt, row stride d_in.
 *   P_out  device fp32, d_out x K_out (columns [P_1 ... P_k], weights absorbed).
 *   P_in   device fp32, d_in  x K_in.
 *   H      device fp32, d_in x d_in symmetric (may be NULL when Ht == NULL).
 * The contractions run on bf16 MFMA with each fp32 operand split into a bf16 pair; the
 * relative error of every product is about 2^-17.
 */
fq_status fq_frame_analysis(void* stream, const void* W, int wt, int64_t d_out, int64_t d_in,
                            const float* P_out, int64_t K_out, const float* P_in, int64_t K_in,
                            const float* H, float* D, float* Ht, void* ws, size_t ws_bytes);
size_t fq_frame_analysis_workspace_bytes(int wt, int64_t d_out, int64_t d_in, int64_t K_out,
                                         int64_t K_in);

/*
 * Quantize the FF-space weights (Alg. 1 steps 2-5, with the OPTQ procedure the paper
 * applies to D and H~, Sec. 3 "Details of the quantization procedure"):
 *  1. mu = mean(D), sigma = std(D) (N - 1) over all of D; D <- clip(D, mu +/- clip_sigmas*sigma).
 *  2. Per-row asymmetric grid from the clipped D: lo = min(0, row min), hi = max(0, row max)
 *     ((lo, hi) = (-1, 1) for an all-zero row); scale = fp32((hi - lo) / (2^bits - 1));
 *     zero = round-half-even(-lo / scale).
 *  3. OPTQ: dead columns (H~_jj == 0) get H~_jj = 1 and D[:, j] = 0; H~ += damp *
 *     mean(diag H~) I; columns are rounded in order with Cholesky error feedback, in
 *     lazy blocks of `block` columns; code = clamp(rne(w / scale) + zero, 0, 2^bits - 1).
 *     All of step 3 runs in fp64.
 *   D       device fp32 K_out x K_in (read only).
 *   Ht      device fp32 K_in x K_in symmetric (the lower triangle is read).
 *   bits    2, 3 or 4 (other widths return FQ_ERR_UNSUPPORTED; the 3- and 4-bit grids
 *           are those of the paper's appendix on segmentation and detection models).
 *   block   >= 1.
 *   codes   device uint32, K_out x ceil(K_in / cpw), cpw = floor(32 / bits) codes per word
 *           (16, 10, 8): column j of row i sits in bits b*(j mod cpw) .. b*(j mod cpw)+b-1
 *           of word floor(j / cpw) of row i (b = bits); pad bits are 0.
 *   scale, zero  device fp32, K_out each (zero is integer valued; bias = -scale * zero).
 * Returns FQ_ERR_NOT_POSITIVE_DEFINITE when the damped H~ is not positive definite
 * (e.g. damp = 0 with K_in > rank H~) and FQ_ERR_NONFINITE when D or H~ holds NaN/Inf;
 * outputs are then unspecified.
 */
fq_status fq_quantize_frames(void* stream, const float* D, const float* Ht, int64_t K_out,
                             int64_t K_in, int bits, int block, double damp,
                             double clip_sigmas, uint32_t* codes, float* scale, float* zero,
                             void* ws, size_t ws_bytes);
size_t fq_quantize_frames_workspace_bytes(int64_t K_out, int64_t K_in, int block);

/*
 * fq_quantize_frames in two phases sharing one workspace (sized by
 * fq_quantize_frames_workspace_bytes(K_out, K_in, block)); prepare + apply on the same
 * workspace gives bit-identical outputs to fq_quantize_frames.
 *   fq_quantize_prepare  reads Ht only: dead columns, damping (step 3 above) and the
 *                        Cholesky factor, into ws.  Asynchronous; its checks are reported
 *                        by the following fq_quantize_apply.
 *   fq_quantize_apply    reads D and the factor in ws: clip, grid and rounding (steps 1-3),
 *                        then synchronizes `stream` and reports the checks of both phases.
 * apply must be ordered after prepare (same stream, or an event the caller records on
 * prepare's stream and makes apply's stream wait for), with the same K_out, K_in, block
 * and workspace.  apply does not modify the factor: one prepare serves any number of
 * applies in stream order (layers that share their input, and so H~, share it too);
 * apply calls on one workspace must not overlap.  Errors as for fq_quantize_frames; the
 * H~ checks of prepare are reported by every apply that follows it.
 */
fq_status fq_quantize_prepare(void* stream, const float* Ht, int64_t K_out, int64_t K_in,
                              int block, double damp, void* ws, size_t ws_bytes);
fq_status fq_quantize_apply(void* stream, const float* D, int64_t K_out, int64_t K_in,
                            int bits, int block, double clip_sigmas, uint32_t* codes,
                            float* scale, float* zero, void* ws, size_t ws_bytes);

/*
 * fq_quantize_apply in its two parts, on the same workspace (apply = grid, then round;
 * the outputs are bit-identical).  The grid reads D only, so it can run beside
 * fq_quantize_prepare.
 *   fq_quantize_grid   reads D only: the clip bounds from D's moments (step 1 above), the
 *                      per-row grid (step 2, writes scale and zero) and the working copy
 *                      of the clipped D, into ws.  Asynchronous; its check (D finite) is
 *                      reported by the following fq_quantize_round.  It writes no part of
 *                      ws that fq_quantize_prepare reads or writes, so the two may run on
 *                      different streams at the same time.
 *   fq_quantize_round  the column-sequential rounding with error feedback (step 3, Alg. 1
 *                      step 4) and the packing into `codes`; then synchronizes `stream`
 *                      and reports the checks of prepare and grid.  It must be ordered
 *                      after both (same stream or events), with the same D, K_out, K_in,
 *                      bits, block and workspace.
 * Errors: as for fq_quantize_apply (clip_sigmas and scale/zero belong to the grid).
 */
fq_status fq_quantize_grid(void* stream, const float* D, int64_t K_out, int64_t K_in, int bits,
                           int block, double clip_sigmas, float* scale, float* zero, void* ws,
                           size_t ws_bytes);
fq_status fq_quantize_round(void* stream, const float* D, int64_t K_out, int64_t K_in, int bits,
                            int block, uint32_t* codes, void* ws, size_t ws_bytes);

/*
 * fq_quantize_round without its synchronization, for a caller that has more work for the
 * stream (the synthesis of the codes, Alg. 1's return value) and wants the device kept
 * busy: fq_quantize_round_async launches the rounding and the packing and returns;
 * fq_quantize_status, called later on the same stream and workspace, synchronizes the
 * stream and reports the checks of prepare, grid and round (the return value
 * fq_quantize_round would have given).  Outputs written before the status call are
 * unspecified when it reports an error.  Arguments and errors as for fq_quantize_round.
 */
fq_status fq_quantize_round_async(void* stream, const float* D, int64_t K_out, int64_t K_in,
                                  int bits, int block, uint32_t* codes, void* ws,
                                  size_t ws_bytes);
fq_status fq_quantize_status(void* stream, int64_t K_out, int64_t K_in, int block, void* ws,
                             size_t ws_bytes);

/*
 * A stream for the work a caller runs beside fq_quantize_prepare (the analysis of W, which
 * only fq_quantize_apply needs).  The factorization that prepare launches is a chain of
 * small dependent kernels that keeps a fraction of the device busy at a time; beside it on
 * an ordinary stream, a kernel with many work-groups takes every compute unit, and each link
 * of the chain then waits for units to drain.  Kernels queued on a stream made here run on
 * every compute unit but `reserve_cus` of them (the first ones in the order of the device's
 * CU mask, hipExtStreamCreateWithCUMask), which stay free for the chain.
 *   reserve_cus  in [0, 3 n_cu / 4], n_cu the current device's compute-unit count; 0 makes
 *                an ordinary non-blocking stream.
 *   *stream      receives the new hipStream_t of the current device (default priority);
 *                release it with fq_side_stream_destroy.
 * A stream with a CU mask synchronizes with the legacy default stream (NULL) as a blocking
 * stream does: the work it runs beside must be queued on another stream, or the two
 * serialize.  The library remembers the streams made here until fq_side_stream_destroy:
 * kernels it queues on them keep many short work-groups (their compute units are shared),
 * where on other streams it may size work-groups to fill the whole device in one round.
 * Errors: FQ_ERR_INVALID_ARG (reserve_cus out of range, stream NULL), FQ_ERR_HIP.
 */
fq_status fq_side_stream_create(int reserve_cus, void** stream);
fq_status fq_side_stream_destroy(void* stream);

/*
 * Synthesis of the dequantized layer (Alg. 1 return value; appendix "Computational
 * Complexity during Inference"):  W_hat = P_out * diag(scale) * (codes - zero) * P_in^T.
 *   codes/scale/zero  as produced by fq_quantize_frames.
 *   P_out  device fp32 d_out x K_out;  P_in device fp32 d_in x K_in.
 *   W_hat  device fp32 d_out x d_in.
 */
fq_status fq_frame_synthesis(void* stream, const uint32_t* codes, const float* scale,
                             const float* zero, int64_t K_out, int64_t K_in,
                             const float* P_out, int64_t d_out, const float* P_in,
                             int64_t d_in, float* W_hat, void* ws, size_t ws_bytes);
/* fq_frame_synthesis for codes of `bits` bits (2, 3 or 4; packed as fq_quantize_frames
 * packs them); fq_frame_synthesis is this with bits = 2.  Same workspace. */
fq_status fq_frame_synthesis_nbit(void* stream, const uint32_t* codes, int bits,
                                  const float* scale, const float* zero, int64_t K_out,
                                  int64_t K_in, const float* P_out, int64_t d_out,
                                  const float* P_in, int64_t d_in, float* W_hat, void* ws,
                                  size_t ws_bytes);
size_t fq_frame_synthesis_workspace_bytes(int64_t K_out, int64_t K_in, int64_t d_out,
                                          int64_t d_in);

/*
 * Layer outputs straight from the stored codes and the frames, without forming Theta^
 * (Sec. 3 "Inference Procedure": the inputs go to their frame representation through the
 * analysis operator P_prev^T, through the quantized D^, and back through the synthesis
 * operator P_l; Theta^ as in the appendix "Computational Complexity during Inference"):
 *   Y = X Theta^T = ((X P_in) (codes - zero)^T diag(scale)) P_out^T
 *   X      device, n_tokens x d_in, element type xt (FQ_F32 / FQ_F16 / FQ_BF16), row
 *          stride ldx >= d_in (elements).
 *   codes/scale/zero  as produced by fq_quantize_frames (K_out x K_in codes).
 *   P_out  device fp32 d_out x K_out;  P_in device fp32 d_in x K_in.
 *   Y      device fp32, n_tokens x d_out, row-major (written; never read).
 *   ws     caller workspace of fq_frame_apply_workspace_bytes(d_in, K_out, K_in) bytes,
 *          16-byte aligned; its contents on entry do not matter.
 * Meant for decode and small batches: every frame and the codes are streamed once per
 * block of 8 tokens (for large token counts form Theta^ with fq_frame_synthesis and use a
 * GEMM).  fp32 arithmetic with fp32 accumulation.  n_tokens == 0 or d_out == 0 is a
 * no-op; d_in, K_out or K_in == 0 writes Y = 0.  Errors (before any launch):
 * FQ_ERR_INVALID_ARG (xt, a dimension outside [0, 2^30), K < d, ldx < d_in, a NULL
 * array), FQ_ERR_WORKSPACE_TOO_SMALL; FQ_ERR_HIP if a launch fails.
 */
fq_status fq_frame_apply(void* stream, const void* X, int xt, int64_t n_tokens, int64_t ldx,
                         int64_t d_in, const uint32_t* codes, const float* scale,
                         const float* zero, int64_t K_out, int64_t K_in, const float* P_out,
                         int64_t d_out, const float* P_in, float* Y, void* ws,
                         size_t ws_bytes);
size_t fq_frame_apply_workspace_bytes(int64_t d_in, int64_t K_out, int64_t K_in);

/*
 * A real tight fusion frame given by its construction instead of a dense matrix (Sec. 2.2
 * "Constructing TFFs"; appendix "Synopsis of Construction of Tight Fusion Frames"):
 *   P = (R1 (x) R2) T / sqrt(k),  d x (k rho), Parseval (P P^T = I),
 * T's column block s < k (rho columns) being the realified subspace s of the complex
 * (k, rho/2, d/2) frame built by spectral tetris and modulation by the k-th roots of
 * unity (complex coordinate j = real pair (2j, 2j+1), complex column c = real pair
 * (2c, 2c+1)), and R1 (x) R2 mapping a vector read row-major as a d1 x d2 matrix M to
 * R1 M R2^T.  Supported: d and rho even, d divisible by rho (the base frame's rows are
 * then blocks of m = d / rho ones), m <= k <= 3968, d1 d2 = d, d2 <= 4096.  R1, R2: device fp32,
 * row-major, owned by the caller.  The transforms below cost d (d1 + d2) + 2 d k FMAs per
 * vector and read no d x K matrix.
 */
typedef struct fq_tff {
  int64_t d, k, rho;
  const float* R1;
  int64_t d1;
  const float* R2;
  int64_t d2;
} fq_tff;

/*
 * Analysis operator on n vectors (Sec. 2 "Operators in Fusion Frames"): U = X P, i.e. row
 * t of U is P^T x_t.  X device n x d, element type xt, row stride ldx >= d; U device fp32
 * n x (k rho), row-major.  ws: fq_tff_analysis_workspace_bytes(n, frame) bytes, 16-byte
 * aligned.  Errors: FQ_ERR_INVALID_ARG (xt, sizes, ldx, NULL arrays, a frame outside the
 * supported set), FQ_ERR_UNSUPPORTED (d not divisible by rho, k > 3968, d2 > 4096),
 * FQ_ERR_WORKSPACE_TOO_SMALL, FQ_ERR_HIP.
 */
fq_status fq_tff_analysis(void* stream, const void* X, int xt, int64_t n, int64_t ldx,
                          const fq_tff* frame, float* U, void* ws, size_t ws_bytes);
size_t fq_tff_analysis_workspace_bytes(int64_t n, const fq_tff* frame);

/*
 * Synthesis operator (the adjoint, same passage): Y = V P^T, row t of Y is P v_t.  V device
 * fp32 n x (k rho); Y device fp32 n x d.  Same workspace rule and errors as the analysis.
 */
fq_status fq_tff_synthesis(void* stream, const float* V, int64_t n, const fq_tff* frame,
                           float* Y, void* ws, size_t ws_bytes);
size_t fq_tff_synthesis_workspace_bytes(int64_t n, const fq_tff* frame);

/*
 * fq_frame_apply with both frames given by their construction (Sec. 3 "Inference
 * Procedure"): Y = ((X P_in) (codes - zero)^T diag(scale)) P_out^T, where P_in is
 * frame_in (d = d_in, K_in = k rho) and P_out is frame_out (d = d_out, K_out = k rho).
 * Reads the codes once per block of 8 tokens and no frame matrix.  X, codes, scale, zero,
 * Y as in fq_frame_apply; ws: fq_frame_apply_tff_workspace_bytes(frame_out, frame_in).
 * Errors as fq_frame_apply and fq_tff_analysis.
 */
fq_status fq_frame_apply_tff(void* stream, const void* X, int xt, int64_t n_tokens,
                             int64_t ldx, const uint32_t* codes, const float* scale,
                             const float* zero, const fq_tff* frame_out,
                             const fq_tff* frame_in, float* Y, void* ws, size_t ws_bytes);
size_t fq_frame_apply_tff_workspace_bytes(const fq_tff* frame_out, const fq_tff* frame_in);
/* fq_frame_apply and fq_frame_apply_tff for codes of `bits` bits (2 or 4, packed as
 * fq_quantize_frames packs them: codes K_out x ceil(K_in / (32 / bits)) words; the
 * appendix on segmentation and detection models quantizes at 4 bits); the 2-bit calls
 * are these with bits = 2.  Same workspaces.  Other widths: FQ_ERR_UNSUPPORTED. */
fq_status fq_frame_apply_nbit(void* stream, const void* X, int xt, int64_t n_tokens, int64_t ldx,
                              int64_t d_in, const uint32_t* codes, int bits, const float* scale,
                              const float* zero, int64_t K_out, int64_t K_in, const float* P_out,
                              int64_t d_out, const float* P_in, float* Y, void* ws,
                              size_t ws_bytes);
fq_status fq_frame_apply_tff_nbit(void* stream, const void* X, int xt, int64_t n_tokens,
                                  int64_t ldx, const uint32_t* codes, int bits, const float* scale,
                                  const float* zero, const fq_tff* frame_out,
                                  const fq_tff* frame_in, float* Y, void* ws, size_t ws_bytes);

/*
 * fq_frame_apply_tff_nbit without a workspace argument and without any allocation, for
 * callers that cannot allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid hipMalloc).  The scratch space is a device array of
 * FQ_NOALLOC_SCRATCH_BYTES inside the library, one per GPU, held until the process ends;
 * its address is looked up on the first call on each device (the stream must belong to
 * the current device).  The call allocates nothing (no hipMalloc, no library routine that
 * allocates) and needs nothing cleared: the array keeps the last call's contents, and
 * every scratch value an output depends on is written earlier in the same call.  Calls
 * on one GPU share its array, so calls that overlap on
 * one GPU (different streams, or host threads without ordering) race and give undefined
 * outputs; order them on one stream.  Arguments, results and errors as
 * fq_frame_apply_tff_nbit; frames whose fq_frame_apply_tff_workspace_bytes exceeds
 * FQ_NOALLOC_SCRATCH_BYTES + 256 return FQ_ERR_UNSUPPORTED before any launch (16 MiB
 * covers frames with 8 (d_in + d_out + K_in + K_out) + d2_out^2 floats up to 4 Mi, e.g.
 * d_in = 28672, d_out = 8192, r = 1.1).
 */
#define FQ_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
fq_status fq_frame_apply_tff_noalloc(void* stream, const void* X, int xt, int64_t n_tokens,
                                     int64_t ldx, const uint32_t* codes, int bits,
                                     const float* scale, const float* zero,
                                     const fq_tff* frame_out, const fq_tff* frame_in, float* Y);

/*
 * The dense frame P (d x k rho, fp32, row stride ldp >= k rho) generated on the device from
 * its construction (the appendix on constructing TFFs; the storage appendix notes that only
 * (k, rho, d) and the rotation need be kept): column s rho + 2c + e of P is the rotated
 * realified vector of subspace s, base-frame row c, real (e = 0) or imaginary (e = 1) part,
 * scaled to a Parseval frame; same conventions and supported set as fq_tff_analysis.
 * ws: fq_tff_materialize_workspace_bytes(frame) bytes, 16-byte aligned.  Errors as
 * fq_tff_analysis.
 */
fq_status fq_tff_materialize(void* stream, const fq_tff* frame, float* P, int64_t ldp, void* ws,
                             size_t ws_bytes);
size_t fq_tff_materialize_workspace_bytes(const fq_tff* frame);

/*
 * S2 with both frames given by their construction (Alg. 1 step 1 and the proxy loss of
 * Sec. 3, with P = (R1 (x) R2) T / sqrt(k) of Sec. 2.2 and the appendix on constructing
 * TFFs): D = P_out^T W P_in and Ht = P_in^T H P_in, the same results as fq_frame_analysis
 * with the materialized frames, computed without them.  Each two-sided product is two
 * row transforms (rotation, then the per-block DFT as batched MFMA products) with a
 * transpose between them: 2 d k + d (d1 + d2) multiply-adds per row and side instead of
 * d k rho.
 *   W          device, d_out x d_in row-major (d_out = frame_out->d, d_in = frame_in->d),
 *              element type wt (FQ_F32, FQ_F16, FQ_BF16); may be NULL when D is NULL.
 *   H          device fp32 d_in x d_in (symmetric); may be NULL when Ht is NULL.
 *   D          device fp32 K_out x K_in (K = k rho) or NULL.
 *   Ht         device fp32 K_in x K_in or NULL; written as (B + B^T) / 2 of the computed
 *              product B, so exactly symmetric.
 * Frames as fq_tff_analysis; in addition d <= 2^21 and K <= 65535 * 32 (else
 * FQ_ERR_UNSUPPORTED).  ws: fq_frame_analysis_tff_workspace_bytes(wt, frame_out,
 * frame_in) bytes, 16-byte aligned.  Stream-ordered; errors as fq_frame_analysis.
 */
fq_status fq_frame_analysis_tff(void* stream, const void* W, int wt, const fq_tff* frame_out,
                                const fq_tff* frame_in, const float* H, float* D, float* Ht,
                                void* ws, size_t ws_bytes);
size_t fq_frame_analysis_tff_workspace_bytes(int wt, const fq_tff* frame_out,
                                             const fq_tff* frame_in);

/*
 * S4 with both frames given by their construction (Alg. 1 return value; the appendix on
 * inference cost): W_hat = P_out diag(scale)(Q - zero) P_in^T from the packed codes of
 * `bits` bits (2, 3 or 4; packed as fq_quantize_frames packs them), the same result as
 * fq_frame_synthesis_nbit with the materialized frames.  Two row syntheses (per-block DFT
 * as batched MFMA products, then the rotation) with a gather between them.
 *   codes, scale, zero  as fq_frame_synthesis_nbit, K_out = frame_out->k rho,
 *                       K_in = frame_in->k rho.
 *   W_hat               device fp32 frame_out->d x frame_in->d.
 * Frames and limits as fq_frame_analysis_tff.  ws: fq_frame_synthesis_tff_workspace_bytes
 * (frame_out, frame_in) bytes, 16-byte aligned.  Stream-ordered; errors as
 * fq_frame_synthesis.
 */
fq_status fq_frame_synthesis_tff(void* stream, const uint32_t* codes, int bits,
                                 const float* scale, const float* zero, const fq_tff* frame_out,
                                 const fq_tff* frame_in, float* W_hat, void* ws, size_t ws_bytes);
size_t fq_frame_synthesis_tff_workspace_bytes(const fq_tff* frame_out, const fq_tff* frame_in);

/*
 * The two rotation factors of a frame drawn on the device from a 64-bit seed (Sec. 2.2 and
 * the appendix on constructing TFFs take a random rotation; the storage appendix keeps
 * only (k, rho, d) and what regenerates it).  The paper names no generator; the recipe:
 * Philox4x32-10 (Salmon et al., SC'11) with key = the seed's two 32-bit halves and
 * counter = (pair index, factor index (0: R1, 1: R2), 0), two uniforms of 53 bits per
 * output, Box-Muller to an n x n Gaussian matrix G (row-major), and the factor is Q of
 * the QR of G with R's diagonal positive (a Haar-distributed orthogonal matrix), formed
 * by fp64 Householder reflections and stored in fp32.
 *   R1, R2   device fp32 d1 x d1 and d2 x d2, row-major, written; usable as fq_tff.R1/R2.
 * 1 <= d1, d2 <= 1024 (larger: FQ_ERR_UNSUPPORTED).  ws:
 * fq_tff_rotation_factors_workspace_bytes(d1, d2) bytes, 16-byte aligned.  Stream-ordered;
 * one work-group forms each factor (about n^3 fp64 operations, milliseconds at n = 224).
 */
fq_status fq_tff_rotation_factors(void* stream, uint64_t seed, int64_t d1, int64_t d2, float* R1,
                                  float* R2, void* ws, size_t ws_bytes);
size_t fq_tff_rotation_factors_workspace_bytes(int64_t d1, int64_t d2);

/*
 * Choice of a constructible frame (Sec. 2.2 "Constructing TFFs" and the appendix on
 * constructing TFFs: spectral tetris builds a unit-norm tight frame of d/2 vectors in
 * C^(rho/2), whose modulation by the k-th roots of unity is a tight fusion frame exactly
 * when no row of that frame has two support columns congruent mod k; with rows supported
 * on runs of consecutive columns, when its longest row support is at most k; realified
 * this is a real (k, rho, d) frame).  Host functions, no device work.
 *   fq_tff_frame_valid  1 if (d, k, rho) passes that rule (d, rho even, spectral tetris
 *                       succeeds for (rho/2, d/2)), else 0.
 *   fq_tff_choose       the frame of redundancy r = k rho / d closest to the request that is
 *                       constructible: k = round(r d / rho) (ties to even), lowered until
 *                       valid (the paper lowers the redundancy when a (k, rho) is not
 *                       valid); and the split d = d1 d2 of its Kronecker rotation (d1 the
 *                       largest divisor of d not above sqrt(d)).  d1 / d2 may be NULL.
 *                       Errors: FQ_ERR_INVALID_ARG (d or rho odd or < 2, r not > 0),
 *                       FQ_ERR_UNSUPPORTED (no valid k >= 1).
 * With the factors drawn by fq_tff_rotation_factors(seed, d1, d2), (d, k, rho, seed) is
 * all a frame needs to be regenerated (the storage appendix).
 */
int fq_tff_frame_valid(int64_t d, int64_t k, int64_t rho);
fq_status fq_tff_choose(int64_t d, double r, int64_t rho, int64_t* k, int64_t* d1, int64_t* d2);

/*
 * Rounding of the frame representation of activations to act_bits-bit integers (appendix
 * "FrameQuant for Activation Quantization?"): per token t (row of U),
 * Delta_t = max_j |U_tj| / (2^(act_bits-1) - 1) and Cq_tj = round(U_tj / Delta_t), with
 * IEEE fp32 divisions and ties to even; a zero row gives Delta_t = 0 and Cq_t = 0.
 *   U device fp32 n x K row-major; Cq device int8 n x K row-major; delta device fp32 n.
 *   act_bits in [2, 8].  No workspace.  Errors: FQ_ERR_INVALID_ARG, FQ_ERR_HIP.
 */
fq_status fq_act_quantize(void* stream, const float* U, int64_t n, int64_t K, int act_bits,
                          int8_t* Cq, float* delta);

/*
 * fq_frame_apply_tff with the inputs' frame representation C = X P_in rounded per token as
 * fq_act_quantize does (same appendix): Y = (Delta C^ (codes - zero)^T diag(scale)) P_out^T,
 * where the products with the codes run exactly in integer arithmetic (int32 sums of
 * int8 x b-bit terms).  Arguments and errors as fq_frame_apply_tff, plus bits, the code
 * width (2 or 4, packed as fq_quantize_frames packs them; 3 returns FQ_ERR_UNSUPPORTED),
 * and act_bits in [2, 8] (the appendix reports W4/A4); ws:
 * fq_frame_apply_tff_actq_workspace_bytes(frame_out, frame_in) bytes (any code width).
 */
fq_status fq_frame_apply_tff_actq(void* stream, const void* X, int xt, int64_t n_tokens,
                                  int64_t ldx, const uint32_t* codes, int bits,
                                  const float* scale, const float* zero,
                                  const fq_tff* frame_out, const fq_tff* frame_in, int act_bits,
                                  float* Y, void* ws, size_t ws_bytes);
size_t fq_frame_apply_tff_actq_workspace_bytes(const fq_tff* frame_out, const fq_tff* frame_in);

/*
 * Diagonal Wiener (linear MMSE) filter at synthesis (appendix "LMMSE estimation from fusion
 * frame measurements"; Sec. 3 "Robustness of Fusion Frames" (b)): the layer output
 * Z = P_l D C (C = P_prev^T A_prev) is estimated from the quantized coefficients as
 * F D^ C instead of P_l D^ C.  The paper uses a diagonal approximation of the filter and
 * does not print it; the reading implemented here is F = P_l diag(g) with one gain per
 * frame-coefficient row, each minimising that row's share ||(D_i - g_i D^_i) C||^2 of the
 * output error on the calibration set:
 *   g_i = (D H~ D^^T)_ii / (D^ H~ D^^T)_ii,   D^ = diag(scale) (codes - zero),
 * and g_i = 1 where the denominator is 0.  The gains fold into the stored scale
 * (scale_i g_i), so every synthesis and inference call applies the filter unchanged.
 *   D      device fp32 K_out x K_in: the unclipped analysis output (as fq_frame_analysis
 *          wrote it; fq_quantize_frames does not modify it).
 *   Ht     device fp32 K_in x K_in: the undamped H~ of the calibration set (symmetric).
 *   codes, bits, scale, zero: as fq_quantize_frames wrote them (bits 2, 3 or 4).
 *   gain   device fp32 K_out, written.
 *   scale_out  device fp32 K_out or NULL: fp32(g_i scale_i); may be the same array as scale.
 * D^ H~ runs on bf16 MFMA (the codes exact, H~ as a bf16 pair: relative error about 2^-17)
 * with fp32 accumulation; the row sums are fp64.  ws: fq_wiener_gains_workspace_bytes
 * (K_out, K_in) bytes, 16-byte aligned.  Errors: FQ_ERR_INVALID_ARG (dimensions, NULL
 * arrays), FQ_ERR_UNSUPPORTED (bits), FQ_ERR_WORKSPACE_TOO_SMALL, FQ_ERR_HIP.
 */
fq_status fq_wiener_gains(void* stream, const float* D, const float* Ht, const uint32_t* codes,
                          int bits, const float* scale, const float* zero, int64_t K_out,
                          int64_t K_in, float* gain, float* scale_out, void* ws, size_t ws_bytes);
size_t fq_wiener_gains_workspace_bytes(int64_t K_out, int64_t K_in);

/* Status text and the calling thread's last error message (never NULL). */
const char* fq_status_string(int status);
const char* fq_last_error(void);

/*
 * Kernel timing (tracing).  While enabled, every kernel the library launches is
 * bracketed with HIP events on the stream it runs on, and work the library would
 * otherwise put on its own auxiliary stream (the factorization's look-ahead) runs on the
 * caller's stream, so that timed kernels of one call never overlap.  fq_profile_query synchronizes
 * those events and returns the launch count and total milliseconds of kernels whose name
 * starts with `prefix` (all kernels for ""), since the last reset.  Not thread-safe.
 */
void fq_profile_enable(int on);
void fq_profile_reset(void);
int fq_profile_query(const char* prefix, int* count, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* FQ_H */
