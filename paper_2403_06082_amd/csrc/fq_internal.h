// Internal declarations shared by the libfq translation units (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace fq {

typedef uint16_t u16;

// ---------------------------------------------------------------- launch bookkeeping
// Every launch goes through prof_begin/prof_end so that the optional kernel timer can
// bracket it with events on the launch stream.
void prof_begin(hipStream_t s, const char* name);
void prof_end(hipStream_t s);
// whether the kernel timer is on (work that would otherwise go to an auxiliary stream
// then stays on the caller's stream, so that no two timed kernels overlap)
bool prof_enabled();
hipError_t last_launch_error();

// ---------------------------------------------------------------- bf16 MFMA GEMM engine
// C = sum over passes p of A[pa[p]] * B[pb[p]], fp32 accumulation, where A is M x K and
// B is K x N, both given as 16-bit planes (bf16, or f16 for the Hessian of f16 inputs).
//   a_kmajor: A(m, k) at a[m * lda + k]   else at a[k * lda + m]
//   b_kmajor: B(k, n) at b[n * ldb + k]   else at b[k * ldb + n]
enum Epilogue {
  EPI_F32 = 0,      // c[row * ldc + col] = acc
  EPI_SPLIT = 1,    // c_hi/c_lo[row * ldc + col] = bf16 pair of acc
  EPI_SYM = 2,      // upper tiles only; c[row][col] and c[col][row] for row <= col
  EPI_PARTIAL = 3,  // upper tiles only, split over K; fp32 partial tiles, tile-major
  EPI_TAIL = 4      // internal: tiles of a short last round, split over K (fp32 partials)
};

struct GemmDesc {
  int M = 0, N = 0, K = 0;
  const u16* a[2] = {nullptr, nullptr};
  const u16* b[2] = {nullptr, nullptr};
  int64_t lda = 0, ldb = 0;
  int npass = 1;
  int pa[3] = {0, 0, 0}, pb[3] = {0, 0, 0};
  bool a_kmajor = true, b_kmajor = true;
  bool f16 = false;              // operands are IEEE half instead of bf16
  int epi = EPI_F32;
  float* c = nullptr;
  int64_t ldc = 0;
  u16* c_hi = nullptr;
  u16* c_lo = nullptr;
  int ksplit = 1;                // EPI_PARTIAL only
  const char* name = "gemm";     // kernel-timer label
  int64_t ldc_pad = 0;           // EPI_SPLIT: output columns [N, ldc_pad) are zeroed
  // batch > 1 (EPI_F32 only): products z < batch read A + z bsa, B + z bsb and write
  // C + z bsc (element strides; bsa and bsb multiples of 8)
  int batch = 1;
  int64_t bsa = 0, bsb = 0, bsc = 0;
  // EPI_F32 (asynchronous path): output row r goes to row (r / 2) rowmap + r % 2 when
  // rowmap > 0 (the frame order of a per-block DFT product)
  int rowmap = 0;
};

// Workspace bytes needed by EPI_PARTIAL for an N x N symmetric product split ksplit ways.
size_t gemm_partial_bytes(int N, int ksplit);
int gemm_sym_tiles(int N);
int64_t gemm_tiles(int64_t M, int64_t N);   // output tiles of an M x N product
// partial: EPI_PARTIAL's workspace, or (for EPI_F32 / EPI_SPLIT) an optional scratch of
// gemm_tail_bytes() that lets a short last round of tiles be split over K.
hipError_t gemm_run(const GemmDesc& d, float* partial, hipStream_t s);
size_t gemm_tail_bytes();
// H (+)= sum of the ksplit partial tiles (fp64), mirrored to full symmetric storage.
hipError_t syrk_reduce(const float* partial, int N, int ksplit, float* H, int64_t ldh,
                       int accumulate, hipStream_t s);

// fp32 / f16 -> bf16 (hi, lo) planes with out[r * ld_out + c]; optional column scale
// (applied in fp32 before the split).  Element type: 0 = f32, 1 = f16.
hipError_t split_bf16(const void* in, int in_type, int64_t ld_in, int rows, int cols,
                      const float* col_scale, u16* hi, u16* lo, int64_t ld_out, hipStream_t s);
// Same with zero padding: out has rows_out >= rows rows and ld_out >= cols columns; rows
// [rows, rows_out) and columns [cols, ld_out) are 0.  Element type 2 = bf16.
hipError_t split_bf16_pad(const void* in, int in_type, int64_t ld_in, int rows, int cols,
                          const float* col_scale, u16* hi, u16* lo, int64_t ld_out,
                          int rows_out, hipStream_t s);
hipError_t fill_zero_f32(float* p, int rows, int cols, int64_t ld, hipStream_t s);

// ---------------------------------------------------------------- layer outputs from codes
// Y = X Theta^T from the packed codes and the frames, tokens in blocks of APPLY_NT.
constexpr int APPLY_NT = 8;
struct ApplyScratch {
  float* part;   // split-K partials of U = X P_in
  float* U;      // APPLY_NT x pad16(K_in)
  float* V;      // APPLY_NT x K_out
};
// floats of scratch (and, with base, the carve-up); base 256-byte aligned
size_t apply_scratch_floats(int64_t d_in, int64_t K_out, int64_t K_in, ApplyScratch* w,
                            float* base);
// X: n x d_in (row stride ldx, element type xt: 0 f32, 1 f16, 2 bf16); Y: n x d_out fp32
// V (rows [0, tokens-per-block) with tokens-per-block = 1, 2, 4 or 8 >= nt) = scale *
// (U (codes - zero)^T) for U with ldu = 16 * ceil(K_in / 16) columns, zero beyond K_in.
// bits: 2 or 4 (nwords = ceil(K_in / 16) or ceil(K_in / 8) per code row)
hipError_t apply_codes(const float* U, int64_t ldu, int nt, const uint32_t* codes,
                       int64_t K_out, int64_t nwords, const float* scale, const float* zero,
                       float* V, hipStream_t s, int bits = 2);
// ---------------------------------------------------------------- structured frames
// A validated tight fusion frame given by its construction (see tff_apply.hip):
// m = d / rho, R1 d1 x d1 and R2 d2 x d2 device fp32, d1 d2 = d.
struct TffDev {
  int64_t d, k, rho, m;
  const float* R1;
  int d1;
  const float* R2;
  int d2;
};
constexpr int64_t TFF_MAX_K = 3968;       // twiddles + one block of a vector within 64 KB of LDS
constexpr int64_t TFF_MAX_D2 = 4096;     // one row of the rotation's d1 x d2 view in LDS
constexpr int64_t TFF_CHUNK = 256;        // vectors per pass of the stand-alone transforms
// U (n x ldu, ldu >= k rho, columns beyond k rho set to 0) = X P; y: n x d scratch
hipError_t tff_analysis(const void* X, int xt, int64_t ldx, int64_t n, const TffDev& F,
                        float* y, float* U, int64_t ldu, hipStream_t s);
// P (d x k rho, row stride ldp) of the frame, nc_max columns at a time; R2t from
// tff_transpose_r2; Z, Pt: nc_max x d scratch each
hipError_t tff_materialize(const TffDev& F, const float* R2t, float* Z, float* Pt, int64_t nc_max,
                           float* P, int64_t ldp, hipStream_t s);
// R2t (d2 x d2) = R2^T, read by tff_synthesis
hipError_t tff_transpose_r2(const TffDev& F, float* R2t, hipStream_t s);

// Structured analysis / synthesis of whole matrices (tff_pass.hip).  Block geometry of a
// frame: nb = rho / 2 blocks of m2 = 2m real coordinates (padded to pm) and k2 = 2k
// frame coordinates (padded to pk), pads multiples of 32.
struct TffPassGeom { int64_t nb, m2, pm, k2, pk; };
TffPassGeom tff_pass_geom(const TffDev& F);
// F_c for all blocks: bf16 (hi, lo) planes of nb x pm x pk each; with colscale (K
// entries), the blocks of P diag(colscale)
hipError_t tff_dft_blocks(const TffDev& F, u16* hi, u16* lo, hipStream_t s,
                          const float* colscale = nullptr);
// out (K x n at stride ldout) = (X P)^T for n rows of X (element type xt, stride ldx).
// Scratch: tmp / O one fp32 buffer of max(n d, n K) (they may alias), Y pair planes of
// n x nb pm each.
hipError_t tff_rows_analysis_t(const void* X, int xt, int64_t ldx, int64_t n, const TffDev& F,
                               const u16* Fhi, const u16* Flo, float* tmp, u16* Yhi, u16* Ylo,
                               float* O, float* out, int64_t ldout, hipStream_t s);
// V planes (n x nb pk, block order) from M (K x n, stride ldm) with row q scaled by scale[q]
hipError_t tff_gather_rows(const float* M, int64_t ldm, int64_t n, const float* scale,
                           const TffDev& F, u16* hi, u16* lo, hipStream_t s);
// V plane (cols x nb pk, block order of F) = (codes - zero)^T, exact bf16: the code
// matrix (F.k F.rho rows, cols columns) read down its columns; zero per code row
hipError_t tff_dequant_gather_t(const uint32_t* codes, int bits, const float* zero, int64_t cols,
                                const TffDev& F, u16* V, hipStream_t s);
// out (n x d at stride ldout) = V P^T from block-order planes (Vlo may be NULL); Z, tmp:
// n x d fp32 scratch each
hipError_t tff_rows_synthesis(const u16* Vhi, const u16* Vlo, int64_t n, const TffDev& F,
                              const u16* Fhi, const u16* Flo, float* Z, float* tmp, float* out,
                              int64_t ldout, hipStream_t s);
hipError_t sym_average(float* X, int64_t n, int64_t ld, hipStream_t s);
// true for a stream made by fq_side_stream_create (part of the device, shared with the
// caller's other streams)
bool is_side_stream(hipStream_t s);

// Seeded Haar factor f (tff_seed.hip): out (n x n fp32) from seed; G, V: n x n fp64
// scratch each, ab: 2n fp64
constexpr int64_t TFF_SEED_MAX_N = 1024;
hipError_t tff_seeded_factor(uint64_t seed, int f, int n, double* G, double* V, double* ab,
                             float* out, hipStream_t s);
// Y (n x ldy) = V P^T with V n x ldv (ldv even), R2t from tff_transpose_r2; z: n x d scratch
hipError_t tff_synthesis(const float* V, int64_t ldv, int64_t n, const TffDev& F,
                         const float* R2t, float* z, float* Y, int64_t ldy, hipStream_t s);

// Per-token rounding of U (n x ldu, K columns) to bits-bit integers: Cq (n x ldc bytes;
// perm_cpw 16 or 8: each code word's columns in the byte order of 2- or 4-bit spread code
// words, 0: natural order), delta (n), and when csum is not NULL the row sums of Cq (n).
hipError_t act_quantize(const float* U, int64_t ldu, int64_t n, int64_t K, int bits,
                        int8_t* Cq, int64_t ldc, int perm_cpw, float* delta, int* csum,
                        hipStream_t s);
// V as apply_codes, from rounded activations and codes of `bits` = 2 or 4 bits
// (ldc = (32 / bits) * nwords bytes)
hipError_t apply_codes_i8(const int8_t* Cq, int64_t ldc, const float* delta, const int* csum,
                          int nt, int bits, const uint32_t* codes, int64_t K_out, int64_t nwords,
                          const float* scale, const float* zero, float* V, hipStream_t s);
hipError_t frame_apply(const void* X, int xt, int64_t n, int64_t ldx, int64_t d_in,
                       const uint32_t* codes, int bits, const float* scale, const float* zero,
                       int64_t K_out, int64_t K_in, const float* P_out, int64_t d_out,
                       const float* P_in, float* Y, const ApplyScratch& w, hipStream_t s);

// ---------------------------------------------------------------- fp64 path
struct QuantScratch {
  double* Y;          // K_out x K_in working matrix (pre-rounding values)
  double* A;          // K_in x K_in: reversed damped H~, factored in place (lower)
  double* R;          // K_in x K_in: R' = R diag(R)^-1, R the upper factor (H~_damped = R R^T)
  double* res;        // K_out x block residuals D - D^ of the current block
  uint8_t* codes8;    // K_out x K_in codes
  double* red;        // reduction partials
  double* scal;       // device scalars: [0] mu [1] sigma [2] lo [3] hi [4] lambda
  double* scale64;    // K_out
  double* zero64;     // K_out
  double* inv_rdiag;  // K_in
  double* lslots;     // 2 x 64 x 64: factors of the last two diagonal blocks
  uint8_t* dead;      // K_in
  int* flags;         // [0] not PD, [1] non-finite
};

hipError_t q_stats(const float* D, int64_t rows, int64_t cols, double clip_sigmas,
                   QuantScratch& w, hipStream_t s);
hipError_t q_hdiag_build(const float* Ht, int64_t K, double damp, QuantScratch& w,
                         hipStream_t s);
// Blocked lower Cholesky of A (K x K, in place); Lslots: 2 x 64 x 64 doubles of scratch.
hipError_t q_cholesky(double* A, int64_t K, double* Lslots, int* flags, hipStream_t s);
hipError_t q_reverse_upper(const double* A, int64_t K, double* R, double* inv_rdiag,
                           hipStream_t s);
hipError_t q_clip_grid(const float* D, int64_t rows, int64_t cols, int bits, QuantScratch& w,
                       float* scale, float* zero, hipStream_t s);
hipError_t q_gptq_block(const float* D, int64_t rows, int64_t cols, int i1, int i2, int o1,
                        int cw, int64_t ld_res, int bits, QuantScratch& w, hipStream_t s);
// C[M x N] = beta * C + alpha * A[M x K] * op(B)   (fp64 MFMA; beta is 0 or 1)
//   b_trans: op(B)(k, n) = B[n * ldb + k]  else B[k * ldb + n]
//   lower_only: only tiles with tile_row >= tile_col (for the Cholesky update)
//   tile: 32, 64 or 128 (register-staged kernel with that tile edge; 32 with K <= 128 and
//         not lower_only fetches every K step at launch), or 0: the 128 x 128
//         LDS-ring kernel where its layout rules hold (row-major operands, K % 16 == 0,
//         16-byte aligned A rows), else the 64 kernel.  The ring kernel is the faster one
//         from about 512 of its tiles up (two rounds of two work-groups per CU).
hipError_t dgemm(int64_t M, int64_t N, int64_t K, double alpha, double beta, const double* A,
                 int64_t lda, const double* B, int64_t ldb, bool b_trans, double* C, int64_t ldc,
                 bool lower_only, hipStream_t s, const char* name, int tile);
hipError_t q_pack2(const uint8_t* codes8, int64_t rows, int64_t cols, uint32_t* out,
                   hipStream_t s);
// out[r * ld_out + c] = code[r][c] - zero[r] (bf16) on a rows_out x ld_out plane, zero
// outside rows x cols; ld_out a multiple of 16 (and 16-byte aligned rows).
// 3- and 4-bit codes: floor(32 / bits) per uint32 word (2-bit: q_pack2 / dequant_bf16)
hipError_t q_pack_nbit(const uint8_t* codes8, int64_t rows, int64_t cols, int bits,
                       uint32_t* out, hipStream_t s);
// dequant_bf16 for any of 2, 3, 4 bits
hipError_t dequant_nbit_bf16(const uint32_t* codes, int bits, const float* zero, int64_t rows,
                             int64_t cols, u16* out, int64_t ld_out, int64_t rows_out,
                             hipStream_t s);
hipError_t dequant_bf16(const uint32_t* codes, const float* zero, int64_t rows, int64_t cols,
                        u16* out, int64_t ld_out, int64_t rows_out, hipStream_t s);

// ---------------------------------------------------------------- diagonal Wiener filter
// gain_i = (D_i . E_i) / (scale_i (Q_i . E_i)) (1 where the denominator is 0) with E = Q H~,
// Q the bf16 plane of codes - zero (row stride ldq); scale_out (may alias scale or be
// NULL) = gain * scale.
hipError_t wiener_rows(const float* D, const float* E, const u16* Q, int64_t ldq, int64_t K_out,
                       int64_t K_in, const float* scale, float* gain, float* scale_out,
                       hipStream_t s);

}  // namespace fq
