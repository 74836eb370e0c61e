// fp64 part of the pass on gfx950: statistics and clip, per-row grid, damped Hessian,
// blocked Cholesky, column-sequential 2-bit rounding with error feedback, lazy trailing
// updates (fp64 MFMA), 2-bit packing and the dequantization feeding the synthesis.
//
// Error feedback through the Cholesky factor itself.  OPTQ rounds column j of a row at
//   w_j = D_j - sum_{m<j} E_m U_mj,   E_m = (w_m - q_m) / U_mm,   U^T U = H^{-1} (U upper).
// With H = R R^T (R upper) one has U = R^{-1}, and E U = D - Q gives E = (D - Q) R, so
//   w_j = D_j + (1 / R_jj) sum_{m<j} (D_m - Q_m) R_mj.
// The kernels carry y_j = R_jj w_j, start from y = D diag(R), add (D_m - Q_m) R_mj after
// each rounded column (eagerly inside a block of columns, lazily as one fp64 GEMM for the
// columns right of the block) and read w_j = y_j / R_jj.  This is an exact rewriting of
// OPTQ's update; it needs the Cholesky factor R only, not the inverse factor U.
// R comes from a lower Cholesky M of J H J (J reverses the index order): R = J M J.
#include "fq_internal.h"

namespace fq {

typedef double doublex4 __attribute__((ext_vector_type(4)));

namespace {

int grid_for(int64_t n, int per_block, int cap = 65536) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g > cap) g = cap;
  if (g < 1) g = 1;
  return (int)g;
}

__device__ __forceinline__ double bcast_lane(double v, int src) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)(b & 0xffffffffll), src);
  const int hi = __builtin_amdgcn_readlane((int)(b >> 32), src);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

__device__ __forceinline__ double shfl_d(double v, int src) {
  const long long b = __double_as_longlong(v);
  const int lo = __shfl((int)(b & 0xffffffffll), src, 64);
  const int hi = __shfl((int)(b >> 32), src, 64);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

template <int NTH>
__device__ __forceinline__ double block_sum(double v, double* sh) {
  for (int o = 32; o > 0; o >>= 1) v += shfl_d(v, (threadIdx.x & 63) ^ o);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) sh[w] = v;
  __syncthreads();
  double r = 0.0;
  if (threadIdx.x == 0) {
    for (int i = 0; i < NTH / 64; ++i) r += sh[i];
  }
  __syncthreads();
  return r;  // valid in thread 0
}

// ------------------------------------------------------------------ statistics
// mode 0: sum of x (and finiteness); mode 1: sum of (x - mu)^2.
constexpr int RED_BLOCKS = 1024;

__global__ __launch_bounds__(256) void k_moments(const float* __restrict__ D, int64_t n,
                                                 int mode, const double* __restrict__ scal,
                                                 double* __restrict__ red, int* flags) {
  __shared__ double sh[4];
  const double mu = mode ? scal[0] : 0.0;
  double acc = 0.0;
  bool bad = false;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += (int64_t)RED_BLOCKS * 256) {
    const double x = (double)D[e];
    if (mode == 0) {
      bad |= !isfinite(x);
      acc += x;
    } else {
      const double d = x - mu;
      acc += d * d;
    }
  }
  if (bad) flags[1] = 1;
  const double s = block_sum<256>(acc, sh);
  if (threadIdx.x == 0) red[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_moments_final(const double* __restrict__ red, int64_t n,
                                                       int mode, double clip_sigmas,
                                                       double* __restrict__ scal) {
  __shared__ double sh[4];
  double acc = 0.0;
  for (int i = threadIdx.x; i < RED_BLOCKS; i += 256) acc += red[i];
  const double s = block_sum<256>(acc, sh);
  if (threadIdx.x == 0) {
    if (mode == 0) {
      scal[0] = s / (double)n;
    } else {
      const double sigma = n > 1 ? sqrt(s / (double)(n - 1)) : 0.0;
      scal[1] = sigma;
      scal[2] = scal[0] - clip_sigmas * sigma;
      scal[3] = scal[0] + clip_sigmas * sigma;
    }
  }
}

// ------------------------------------------------------------------ damped, reversed H~
// Dead columns (zero diagonal) and lambda = damp * mean(diag), after the dead fix.
__global__ __launch_bounds__(256) void k_hdiag(const float* __restrict__ Ht, int64_t K,
                                               double damp, uint8_t* __restrict__ dead,
                                               double* __restrict__ scal) {
  __shared__ double sh[4];
  double acc = 0.0;
  for (int64_t j = threadIdx.x; j < K; j += 256) {
    const double d = (double)Ht[j * K + j];
    const bool z = (d == 0.0);
    dead[j] = z ? 1 : 0;
    acc += z ? 1.0 : d;
  }
  const double s = block_sum<256>(acc, sh);
  if (threadIdx.x == 0) scal[4] = damp * s / (double)K;
}

// A[i][j] = Hd[K-1-i][K-1-j] for j <= i (lower), Hd the damped H~; zero above.
__global__ __launch_bounds__(256) void k_build_rev(const float* __restrict__ Ht, int64_t K,
                                                   const uint8_t* __restrict__ dead,
                                                   const double* __restrict__ scal,
                                                   double* __restrict__ A, int* flags) {
  const double lam = scal[4];
  const int64_t total = K * K;
  bool bad = false;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t i = e / K, j = e - i * K;
    double v = 0.0;
    if (j <= i) {
      const int64_t si = K - 1 - i, sj = K - 1 - j;
      v = (double)Ht[si * K + sj];
      bad |= !isfinite(v);
      if (i == j) v = (dead[si] ? 1.0 : v) + lam;
    }
    A[e] = v;
  }
  if (bad) flags[1] = 1;
}

// ------------------------------------------------------------------ Cholesky
// Factor the kb x kb diagonal block at (k0, k0) in place (lower), one wave64: lane r
// holds row r of the block (padded with identity rows beyond kb).
__global__ __launch_bounds__(64) void k_potrf64(double* __restrict__ A, int64_t lda, int64_t k0,
                                                int kb, int* flags) {
  const int r = threadIdx.x;
  double a[64];
#pragma unroll
  for (int c = 0; c < 64; ++c) {
    double v = (r == c) ? 1.0 : 0.0;
    if (r < kb && c < kb && c <= r) v = A[(k0 + r) * lda + k0 + c];
    a[c] = v;
  }
  bool notpd = false;
#pragma unroll
  for (int c = 0; c < 64; ++c) {
    double piv = bcast_lane(a[c], c);
    if (!(piv > 0.0)) {
      notpd = true;
      piv = 1.0;
    }
    const double d = sqrt(piv);
    const double inv = 1.0 / d;
    if (r > c) a[c] *= inv;
    else if (r == c) a[c] = d;
    const double lc = a[c];
#pragma unroll
    for (int cc = c + 1; cc < 64; ++cc) {
      const double l2 = bcast_lane(lc, cc);
      if (r >= cc) a[cc] -= lc * l2;
    }
  }
  if (notpd && r == 0) flags[0] = 1;
  if (r < kb) {
#pragma unroll
    for (int c = 0; c < 64; ++c)
      if (c <= r && c < kb) A[(k0 + r) * lda + k0 + c] = a[c];
  }
}

// Panel below the diagonal block: rows i in [k0+kb, K), X = A[i, k0:k0+kb] L_kk^{-T}
// (forward substitution, one row per thread; the rows and L_kk live in LDS).
__global__ __launch_bounds__(64) void k_trsm64(double* __restrict__ A, int64_t lda, int64_t K,
                                               int64_t k0, int kb) {
  __shared__ double L[64][65];
  __shared__ double X[64][65];
  const int t = threadIdx.x;
  const int64_t i0 = k0 + kb + (int64_t)blockIdx.x * 64;
  for (int e = t; e < 64 * 64; e += 64) {
    const int r = e >> 6, c = e & 63;
    L[r][c] = (r < kb && c < kb && c <= r) ? A[(k0 + r) * lda + k0 + c] : (r == c ? 1.0 : 0.0);
    const int64_t gi = i0 + r;
    X[r][c] = (gi < K && c < kb) ? A[gi * lda + k0 + c] : 0.0;
  }
  __syncthreads();
  for (int c = 0; c < kb; ++c) {
    double v = X[t][c];
    for (int m = 0; m < c; ++m) v -= X[t][m] * L[c][m];
    X[t][c] = v / L[c][c];
  }
  __syncthreads();
  for (int e = t; e < 64 * 64; e += 64) {
    const int r = e >> 6, c = e & 63;
    const int64_t gi = i0 + r;
    if (gi < K && c < kb) A[gi * lda + k0 + c] = X[r][c];
  }
}

// R[i][j] = M[K-1-i][K-1-j] (upper), rdiag / inv_rdiag.
__global__ __launch_bounds__(256) void k_reverse_upper(const double* __restrict__ M, int64_t K,
                                                       double* __restrict__ R,
                                                       double* __restrict__ rdiag,
                                                       double* __restrict__ inv_rdiag) {
  const int64_t total = K * K;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t i = e / K, j = e - i * K;
    double v = 0.0;
    if (i <= j) v = M[(K - 1 - i) * K + (K - 1 - j)];
    R[e] = v;
    if (i == j) {
      rdiag[i] = v;
      inv_rdiag[i] = 1.0 / v;
    }
  }
}

// ------------------------------------------------------------------ clip + grid
// One work-group per row: clip at [lo, hi], per-row min/max grid, Y = clipped D * R_jj
// (dead columns zero).
__global__ __launch_bounds__(256) void k_clip_grid(const float* __restrict__ D, int64_t cols,
                                                   int maxq, const double* __restrict__ scal,
                                                   const uint8_t* __restrict__ dead,
                                                   const double* __restrict__ rdiag,
                                                   double* __restrict__ Y, float* __restrict__ scale,
                                                   float* __restrict__ zero,
                                                   double* __restrict__ scale64,
                                                   double* __restrict__ zero64) {
  __shared__ double smin[4], smax[4];
  const int64_t r = blockIdx.x;
  const double lo_b = scal[2], hi_b = scal[3];
  const float* row = D + r * cols;
  double mn = 0.0, mx = 0.0;   // min(0, .), max(0, .)
  for (int64_t j = threadIdx.x; j < cols; j += 256) {
    const double x = fmin(fmax((double)row[j], lo_b), hi_b);
    mn = fmin(mn, x);
    mx = fmax(mx, x);
  }
  for (int o = 32; o > 0; o >>= 1) {
    mn = fmin(mn, shfl_d(mn, (threadIdx.x & 63) ^ o));
    mx = fmax(mx, shfl_d(mx, (threadIdx.x & 63) ^ o));
  }
  if ((threadIdx.x & 63) == 0) {
    smin[threadIdx.x >> 6] = mn;
    smax[threadIdx.x >> 6] = mx;
  }
  __syncthreads();
  mn = fmin(fmin(smin[0], smin[1]), fmin(smin[2], smin[3]));
  mx = fmax(fmax(smax[0], smax[1]), fmax(smax[2], smax[3]));
  if (mn == 0.0 && mx == 0.0) {
    mn = -1.0;
    mx = 1.0;
  }
  const float s32 = (float)((mx - mn) / (double)maxq);
  const double s = (double)s32;
  const double z = rint(-mn / s);
  if (threadIdx.x == 0) {
    scale[r] = s32;
    zero[r] = (float)z;
    scale64[r] = s;
    zero64[r] = z;
  }
  double* yrow = Y + r * cols;
  for (int64_t j = threadIdx.x; j < cols; j += 256) {
    const double x = dead[j] ? 0.0 : fmin(fmax((double)row[j], lo_b), hi_b);
    yrow[j] = x * rdiag[j];
  }
}

// ------------------------------------------------------------------ rounding block
// Columns [i1, i2) (at most 128) of every row.  512 threads = 8 waves; a wave is four
// groups of 16 lanes; a group owns 2 rows and lane g of the group holds columns
// 8g .. 8g+7 of the block for both rows.  Column j is decided by its owner lane, its
// residual D_j - D^_j is broadcast to the group, and every lane folds it into its own
// columns with the R row from LDS.
constexpr int GB = 128;
constexpr int GTH = 512;
constexpr int GROWS = GTH / 16 * 2;   // 64 rows per work-group

__global__ __launch_bounds__(GTH) void k_gptq_block(
    const float* __restrict__ D, int64_t rows, int64_t cols, int i1, int b, int64_t res_col0,
    int64_t ld_res, int maxq, const double* __restrict__ scal, const uint8_t* __restrict__ dead,
    const double* __restrict__ R, const double* __restrict__ inv_rdiag,
    const double* __restrict__ scale64, const double* __restrict__ zero64,
    const double* __restrict__ Y, uint8_t* __restrict__ codes8, double* __restrict__ res) {
  __shared__ double Rs[GB * GB];
  for (int e = threadIdx.x; e < GB * GB; e += GTH) {
    const int rr = e / GB, cc = e % GB;
    Rs[e] = (rr < b && cc < b) ? R[(int64_t)(i1 + rr) * cols + i1 + cc] : 0.0;
  }
  __shared__ double ird[GB];
  if (threadIdx.x < GB) ird[threadIdx.x] = threadIdx.x < b ? inv_rdiag[i1 + threadIdx.x] : 0.0;
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int g = lane & 15;                         // position inside the group
  const int grp = (threadIdx.x >> 4);              // group index in the work-group
  const int gbase = lane & ~15;                    // first lane of the group
  const int64_t r0 = (int64_t)blockIdx.x * GROWS + grp * 2;
  const double lo_b = scal[2], hi_b = scal[3];

  double y[2][8], d0[2][8], rr_[2][8];
  uint8_t q8[2][8];
  double s[2], is[2], z[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int64_t r = r0 + k;
    const bool ok = r < rows;
    s[k] = ok ? scale64[r] : 1.0;
    is[k] = 1.0 / s[k];
    z[k] = ok ? zero64[r] : 0.0;
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
      const int c = g * 8 + cc;
      const bool in = ok && c < b;
      y[k][cc] = in ? Y[r * cols + i1 + c] : 0.0;
      double x = 0.0;
      if (in && !dead[i1 + c]) x = fmin(fmax((double)D[r * cols + i1 + c], lo_b), hi_b);
      d0[k][cc] = x;
      rr_[k][cc] = 0.0;
      q8[k][cc] = 0;
    }
  }

  for (int o = 0; o < 16; ++o) {
    if (o * 8 >= b) break;
#pragma unroll
    for (int jj = 0; jj < 8; ++jj) {
      const int j = o * 8 + jj;
      if (j >= b) break;
      double res_own[2] = {0.0, 0.0};
      if (g == o) {
        const double ir = ird[j];
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const double w = y[k][jj] * ir;
          const double t = w * is[k];
          const double q = fmin(fmax(rint(t) + z[k], 0.0), (double)maxq);
          const double dq = s[k] * (q - z[k]);
          const double e = d0[k][jj] - dq;
          res_own[k] = e;
          rr_[k][jj] = e;
          q8[k][jj] = (uint8_t)q;
        }
      }
      const double e0 = shfl_d(res_own[0], gbase + o);
      const double e1 = shfl_d(res_own[1], gbase + o);
      const double* Rrow = Rs + j * GB + g * 8;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        const double rv = Rrow[cc];
        y[0][cc] += e0 * rv;
        y[1][cc] += e1 * rv;
      }
    }
  }

#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int64_t r = r0 + k;
    if (r >= rows) continue;
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
      const int c = g * 8 + cc;
      if (c < b) {
        codes8[r * cols + i1 + c] = q8[k][cc];
        res[r * ld_res + res_col0 + c] = rr_[k][cc];
      }
    }
  }
}

// ------------------------------------------------------------------ fp64 MFMA GEMM
// C[M x N] += alpha * A[M x K] * op(B).  Tile 64 x 64, K step 16, 256 threads (2 x 2
// waves of 32 x 32, each 2 x 2 v_mfma_f64_16x16x4 blocks).
constexpr int DT = 64, DK = 16;

__global__ __launch_bounds__(256) void k_dgemm(int64_t M, int64_t N, int64_t K, double alpha,
                                               const double* __restrict__ A, int64_t lda,
                                               const double* __restrict__ B, int64_t ldb,
                                               int b_trans, double* __restrict__ C, int64_t ldc,
                                               int lower_only, int tiles_n) {
  __shared__ double As[DT][DK + 1];
  __shared__ double Bs[DK][DT + 1];
  int tm, tn;
  if (lower_only) {
    int t = blockIdx.x, row = 0;
    while (t > row) { t -= row + 1; ++row; }
    tm = row;
    tn = t;
  } else {
    tm = blockIdx.x / tiles_n;
    tn = blockIdx.x - tm * tiles_n;
  }
  const int64_t m0 = (int64_t)tm * DT, n0 = (int64_t)tn * DT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  doublex4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = (doublex4){0.0, 0.0, 0.0, 0.0};

  for (int64_t k0 = 0; k0 < K; k0 += DK) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = tid + q * 256;
      {  // A tile: 64 rows x 16 k, row-major
        const int r = e >> 4, c = e & 15;
        const int64_t gm = m0 + r, gk = k0 + c;
        As[r][c] = (gm < M && gk < K) ? A[gm * lda + gk] : 0.0;
      }
      if (b_trans) {  // op(B)(k, n) = B[n * ldb + k]
        const int n = e >> 4, c = e & 15;
        const int64_t gn = n0 + n, gk = k0 + c;
        Bs[c][n] = (gn < N && gk < K) ? B[gn * ldb + gk] : 0.0;
      } else {        // B[k * ldb + n]
        const int c = e >> 6, n = e & 63;
        const int64_t gn = n0 + n, gk = k0 + c;
        Bs[c][n] = (gn < N && gk < K) ? B[gk * ldb + gn] : 0.0;
      }
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < DK; kk += 4) {
      double af[2], bfv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = As[wm * 32 + i * 16 + (lane & 15)][kk + (lane >> 4)];
#pragma unroll
      for (int j = 0; j < 2; ++j) bfv[j] = Bs[kk + (lane >> 4)][wn * 32 + j * 16 + (lane & 15)];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(af[i], bfv[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  // 16x16 f64 accumulator layout: value v of lane l is row l/16 + 4*v, column l%16.
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int64_t row = m0 + wm * 32 + i * 16 + (lane >> 4) + 4 * v;
        const int64_t col = n0 + wn * 32 + j * 16 + (lane & 15);
        if (row < M && col < N) C[row * ldc + col] += alpha * acc[i][j][v];
      }
}

// ------------------------------------------------------------------ pack / dequant
__global__ __launch_bounds__(256) void k_pack2(const uint8_t* __restrict__ c8, int64_t rows,
                                               int64_t cols, uint32_t* __restrict__ out) {
  const int64_t nw = (cols + 15) / 16;
  const int64_t total = rows * nw;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / nw, w = e - r * nw;
    const int64_t c0 = w * 16;
    const uint8_t* src = c8 + r * cols + c0;
    uint32_t word = 0;
    if (c0 + 16 <= cols && ((reinterpret_cast<uintptr_t>(src) & 15) == 0)) {
      const uint4 v = *reinterpret_cast<const uint4*>(src);
      const uint32_t d[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int bt = 0; bt < 4; ++bt) word |= ((d[q] >> (8 * bt)) & 3u) << (2 * (q * 4 + bt));
    } else {
      for (int k = 0; k < 16; ++k)
        if (c0 + k < cols) word |= ((uint32_t)src[k] & 3u) << (2 * k);
    }
    out[e] = word;
  }
}

__global__ __launch_bounds__(256) void k_dequant(const uint32_t* __restrict__ codes,
                                                 const float* __restrict__ zero, int64_t rows,
                                                 int64_t cols, u16* __restrict__ out,
                                                 int64_t ld_out) {
  const int64_t nw = (cols + 15) / 16;
  const int64_t total = rows * nw;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / nw, w = e - r * nw;
    const uint32_t word = codes[e];
    const float z = zero[r];
    u16* dst = out + r * ld_out + w * 16;
    uint32_t h[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const float v = (float)((word >> (2 * k)) & 3u) - z;   // small integer, exact in bf16
      h[k] = __float_as_uint(v) >> 16;
    }
    if (w * 16 + 16 <= cols && ((reinterpret_cast<uintptr_t>(dst) & 15) == 0)) {
      *reinterpret_cast<uint4*>(dst) = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16),
                                                  h[4] | (h[5] << 16), h[6] | (h[7] << 16));
      *reinterpret_cast<uint4*>(dst + 8) = make_uint4(h[8] | (h[9] << 16), h[10] | (h[11] << 16),
                                                      h[12] | (h[13] << 16), h[14] | (h[15] << 16));
    } else {
      for (int k = 0; k < 16; ++k)
        if (w * 16 + k < cols) dst[k] = (u16)h[k];
    }
  }
}

}  // namespace

// ====================================================================== launchers
hipError_t q_stats(const float* D, int64_t rows, int64_t cols, double clip_sigmas,
                   QuantScratch& w, hipStream_t s) {
  const int64_t n = rows * cols;
  prof_begin(s, "q_moments");
  hipLaunchKernelGGL(k_moments, dim3(RED_BLOCKS), dim3(256), 0, s, D, n, 0, w.scal, w.red, w.flags);
  hipLaunchKernelGGL(k_moments_final, dim3(1), dim3(256), 0, s, w.red, n, 0, clip_sigmas, w.scal);
  hipLaunchKernelGGL(k_moments, dim3(RED_BLOCKS), dim3(256), 0, s, D, n, 1, w.scal, w.red, w.flags);
  hipLaunchKernelGGL(k_moments_final, dim3(1), dim3(256), 0, s, w.red, n, 1, clip_sigmas, w.scal);
  prof_end(s);
  return last_launch_error();
}

hipError_t q_hdiag_build(const float* Ht, int64_t K, double damp, QuantScratch& w,
                         hipStream_t s) {
  prof_begin(s, "q_hbuild");
  hipLaunchKernelGGL(k_hdiag, dim3(1), dim3(256), 0, s, Ht, K, damp, w.dead, w.scal);
  hipLaunchKernelGGL(k_build_rev, dim3(grid_for(K * K, 256)), dim3(256), 0, s, Ht, K, w.dead,
                     w.scal, w.A, w.flags);
  prof_end(s);
  return last_launch_error();
}

hipError_t q_cholesky(double* A, int64_t K, int* flags, hipStream_t s) {
  for (int64_t k0 = 0; k0 < K; k0 += 64) {
    const int kb = (int)((K - k0) < 64 ? (K - k0) : 64);
    prof_begin(s, "chol_potrf");
    hipLaunchKernelGGL(k_potrf64, dim3(1), dim3(64), 0, s, A, K, k0, kb, flags);
    prof_end(s);
    const int64_t rest = K - k0 - kb;
    if (rest > 0) {
      prof_begin(s, "chol_trsm");
      hipLaunchKernelGGL(k_trsm64, dim3(grid_for(rest, 64, 1 << 30)), dim3(64), 0, s, A, K, K, k0, kb);
      prof_end(s);
      const double* P = A + (k0 + kb) * K + k0;
      hipError_t e = dgemm(rest, rest, kb, -1.0, P, K, P, K, true, A + (k0 + kb) * K + (k0 + kb),
                           K, true, s);
      if (e != hipSuccess) return e;
    }
  }
  return last_launch_error();
}

hipError_t q_reverse_upper(const double* A, int64_t K, double* R, double* inv_rdiag,
                           hipStream_t s) {
  // rdiag is stored right after inv_rdiag (2 K doubles)
  prof_begin(s, "q_reverse");
  hipLaunchKernelGGL(k_reverse_upper, dim3(grid_for(K * K, 256)), dim3(256), 0, s, A, K, R,
                     inv_rdiag + K, inv_rdiag);
  prof_end(s);
  return last_launch_error();
}

hipError_t q_clip_grid(const float* D, int64_t rows, int64_t cols, int bits, QuantScratch& w,
                       float* scale, float* zero, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  prof_begin(s, "q_clip_grid");
  hipLaunchKernelGGL(k_clip_grid, dim3(rows), dim3(256), 0, s, D, cols, (1 << bits) - 1, w.scal,
                     w.dead, w.inv_rdiag + cols, w.Y, scale, zero, w.scale64, w.zero64);
  prof_end(s);
  return last_launch_error();
}

hipError_t q_gptq_block(const float* D, int64_t rows, int64_t cols, int i1, int i2, int o1,
                        int64_t ld_res, int bits, QuantScratch& w, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  prof_begin(s, "gptq_block");
  hipLaunchKernelGGL(k_gptq_block, dim3(grid_for(rows, GROWS, 1 << 30)), dim3(GTH), 0, s, D, rows,
                     cols, i1, i2 - i1, (int64_t)(i1 - o1), ld_res, (1 << bits) - 1, w.scal,
                     w.dead, w.R, w.inv_rdiag, w.scale64, w.zero64, w.Y, w.codes8, w.res);
  prof_end(s);
  return last_launch_error();
}

hipError_t dgemm(int64_t M, int64_t N, int64_t K, double alpha, const double* A, int64_t lda,
                 const double* B, int64_t ldb, bool b_trans, double* C, int64_t ldc,
                 bool lower_only, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return hipSuccess;
  const int tiles_m = (int)((M + DT - 1) / DT), tiles_n = (int)((N + DT - 1) / DT);
  const int64_t grid = lower_only ? (int64_t)tiles_m * (tiles_m + 1) / 2 : (int64_t)tiles_m * tiles_n;
  prof_begin(s, lower_only ? "chol_syrk" : "gptq_update");
  hipLaunchKernelGGL(k_dgemm, dim3((unsigned)grid), dim3(256), 0, s, M, N, K, alpha, A, lda, B,
                     ldb, (int)b_trans, C, ldc, (int)lower_only, tiles_n);
  prof_end(s);
  return last_launch_error();
}

hipError_t q_pack2(const uint8_t* codes8, int64_t rows, int64_t cols, uint32_t* out,
                   hipStream_t s) {
  const int64_t nw = rows * ((cols + 15) / 16);
  if (nw <= 0) return hipSuccess;
  prof_begin(s, "pack2");
  hipLaunchKernelGGL(k_pack2, dim3(grid_for(nw, 256)), dim3(256), 0, s, codes8, rows, cols, out);
  prof_end(s);
  return last_launch_error();
}

hipError_t dequant_bf16(const uint32_t* codes, const float* zero, int64_t rows, int64_t cols,
                        u16* out, int64_t ld_out, hipStream_t s) {
  const int64_t nw = rows * ((cols + 15) / 16);
  if (nw <= 0) return hipSuccess;
  prof_begin(s, "dequant");
  hipLaunchKernelGGL(k_dequant, dim3(grid_for(nw, 256)), dim3(256), 0, s, codes, zero, rows, cols,
                     out, ld_out);
  prof_end(s);
  return last_launch_error();
}

}  // namespace fq
