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

#include <algorithm>
#include <mutex>

namespace fq {


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
  auto add = [&](float xf) {
    const double x = (double)xf;
    if (mode == 0) {
      bad |= !isfinite(x);
      acc += x;
    } else {
      const double d = x - mu;
      acc += d * d;
    }
  };
  const int64_t stride = (int64_t)RED_BLOCKS * 256;
  // 16-byte loads over the aligned bulk, then the remainder one by one
  const int64_t n4 = ((reinterpret_cast<uintptr_t>(D) & 15) == 0) ? n / 4 : 0;
  const float4* D4 = reinterpret_cast<const float4*>(D);
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < n4; e += stride) {
    const float4 v = D4[e];
    add(v.x); add(v.y); add(v.z); add(v.w);
  }
  for (int64_t e = 4 * n4 + (int64_t)blockIdx.x * 256 + threadIdx.x; e < n; e += stride)
    add(D[e]);
  if (bad) flags[2] = 1;                 // D non-finite (flags[1]: H~ non-finite)
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
// 1 / sqrt(x) to full double precision: hardware estimate plus two Newton steps.
__device__ __forceinline__ double rsqrt_d(double x) {
  double y = __builtin_amdgcn_rsq(x);
  double h = 0.5 * x;
  y = y * fma(-h * y, y, 1.5);
  y = y * fma(-h * y, y, 1.5);
  return y;
}

// ---- 64 x 64 diagonal-block factorization and the inverse of the factor, L_kk and
// Z = L_kk^-1, by columns: the pivot of column C comes from its row's lane by readlane,
// the column is scaled and published through LDS, and every later column receives the
// rank-1 update (a[k] -= L_rC L_kC).  Row C of Z is finished with column C (z_C /= L_CC)
// and published beside it; later rows receive z_k -= L_kC z_C.

// pin the listed slots: without it the compiler sinks updates into later columns and keeps
// every broadcast value alive
template <int LO, int HI, int N>
__device__ __forceinline__ void pin_slots(double (&a)[N]) {
  if constexpr (LO < HI) {
    if constexpr (HI - LO >= 4) {
      asm volatile("" : "+v"(a[LO]), "+v"(a[LO + 1]), "+v"(a[LO + 2]), "+v"(a[LO + 3]));
      pin_slots<LO + 4, HI>(a);
    } else {
      asm volatile("" : "+v"(a[LO]));
      pin_slots<LO + 1, HI>(a);
    }
  }
}

// The columns are spread over the four waves of the work-group: wave W
// holds columns [16 W, 16 W + 16) of the block (lane r = row r) and rows [16 W, 16 W + 16)
// of Z = L^{-1} (lane j = column j).  Column C is published by its owner wave (the
// scaled column of L, row C of Z scaled by 1 / L_CC) before the barrier of step C; after
// it every wave applies column C to its own columns of the block and its own rows of Z.
// The owner of column C + 1 applies column C to that column first and publishes it, then
// the rest.  Each entry receives its updates in column order.
template <int W, int C>
__device__ __forceinline__ void f4_publish(double (&a)[16], double (&z)[16], int r,
                                           double* colC, double* zrowC, double* invd,
                                           bool& notpd) {
  constexpr int S = C - 16 * W;
  double piv = bcast_lane(a[S], C);
  if (!(piv > 0.0)) {
    notpd = true;
    piv = 1.0;
  }
  const double inv = rsqrt_d(piv);
  a[S] = (r == C) ? piv * inv : a[S] * inv;
  colC[r] = a[S];
  z[S] *= inv;
  zrowC[r] = z[S];
  if (r == C) invd[C] = inv;
}

template <int W, int C>
__device__ __forceinline__ void f4_step(double (&a)[16], double (&z)[16], int r,
                                        double (*col)[64], double (*zrow)[64], double* invd,
                                        bool& notpd) {
  constexpr int LO = 16 * W, HI = LO + 16;
  constexpr int K0 = (C + 1 > LO) ? C + 1 : LO;
  if constexpr (K0 < HI) {
    constexpr int G = K0 & ~1;
    constexpr int NV = (HI - G) / 2;
    const double lrc = col[C & 1][r];
    const double zc = zrow[C & 1][r];
    double2 v[NV];
    const double2* cp = reinterpret_cast<const double2*>(col[C & 1] + G);
#pragma unroll
    for (int q = 0; q < NV; ++q) v[q] = cp[q];
    constexpr bool NEXT = (C + 1 < 64) && ((C + 1) / 16 == W);
    if constexpr (NEXT) {
      constexpr int k = C + 1;
      const double lk = ((k - G) & 1) ? v[(k - G) >> 1].y : v[(k - G) >> 1].x;
      a[k - LO] -= lrc * lk;
      z[k - LO] -= zc * lk;
      f4_publish<W, C + 1>(a, z, r, col[(C + 1) & 1], zrow[(C + 1) & 1], invd, notpd);
    }
#pragma unroll
    for (int k = G; k < HI; ++k) {
      if (k > C + (NEXT ? 1 : 0)) {
        const double lk = ((k - G) & 1) ? v[(k - G) >> 1].y : v[(k - G) >> 1].x;
        a[k - LO] -= lrc * lk;
        z[k - LO] -= zc * lk;
      }
    }
    pin_slots<0, 16>(a);
    pin_slots<0, 16>(z);
  }
  if constexpr (C + 1 < 64) {
    __syncthreads();
    f4_step<W, C + 1>(a, z, r, col, zrow, invd, notpd);
  }
}

// Dg: the block (lower part, identity beyond kb); writes L (zero above the diagonal) back
// to Dg and Z to Zs[k][c]; true when a pivot was not positive
template <int W>
__device__ __forceinline__ bool f4_run(double (*Dg)[65], double (*Zs)[65], int r,
                                       double (*col)[64], double (*zrow)[64], double* invd) {
  constexpr int LO = 16 * W;
  double a[16], z[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    a[i] = Dg[r][LO + i];
    z[i] = (LO + i == r) ? 1.0 : 0.0;
  }
  bool notpd = false;
  if constexpr (W == 0) f4_publish<0, 0>(a, z, r, col[0], zrow[0], invd, notpd);
  __syncthreads();
  f4_step<W, 0>(a, z, r, col, zrow, invd, notpd);
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    Dg[r][LO + i] = (LO + i <= r) ? a[i] : 0.0;
    Zs[LO + i][r] = z[i];
  }
  return notpd;
}

// ---- one block column of the factorization in one launch (left-looking inside a panel).
// Block column [k0, k0 + kb) (kb <= 64) of the panel that starts at column j0 <= k0, every
// update from earlier panels already applied.  Work-group 0 owns the diagonal block's rows;
// the rows below, in slabs of 64 from k0 + kb, are dealt to work-groups 1 .. gridDim.x - 1
// (slab q to work-group 1 + q mod (gridDim.x - 1)).  Each work-group of 4 waves:
//  1. brings the diagonal block up to date with the panel's earlier columns [j0, k0)
//     (left-looking, fp64 MFMA, a 32 x 32 quadrant per wave):  B -= L[k0:, j0:k0] L[k0:, j0:k0]^T
//  2. factors it and forms its inverse, the columns spread over the four waves (one row
//     per lane), redundantly in every work-group, so that no work-group waits for another;
//  3. work-group 0 stores L_kk to the slot Lout (every work-group reads the diagonal block
//     of A, so it must stay unchanged during this launch) and moves the previous block's
//     factor from its slot Lprev into A (rows this launch does not read); every other
//     work-group, for each of its slabs, applies the same left-looking update to the slab's
//     rows of the block column and stores X = B L_kk^-T (MFMA).
// All reads are of columns finished by earlier launches or of the block column before it
// is written, and every work-group writes only its own rows of A: no ordering between
// work-groups is needed.
constexpr int CB = 64, CBP = 65;     // block edge, LDS row pitch (conflict-free fragments)

// acc (a 32 x 32 quadrant of a 64 x 64 product per wave) = sum over k in [j0, k0) of
// L[r0 + i][k] L[d0 + j][k] for the rows r0 .. r0 + nr and d0 .. d0 + nd (zero beyond).
// k0 - j0 is a multiple of 16.  The loads of up to four chunks of 16 k are issued
// together, so the memory latency is paid once per four chunks rather than per chunk.
__device__ __forceinline__ void chol_left_update(const double* __restrict__ A, int64_t lda,
                                                 int64_t j0, int64_t k0, int64_t r0, int nr,
                                                 int64_t d0, int nd, double (*Ls)[CB + 8],
                                                 double (*Ld)[CB + 8], double (&acc)[4][4],
                                                 int tid, int arow, int bcol, int kq) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  // thread t stages row t / 4, 4 consecutive k, of both operands (k-major)
  const int r = tid >> 2, kq4 = (tid & 3) * 4;
  const int64_t rd = d0 + min(r, nd - 1), rr = r0 + min(r, nr - 1);
  const int nch = (int)((k0 - j0) / 16);
  for (int g0 = 0; g0 < nch; g0 += 4) {
    double vd[4][4], vs[4][4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (g0 + q < nch) {
        const int64_t kk0 = j0 + 16 * (g0 + q);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          vd[q][c] = (r < nd) ? A[rd * lda + kk0 + kq4 + c] : 0.0;
          vs[q][c] = (r < nr) ? A[rr * lda + kk0 + kq4 + c] : 0.0;
        }
      }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (g0 + q >= nch) break;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        Ld[kq4 + c][r] = vd[q][c];
        Ls[kq4 + c][r] = vs[q][c];
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < 16; kk += 4) {
        double af[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = Ls[kk + kq][arow + 8 * i];
#pragma unroll
        for (int j = 0; j < 4; ++j) bf[j] = Ld[kk + kq][bcol + 8 * j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f64_4x4x4f64(af[i], bf[j], acc[i][j], 0, 0, 0);
      }
      __syncthreads();
    }
  }
}

// chol_left_update for two row sets sharing the second operand: accD = sum L[d][k] L[d][k]
// (the diagonal block's rows d0 .. d0 + nd) and accS = sum L[s][k] L[d][k] (a slab's rows
// r0 .. r0 + nr; nr = 0: accS stays 0), one pass over the columns [j0, k0).
__device__ __forceinline__ void chol_left_update2(const double* __restrict__ A, int64_t lda,
                                                  int64_t j0, int64_t k0, int64_t r0, int nr,
                                                  int64_t d0, int nd, double (*Ls)[CB + 8],
                                                  double (*Ld)[CB + 8], double (&accD)[4][4],
                                                  double (&accS)[4][4], int tid, int arow,
                                                  int bcol, int kq) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      accD[i][j] = 0.0;
      accS[i][j] = 0.0;
    }
  const int r = tid >> 2, kq4 = (tid & 3) * 4;
  // every address in range, also for an empty slab (nr = 0: the diagonal rows)
  const int64_t rd = d0 + min(r, nd - 1), rr = nr > 0 ? r0 + min(r, nr - 1) : rd;
  const int nch = (int)((k0 - j0) / 16);
  for (int g0 = 0; g0 < nch; g0 += 4) {
    double vd[4][4], vs[4][4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (g0 + q < nch) {
        const int64_t kk0 = j0 + 16 * (g0 + q);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          vd[q][c] = (r < nd) ? A[rd * lda + kk0 + kq4 + c] : 0.0;
          vs[q][c] = (r < nr) ? A[rr * lda + kk0 + kq4 + c] : 0.0;
        }
      }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (g0 + q >= nch) break;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        Ld[kq4 + c][r] = vd[q][c];
        Ls[kq4 + c][r] = vs[q][c];
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < 16; kk += 4) {
        double ad[4], as[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          ad[i] = Ld[kk + kq][arow + 8 * i];
          as[i] = Ls[kk + kq][arow + 8 * i];
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) bf[j] = Ld[kk + kq][bcol + 8 * j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            accD[i][j] = __builtin_amdgcn_mfma_f64_4x4x4f64(ad[i], bf[j], accD[i][j], 0, 0, 0);
            accS[i][j] = __builtin_amdgcn_mfma_f64_4x4x4f64(as[i], bf[j], accS[i][j], 0, 0, 0);
          }
      }
      __syncthreads();
    }
  }
}

__global__ __launch_bounds__(256) void k_chol_block(double* __restrict__ A, int64_t lda, int64_t K,
                                                    int64_t j0, int64_t k0, int kb,
                                                    double* __restrict__ Lout,
                                                    const double* __restrict__ Lprev,
                                                    int64_t kp0, int kpb,
                                                    int* __restrict__ flags) {
  __shared__ double Dg[CB][CBP];                       // diagonal block, then L_kk
  __shared__ double Sg[CB][CBP];                       // a slab's rows of the block column
  __shared__ double Zs[CB][CBP];                       // L_kk^-1 (Zs[k][c] = (L^-1)[k][c])
  __shared__ double Ls[16][CB + 8], Ld[16][CB + 8];    // update staging, k-major
  __shared__ __attribute__((aligned(16))) double col[2][64];     // broadcast column of L
  __shared__ __attribute__((aligned(16))) double zrow[2][64];    // broadcast row of L^-1
  __shared__ double invd[64];                                    // 1 / L_jj
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int w = blockIdx.x;
  const int wm = wave >> 1, wn = wave & 1;
  const int blk = (lane >> 2) & 3, bi = blk >> 1, bj = blk & 1, q4 = lane & 3, kq = lane >> 4;
  const int arow = wm * 32 + 4 * bi + q4;
  const int bcol = wn * 32 + 4 * bj + q4;
  const int r0 = wm * 32 + 4 * bi + kq, c0 = wn * 32 + 4 * bj + q4;   // accumulator origin
  double acc[4][4];
  const int64_t below = K - k0 - kb;
  const int64_t nslab = (below + CB - 1) / CB;
  // the first slab of this work-group (work-groups 1 ..): brought up to date in the same
  // pass as the diagonal block, its values fetched with the block's, before the factor
  const int64_t rs1 = k0 + kb + CB * (int64_t)(w - 1);
  const int nr1 = (w >= 1 && w - 1 < nslab) ? (int)min<int64_t>(CB, K - rs1) : 0;
  // work-group 0: the previous block's factor, fetched now and stored at the end
  double lp[CB * CB / 256];
  if (w == 0 && Lprev) {
#pragma unroll
    for (int q = 0; q < CB * CB / 256; ++q) lp[q] = Lprev[tid + 256 * q];
  }

  // ---- 1. the diagonal block, updated, as the factorization expects it: lower part,
  // identity rows and columns beyond kb, zero above the diagonal; the first slab's rows of
  // the block column, updated, into Sg
  {
    double dv[4][4], sv[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = r0 + 8 * i, c = c0 + 8 * j;
        dv[i][j] = A[(k0 + min(r, kb - 1)) * lda + k0 + min(c, kb - 1)];
        // (no slab: a diagonal row, so that the address stays in range)
        const int64_t srow = nr1 > 0 ? rs1 + min(r, nr1 - 1) : k0 + min(r, kb - 1);
        sv[i][j] = A[srow * lda + k0 + min(c, kb - 1)];
      }
    double accS[4][4];
    chol_left_update2(A, lda, j0, k0, rs1, nr1, k0, kb, Ls, Ld, acc, accS, tid, arow, bcol, kq);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = r0 + 8 * i, c = c0 + 8 * j;
        Dg[r][c] = (r < kb && c <= r) ? dv[i][j] - acc[i][j] : (r == c ? 1.0 : 0.0);
        Sg[r][c] = (r < nr1 && c < kb) ? sv[i][j] - accS[i][j] : 0.0;
      }
  }
  __syncthreads();

  // ---- 2. factor and inverse, the columns spread over the four waves
  {
    bool notpd;
    if (wave == 0) notpd = f4_run<0>(Dg, Zs, lane, col, zrow, invd);
    else if (wave == 1) notpd = f4_run<1>(Dg, Zs, lane, col, zrow, invd);
    else if (wave == 2) notpd = f4_run<2>(Dg, Zs, lane, col, zrow, invd);
    else notpd = f4_run<3>(Dg, Zs, lane, col, zrow, invd);
    if (notpd && lane == 0 && w == 0) flags[0] = 1;
  }
  __syncthreads();

  // ---- 3. L_kk to its slot and the previous factor into A, or the slabs' rows of L
  if (w == 0) {
#pragma unroll
    for (int q = 0; q < CB * CB / 256; ++q) {
      const int e = tid + 256 * q, i = e >> 6, c = e & 63;
      Lout[e] = Dg[i][c];
      if (Lprev && i < kpb && c < kpb) A[(kp0 + i) * lda + kp0 + c] = lp[q];
    }
    return;
  }
  for (int64_t q = w - 1; q < nslab; q += gridDim.x - 1) {
    const int64_t rs = k0 + kb + CB * q;
    const int nr = (int)min<int64_t>(CB, K - rs);
    if (q != w - 1) {     // the first slab's rows are in Sg already
      chol_left_update(A, lda, j0, k0, rs, nr, k0, kb, Ls, Ld, acc, tid, arow, bcol, kq);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = r0 + 8 * i, c = c0 + 8 * j;
          const double b = A[(rs + min(r, nr - 1)) * lda + k0 + min(c, kb - 1)];
          Sg[r][c] = (r < nr && c < kb) ? b - acc[i][j] : 0.0;
        }
      __syncthreads();
    }
    // X[r][c] = sum_k Sg[r][k] Zs[c][k]  (A = Sg, B(k, c) = Zs[c][k])
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
    for (int kk = 0; kk < CB; kk += 4) {
      double af[4], bf[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = Sg[arow + 8 * i][kk + kq];
#pragma unroll
      for (int j = 0; j < 4; ++j) bf[j] = Zs[bcol + 8 * j][kk + kq];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_4x4x4f64(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = r0 + 8 * i, c = c0 + 8 * j;
        if (r < nr && c < kb) A[(rs + r) * lda + k0 + c] = acc[i][j];
      }
    __syncthreads();          // Sg is reused by the next slab
  }
}

// The last diagonal block's factor from its slot into A (k_chol_block moves every other).
__global__ __launch_bounds__(256) void k_chol_last(double* __restrict__ A, int64_t lda,
                                                   const double* __restrict__ L, int64_t k0, int kb) {
  for (int e = threadIdx.x; e < CB * CB; e += 256) {
    const int i = e >> 6, c = e & 63;
    if (i < kb && c < kb) A[(k0 + i) * lda + k0 + c] = L[e];
  }
}

// The upper factor of the damped H~ = R R^T is R[i][j] = M[K-1-i][K-1-j] (M the lower
// factor of the reversed matrix).  The rounding works with its columns scaled to a unit
// diagonal, R' = R diag(R)^-1: with Y = (clipped D) diag(R), OPTQ's error feedback y_c +=
// e_J R_Jc becomes u_c += e_J R'_Jc on u = y / R_cc, the unscaled pre-rounding values, so
// the rounding reads u_J directly and the working matrix starts as the clipped D.
// inv_rdiag[j] = 1 / R_jj first, then R' row by row.
__global__ __launch_bounds__(256) void k_rev_diag(const double* __restrict__ M, int64_t K,
                                                  double* __restrict__ inv_rdiag) {
  const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (j < K) inv_rdiag[j] = 1.0 / M[(K - 1 - j) * K + (K - 1 - j)];
}

__global__ __launch_bounds__(256) void k_reverse_upper(const double* __restrict__ M, int64_t K,
                                                       const double* __restrict__ inv_rdiag,
                                                       double* __restrict__ R) {
  for (int64_t i = blockIdx.x; i < K; i += gridDim.x) {
    const double* mrow = M + (K - 1 - i) * K + (K - 1);     // M[K-1-i][K-1-j] = mrow[-j]
    double* rrow = R + i * K;
    for (int64_t j = threadIdx.x; j < K; j += 256)
      rrow[j] = j < i ? 0.0 : (j == i ? 1.0 : mrow[-j] * inv_rdiag[j]);
  }
}

// ------------------------------------------------------------------ clip + grid
// One work-group per row: clip at [lo, hi], per-row min/max grid, Y = clipped D (the
// unscaled pre-rounding values; dead columns are masked by the rounding).
__global__ __launch_bounds__(256) void k_clip_grid(const float* __restrict__ D, int64_t cols,
                                                   int maxq, const double* __restrict__ scal,
                                                   double* __restrict__ Y, float* __restrict__ scale,
                                                   float* __restrict__ zero,
                                                   double* __restrict__ scale64,
                                                   double* __restrict__ zero64) {
  __shared__ double smin[4], smax[4];
  const int64_t r = blockIdx.x;
  const double lo_b = scal[2], hi_b = scal[3];
  const float* row = D + r * cols;
  // the row is read once: the first CK of each thread's elements stay in registers for
  // the second pass (rows up to 256 CK columns), the rest are read again
  constexpr int CK = 24;
  float keep[CK];
#pragma unroll
  for (int q = 0; q < CK; ++q) {
    const int64_t j = threadIdx.x + 256 * q;
    keep[q] = row[j < cols ? j : cols - 1];
  }
  double mn = 0.0, mx = 0.0;   // min(0, .), max(0, .)
#pragma unroll
  for (int q = 0; q < CK; ++q) {
    if (threadIdx.x + 256 * q < cols) {
      const double x = fmin(fmax((double)keep[q], lo_b), hi_b);
      mn = fmin(mn, x);
      mx = fmax(mx, x);
    }
  }
  for (int64_t j = threadIdx.x + 256 * CK; j < cols; j += 256) {
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
#pragma unroll
  for (int q = 0; q < CK; ++q) {
    const int64_t j = threadIdx.x + 256 * q;
    if (j < cols) yrow[j] = fmin(fmax((double)keep[q], lo_b), hi_b);
  }
  for (int64_t j = threadIdx.x + 256 * CK; j < cols; j += 256)
    yrow[j] = fmin(fmax((double)row[j], lo_b), hi_b);
}

// ------------------------------------------------------------------ rounding block
// Columns [i1, i1 + b) (b <= 128) of every row.  768 threads = 12 waves (three per SIMD:
// the column chain is latency bound, so more rows in flight per CU rather than more work
// per lane); each wave is four 16-lane DPP rows ("groups"), a group owns GRK rows of D.
constexpr int GB = 128;
constexpr int GRK = 1;                 // rows per 16-lane group
constexpr int GTH = 768;
constexpr int GROWS = GTH / 16 * GRK;  // 48 rows per work-group (253 groups for 12112 rows)

// Column-sequential rounding of one chunk of at most GB columns.  A group of 16 lanes
// holds GRK rows; lane g owns columns g + 16 cc (cc < 8), so the lanes of a group read a
// row of R as 16 consecutive doubles (no bank conflicts) and load / store rows of Y, D,
// codes and residuals contiguously.  Column j is rounded by its owner lane j % 16, its
// residual broadcast to the group with a DPP row broadcast, and every lane folds it into
// its own later columns: y_c += e_j R'_jc (R' = R diag(R)^-1, zero for c < j).
template <int O>
__device__ __forceinline__ double row_bcast(double v) {
  const long long b = __double_as_longlong(v);
  // every lane of a row receives the source lane's value, so no lane keeps an old value
  const int lo = __builtin_amdgcn_mov_dpp((int)(b & 0xffffffffll), 0x150 + O, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_mov_dpp((int)(b >> 32), 0x150 + O, 0xf, 0xf, false);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

struct RoundState {
  double y[GRK][8], d0[GRK][8], rr[GRK][8];
  double s[GRK], is[GRK], z[GRK];
};

// column J; rn: row J of R' (unit diagonal) at this lane's columns; rn1: the same for
// column J + 1 (rows of R' are read from LDS two columns ahead)
// FULL: a whole chunk (b = GB), so that no column needs the early exit (an exit after
// every column makes the compiler rematerialize the state's constant parts at each one)
template <int J, bool FULL>
__device__ __forceinline__ void round_col(RoundState& st, const double* __restrict__ Rs, int b,
                                          int g, double maxq, const double (&rn)[8],
                                          const double (&rn1)[8]) {
  if constexpr (J < GB) {
    if constexpr (!FULL) {
      if (J >= b) return;
    }
    constexpr int O = J & 15, C = J >> 4;
    double rnext[8];
    // slots cc below (J + 2) / 16 hold columns before J + 2 in every lane: R' is upper
    // triangular there, so column J + 2 neither reads nor updates them
    if constexpr (J + 2 < GB) {
#pragma unroll
      for (int cc = 0; cc < 8; ++cc)
        if (cc >= ((J + 2) >> 4)) rnext[cc] = Rs[(J + 2) * GB + g + 16 * cc];
    }
    double e[GRK];
#pragma unroll
    for (int k = 0; k < GRK; ++k) {
      // t = w / scale in code units; the code relative to the zero point is
      // clamp(rne(t), -zero, maxq - zero) (the zero point is an integer)
      const double t = st.y[k][C] * st.is[k];
      const double qz = fmin(fmax(rint(t), -st.z[k]), maxq - st.z[k]);
      const double ek = fma(-st.s[k], qz, st.d0[k][C]);
      if (g == O) {
        st.rr[k][C] = ek;
      }
      // the select happens here (left to itself, the compiler may keep every column's
      // residual to the end and select there, which spills)
      asm volatile("" : "+v"(st.rr[k][C]));
      e[k] = row_bcast<O>(ek);
    }
    // slots below C hold columns before J (R_Jc = 0): no update; slot C is updated in
    // every lane (lanes whose column there is <= J add e R_Jc = 0, or touch the finished
    // column J, which is not read again)
#pragma unroll
    for (int cc = 0; cc < 8; ++cc)
      if (cc >= C)
#pragma unroll
        for (int k = 0; k < GRK; ++k) st.y[k][cc] += e[k] * rn[cc];
    // pin the updated values here: otherwise the compiler sinks each update to the column
    // that reads it and keeps every broadcast residual alive
#pragma unroll
    for (int k = 0; k < GRK; ++k)
#pragma unroll
      for (int cc = 0; cc < 8; cc += 2)
        if (cc + 1 >= C) asm volatile("" : "+v"(st.y[k][cc]), "+v"(st.y[k][cc + 1]));
    if constexpr (J + 1 < GB) round_col<J + 1, FULL>(st, Rs, b, g, maxq, rn1, rnext);
  }
}

// ---- the span's earlier chunks folded into this chunk's columns before they are rounded:
// for each earlier chunk (in order), y += res[:, chunk] R'[chunk rows, this chunk's
// columns], a GROWS x b x cw product on v_mfma_f64_4x4x4f64.  The operands go through LDS
// (the R block's space, before the block is staged) in k steps of 16; every product
// element sums its k in the fp64 GEMM's order and is added to y as that GEMM's epilogue
// adds it, so the values are the ones the in-span GEMM would leave in Y.  Wave w forms
// rows 8 (w % 6) .. + 8 and columns 64 (w / 6) .. + 64 (eight 8 x 8 sub-tiles).
constexpr int SU_AP = GROWS + 8;                    // A slot: [k][row]
constexpr int SU_BP = GB + 8;                       // B slot: [k][col]
constexpr int SU_SLOT = 16 * SU_AP + 16 * SU_BP;
constexpr int SU_PP = GB + 2;                       // product tile pitch
static_assert(GTH == 768 && GROWS == 48 && GRK == 1, "span update layout assumes 48 rows, 12 waves");
static_assert(2 * SU_SLOT + GROWS * SU_PP <= GB * GB, "span update scratch fits in the R block's LDS");

__device__ __forceinline__ void su_load(const double* __restrict__ res, int64_t ld_res,
                                        const double* __restrict__ R, int64_t cols, int64_t wr0,
                                        int64_t rows, int64_t rrow0, int col0, int kc, int b,
                                        int i1, int kb, double& av, double (&bv)[3]) {
  const int t = threadIdx.x;
  {  // A: row t / 16, k t % 16 of the chunk's residuals
    const int row = t >> 4, k = kb + (t & 15);
    const int64_t r = wr0 + row;
    av = (r < rows && k < kc) ? res[r * ld_res + col0 + k] : 0.0;
  }
#pragma unroll
  for (int q = 0; q < 3; ++q) {  // B: k = e / 128, column e % 128 of R' rows of the chunk
    const int e = t + GTH * q;
    const int k = kb + (e >> 7), c = e & 127;
    bv[q] = (e < 16 * GB && k < kc && c < b) ? R[(rrow0 + k) * cols + i1 + c] : 0.0;
  }
}

__device__ __forceinline__ void su_store(double* slot, double av, const double (&bv)[3]) {
  const int t = threadIdx.x;
  slot[(t & 15) * SU_AP + (t >> 4)] = av;
  double* bs = slot + 16 * SU_AP;
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    const int e = t + GTH * q;
    if (e < 16 * GB) bs[(e >> 7) * SU_BP + (e & 127)] = bv[q];
  }
}

__device__ __forceinline__ void span_update(RoundState& st, double* lds,
                                            const double* __restrict__ res, int64_t ld_res,
                                            int64_t res_col0, int cw,
                                            const double* __restrict__ R, int64_t cols, int i1,
                                            int b, int64_t rows, int64_t wr0, int grp, int g) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int blk = (lane >> 2) & 3, bi = blk >> 1, bj = blk & 1, q4 = lane & 3, kq = lane >> 4;
  const int arow = 8 * (w % 6) + 4 * bi + q4, bcol = 64 * (w / 6) + 4 * bj + q4;
  double* P = lds + 2 * SU_SLOT;
  const int64_t s1 = i1 - res_col0;
  for (int64_t col0 = 0; col0 < res_col0; col0 += cw) {
    const int kc = (int)min<int64_t>(cw, res_col0 - col0);
    const int nks = (kc + 15) / 16;
    double acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.0;
    double av, bv[3];
    su_load(res, ld_res, R, cols, wr0, rows, s1 + col0, (int)col0, kc, b, i1, 0, av, bv);
    su_store(lds, av, bv);
    __syncthreads();
    for (int ks = 0; ks < nks; ++ks) {
      const double* slot = lds + (ks & 1) * SU_SLOT;
      const bool more = ks + 1 < nks;
      if (more) su_load(res, ld_res, R, cols, wr0, rows, s1 + col0, (int)col0, kc, b, i1,
                        16 * (ks + 1), av, bv);
#pragma unroll
      for (int kk = 0; kk < 16; kk += 4) {
        const double af = slot[(kk + kq) * SU_AP + arow];
        double bf[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) bf[j] = slot[16 * SU_AP + (kk + kq) * SU_BP + bcol + 8 * j];
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = __builtin_amdgcn_mfma_f64_4x4x4f64(af, bf[j], acc[j], 0, 0, 0);
      }
      if (more) su_store(lds + ((ks + 1) & 1) * SU_SLOT, av, bv);
      __syncthreads();
    }
    // lane l holds row 4 bi + l / 16 and column 4 bj + l % 4 of each 8 x 8 sub-tile
#pragma unroll
    for (int j = 0; j < 8; ++j)
      P[(8 * (w % 6) + 4 * bi + kq) * SU_PP + 64 * (w / 6) + 4 * bj + q4 + 8 * j] = acc[j];
    __syncthreads();
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) st.y[0][cc] += P[grp * SU_PP + g + 16 * cc];
    __syncthreads();
  }
}

typedef __attribute__((address_space(3))) void lds_void;

// Global -> LDS copies (wave-uniform base + per-lane byte offset; lane l lands at
// lds + 16 l or lds + 4 l).  Inline assembly, so that the compiler does not make every
// later LDS read wait for them: completion is tracked by the explicit vmcnt wait.
__device__ __forceinline__ void lds_copy16(const char* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               : : "v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
__device__ __forceinline__ void lds_copy4(const char* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1"
               : : "v"(off), "s"(base), "s"(lds) : "memory", "m0");
}

// The same products with the operands copied global -> LDS by the DMA path
// (global_load_lds), three k steps of 16 in flight ahead of the one being multiplied
// (four slots), and the running sum kept in the product's register layout across the
// span's earlier chunks (per chunk: acc = its product, then sum += acc, the order and
// roundings of the GEMM route).  For whole 128-column chunks with 16-byte aligned rows of
// res and R.  Slot: A rows of 128 bytes, k at position k ^ 2 (row & 7); B k-rows of 1 KB,
// column n at position n ^ 8 (k-row & 3) (the LDS-ring kernel's layouts).  Waves 0..7
// copy B k-rows w and w + 8, waves 8..10 two A row groups of 8 each, wave 11 nothing:
// every copying wave has exactly two copies per step in flight.  Wave w multiplies rows
// 16 (w / 4) .. + 16 and columns 32 (w % 4) .. + 32 (2 x 4 sub-tiles of 8 x 8: six LDS
// reads per eight MFMAs).
constexpr int SA_BYTES = GROWS * 128;               // 6 KB
constexpr int SB_BYTES = 16 * 1024;                 // 16 KB
constexpr int SS_BYTES = SA_BYTES + SB_BYTES;
constexpr int SS_N = 4;                             // slots
static_assert(SS_N * SS_BYTES <= GB * GB * 8 && GROWS * SU_PP * 8 <= GB * GB * 8,
              "span update slots fit in the R block's LDS");

__device__ __forceinline__ bool span_async_ok(const double* res, int64_t ld_res,
                                              const double* R, int64_t cols, int b, int cw) {
  return b == GB && cw == GB && (cols & 1) == 0 && (ld_res & 1) == 0 &&
         ((reinterpret_cast<uintptr_t>(res) | reinterpret_cast<uintptr_t>(R)) & 15) == 0;
}

__device__ __forceinline__ void span_update_async(RoundState& st, double* lds,
                                                  const double* __restrict__ res,
                                                  int64_t ld_res, int64_t res_col0,
                                                  const double* __restrict__ R, int64_t cols,
                                                  const double* __restrict__ Y, int i1,
                                                  int64_t rows, int64_t wr0, int grp, int g) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int blk = (lane >> 2) & 3, bi = blk >> 1, bj = blk & 1, q4 = lane & 3, kq = lane >> 4;
  const int wr = w >> 2, wc = w & 3;                // 16-row group, 32-column group
  const int ra7 = 4 * bi + q4;                      // fragment row mod 8
  const int nst = (int)(res_col0 / 16);             // k steps (8 per earlier chunk)
  const int64_t s1 = i1 - res_col0;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void*)lds;
  // this wave's copy offsets (bytes from the step's source base)
  uint32_t off[2];
  const char* srcA = reinterpret_cast<const char*>(res + wr0 * ld_res);
  const char* srcB = reinterpret_cast<const char*>(R + s1 * cols + i1);
  if (w < 8) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int kr = w + 8 * i;
      off[i] = (uint32_t)((kr * cols + ((2 * lane) ^ (8 * (kr & 3)))) * 8);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int r = 8 * (2 * (w - 8) + i) + (lane >> 3), c = lane & 7;
      const int64_t gr = min<int64_t>(wr0 + r, rows - 1) - wr0;
      off[i] = (uint32_t)((gr * ld_res + 2 * (c ^ (r & 7))) * 8);
    }
  }
  auto issue = [&](int s) {
    const uint32_t slot = lds0 + (uint32_t)((s % SS_N) * SS_BYTES);
    if (w < 8) {
      const char* b = srcB + (int64_t)s * 16 * cols * 8;
#pragma unroll
      for (int i = 0; i < 2; ++i) lds_copy16(b, off[i], slot + SA_BYTES + (w + 8 * i) * 1024);
    } else if (w < 11) {
      const char* a = srcA + (int64_t)s * 16 * 8;
#pragma unroll
      for (int i = 0; i < 2; ++i) lds_copy16(a, off[i], slot + (2 * (w - 8) + i) * 1024);
    }
  };
  auto barrier = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };
  // fragment offsets inside a slot: A rows 16 wr + 8 i + ra7, k = 4 t + kq; B k-row
  // 4 t + kq, columns 32 wc + 4 bj + q4 + 8 j
  uint32_t xa[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int t = 0; t < 4; ++t)
      xa[i][t] = (uint32_t)((16 * wr + 8 * i + ra7) * 128 + 8 * ((4 * t + kq) ^ (2 * ra7)));
  const int bc = 32 * wc + 4 * bj + q4;
  // the running sum, from Y, in the product's layout (rows 16 wr + 8 i + 4 bi + kq,
  // columns bc + 8 j)
  double sum[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int64_t r = min<int64_t>(wr0 + 16 * wr + 8 * i + 4 * bi + kq, rows - 1);
#pragma unroll
    for (int j = 0; j < 4; ++j) sum[i][j] = Y[r * cols + i1 + bc + 8 * j];
  }
  double acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
  for (int s = 0; s < SS_N - 1 && s < nst; ++s) issue(s);
  for (int s = 0; s < nst; ++s) {
    // this step's copies landed (each wave its own, then all): at most the later issued
    // steps (two copies each) may still be in flight
    const int later = min(SS_N - 2, nst - 1 - s);
    if (w < 11) {
      if (later >= 2) __builtin_amdgcn_s_waitcnt(0x0F70 | 4);
      else if (later == 1) __builtin_amdgcn_s_waitcnt(0x0F70 | 2);
      else __builtin_amdgcn_s_waitcnt(0x0F70);
    }
    barrier();
    if (s + SS_N - 1 < nst) issue(s + SS_N - 1);
    const char* slot = reinterpret_cast<const char*>(lds) + (s % SS_N) * SS_BYTES;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      double af[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = *reinterpret_cast<const double*>(slot + xa[i][t]);
      const int kr = 4 * t + kq;
      double bf[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bf[j] = *reinterpret_cast<const double*>(slot + SA_BYTES + kr * 1024 +
                                                 8 * ((bc + 8 * j) ^ (8 * (kr & 3))));
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_4x4x4f64(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if ((s & 7) == 7) {       // the end of an earlier chunk: add its product
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          sum[i][j] += acc[i][j];
          acc[i][j] = 0.0;
        }
    }
  }
  barrier();                  // every slot read; the product tile goes over them
  double* P = lds;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
      P[(16 * wr + 8 * i + 4 * bi + kq) * SU_PP + bc + 8 * j] = sum[i][j];
  __syncthreads();
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) st.y[0][cc] = P[grp * SU_PP + g + 16 * cc];
  __syncthreads();
}

__global__ __launch_bounds__(GTH) void k_gptq_block(
    const float* __restrict__ D, int64_t rows, int64_t cols, int i1, int b, int64_t res_col0,
    int cw, int64_t ld_res, int maxq, const double* __restrict__ scal,
    const uint8_t* __restrict__ dead, const double* __restrict__ R,
    const double* __restrict__ scale64, const double* __restrict__ zero64,
    const double* __restrict__ Y, uint8_t* __restrict__ codes8, double* __restrict__ res) {
  __shared__ __attribute__((aligned(16))) double Rs[GB * GB];
  const int lane = threadIdx.x & 63;
  const int g = lane & 15;                         // position inside the 16-lane group
  const int grp = threadIdx.x >> 4;                // group index in the work-group
  const int64_t r0 = (int64_t)blockIdx.x * GROWS + grp * GRK;
  const double lo_b = scal[2], hi_b = scal[3];

  RoundState st;
  // y: this chunk's columns of Y, plus the residuals of the span's earlier chunks
  if (res_col0 > 0 && span_async_ok(res, ld_res, R, cols, b, cw)) {
    span_update_async(st, Rs, res, ld_res, res_col0, R, cols, Y, i1, rows,
                      (int64_t)blockIdx.x * GROWS, grp, g);
  } else {
    {
      const int64_t r = min(r0, rows - 1);
      double yv[8];
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) yv[cc] = Y[r * cols + i1 + min(g + 16 * cc, b - 1)];
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) st.y[0][cc] = yv[cc];
    }
    if (res_col0 > 0)
      span_update(st, Rs, res, ld_res, res_col0, cw, R, cols, i1, b, rows,
                  (int64_t)blockIdx.x * GROWS, grp, g);
  }
  // the grid, the clipped D, and the masks: columns outside the chunk, dead columns (the
  // products above add exact zeros there, R' being zero off the diagonal) and rows
  // outside D hold y = 0
  {
    float dv[GRK][8];
    uint8_t dd[8];
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) dd[cc] = dead[i1 + min(g + 16 * cc, b - 1)];
#pragma unroll
    for (int k = 0; k < GRK; ++k) {
      const int64_t r = min(r0 + k, rows - 1);
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) dv[k][cc] = D[r * cols + i1 + min(g + 16 * cc, b - 1)];
    }
#pragma unroll
    for (int k = 0; k < GRK; ++k) {
      const int64_t r = r0 + k;
      const bool ok = r < rows;
      const int64_t rc = ok ? r : rows - 1;
      st.s[k] = ok ? scale64[rc] : 1.0;
      st.is[k] = 1.0 / st.s[k];
      st.z[k] = ok ? zero64[rc] : 0.0;
#pragma unroll
      for (int cc = 0; cc < 8; ++cc) {
        const bool in = ok && g + 16 * cc < b;
        st.y[k][cc] = (in && !dd[cc]) ? st.y[k][cc] : 0.0;
        st.d0[k][cc] = (in && !dd[cc]) ? fmin(fmax((double)dv[k][cc], lo_b), hi_b) : 0.0;
        st.rr[k][cc] = 0.0;
      }
    }
  }

  // R' block: Rs[rr][cc] = R'[i1 + rr][i1 + cc] for rr, cc < b, 0 elsewhere.  A whole
  // chunk with 16-byte aligned rows goes global -> LDS by the DMA path, one copy per row,
  // all in flight together; otherwise every load is issued unconditionally from a clamped
  // in-bounds address, a batch of a thread's at once.
  if (b == GB && (cols & 1) == 0 && (reinterpret_cast<uintptr_t>(R) & 15) == 0) {
    const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_void*)Rs;
    // the block's first element, made wave-uniform for the copy's scalar base
    const uint64_t bp = reinterpret_cast<uint64_t>(R + (int64_t)i1 * cols + i1);
    const char* base = reinterpret_cast<const char*>(
        ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(bp >> 32)) << 32) |
        (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)bp));
    for (int row = w; row < GB; row += GTH / 64)
      lds_copy16(base, (uint32_t)((row * cols + 2 * lane) * 8), lds0 + (uint32_t)(row * GB * 8));
    __builtin_amdgcn_s_waitcnt(0x0F70);               // vmcnt(0): this wave's rows landed
  } else {
    constexpr int NE = GB * GB, PER = (NE + GTH - 1) / GTH, BATCH = 16;
#pragma unroll
    for (int q0 = 0; q0 < PER; q0 += BATCH) {
      double v[BATCH];
#pragma unroll
      for (int q = 0; q < BATCH; ++q) {
        const int e = min((int)threadIdx.x + (q0 + q) * GTH, NE - 1);
        const int rr = min(e / GB, b - 1), cc = min(e % GB, b - 1);
        v[q] = R[(int64_t)(i1 + rr) * cols + i1 + cc];
      }
#pragma unroll
      for (int q = 0; q < BATCH; ++q) {
        const int e = (int)threadIdx.x + (q0 + q) * GTH;
        if (q0 + q < PER && e < NE) Rs[e] = ((e / GB) < b && (e % GB) < b) ? v[q] : 0.0;
      }
    }
  }

  __syncthreads();

  double rn[8];
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) rn[cc] = Rs[g + 16 * cc];
  double rn1[8];
#pragma unroll
  for (int cc = 0; cc < 8; ++cc) rn1[cc] = Rs[GB + g + 16 * cc];
  if (b == GB) round_col<0, true>(st, Rs, b, g, (double)maxq, rn, rn1);
  else round_col<0, false>(st, Rs, b, g, (double)maxq, rn, rn1);

#pragma unroll
  for (int k = 0; k < GRK; ++k) {
    const int64_t r = r0 + k;
    if (r >= rows) continue;
#pragma unroll
    for (int cc = 0; cc < 8; ++cc) {
      const int c = g + 16 * cc;
      if (c < b) {
        // the code from the kept residual: e = fma(-s, qz, d0) is exact to within an ulp
        // of e, so (d0 - e) / s is qz to within 2^-50 and rounds back to it
        const double qz = rint((st.d0[k][cc] - st.rr[k][cc]) * st.is[k]);
        codes8[r * cols + i1 + c] = (uint8_t)(qz + st.z[k]);
        res[r * ld_res + res_col0 + c] = st.rr[k][cc];
      }
    }
  }
}

// ------------------------------------------------------------------ fp64 MFMA GEMM
// C[M x N] = beta * C + alpha * A[M x K] * op(B).  Tile DT x DT (64 or 128), K step 16,
// 256 threads = 2 x 2 waves of DT/2 x DT/2.  Operands are staged k-major in LDS ([k][m],
// [k][n]) and the next K step is fetched into registers while the current one is
// multiplied.  C must not overlap A or B (tiles read operands that other tiles write).
//
// The products use v_mfma_f64_4x4x4f64, which on gfx950 sustains about 1.6x the fp64
// rate of the 16x16x4 form.  One instruction is four independent 4 x 4 x 4 products
// (blocks b = 0..3); lane l holds A_b[i][k] at l = 4b + i + 16k, B_b[k][j] at
// l = 4b + j + 16k and D_b[i][j] at l = 4b + j + 16i.  The blocks are laid 2 x 2
// (b = 2 bi + bj) over an 8 x 8 output sub-tile, so every A value feeds two blocks and
// every B value two.
constexpr int DK = 16, DPAD = 8;   // row pitch = DT + 8 doubles: the four k rows of a
                                   // fragment read fall on disjoint banks

struct DgemmArgs {
  int64_t M, N, K;
  double alpha, beta;
  const double* A; int64_t lda;
  const double* B; int64_t ldb;
  double* C; int64_t ldc;
  int b_trans, lower_only, tiles_n;
  int b16;                    // B 16-byte aligned with an even ldb (ring kernel)
};

// One K step (16) of the DT x DT tile's operands: each of the 256 threads fetches DT / 16
// doubles of A and of op(B) (zero outside the matrices).
template <int DT>
__device__ __forceinline__ void dg_load(const DgemmArgs& p, int64_t m0, int64_t n0, int64_t k0,
                                        double (&ra)[DT / 16], double (&rb)[DT / 16], int tid) {
  constexpr int PER = DT / 16;             // doubles per thread per operand
  constexpr int TPR = 16 / PER;            // threads per 16-wide k row
  {  // A: row m0 + tid / TPR, k0 + PER * (tid % TPR)
    const int64_t gm = m0 + tid / TPR;
    const int64_t gk = k0 + PER * (tid % TPR);
#pragma unroll
    for (int q = 0; q < PER; ++q)
      ra[q] = (gm < p.M && gk + q < p.K) ? p.A[gm * p.lda + gk + q] : 0.0;
  }
  if (p.b_trans) {  // op(B)(k, n) = B[n * ldb + k]
    const int64_t gn = n0 + tid / TPR;
    const int64_t gk = k0 + PER * (tid % TPR);
#pragma unroll
    for (int q = 0; q < PER; ++q)
      rb[q] = (gn < p.N && gk + q < p.K) ? p.B[gn * p.ldb + gk + q] : 0.0;
  } else {          // B[k * ldb + n]: row k0 + tid / (DT / PER), n0 + PER * (tid % (DT / PER))
    constexpr int TPN = DT / PER;
    const int64_t gk = k0 + tid / TPN;
    const int64_t gn = n0 + PER * (tid % TPN);
#pragma unroll
    for (int q = 0; q < PER; ++q)
      rb[q] = (gk < p.K && gn + q < p.N) ? p.B[gk * p.ldb + gn + q] : 0.0;
  }
}

template <int DT>
__device__ __forceinline__ void dg_store(const DgemmArgs& p, double (*As)[DT + DPAD],
                                         double (*Bs)[DT + DPAD], const double (&ra)[DT / 16],
                                         const double (&rb)[DT / 16], int tid) {
  constexpr int PER = DT / 16;
  constexpr int TPR = 16 / PER;
#pragma unroll
  for (int q = 0; q < PER; ++q) As[PER * (tid % TPR) + q][tid / TPR] = ra[q];
  if (p.b_trans) {
#pragma unroll
    for (int q = 0; q < PER; ++q) Bs[PER * (tid % TPR) + q][tid / TPR] = rb[q];
  } else {
    constexpr int TPN = DT / PER;
#pragma unroll
    for (int q = 0; q < PER; ++q) Bs[tid / TPN][PER * (tid % TPN) + q] = rb[q];
  }
}

template <int DT>
__global__ __launch_bounds__(256) void k_dgemm(DgemmArgs p) {
  __shared__ double As[2][DK][DT + DPAD];
  __shared__ double Bs[2][DK][DT + DPAD];
  int tm, tn;
  if (p.lower_only) {
    int t = blockIdx.x, row = 0;
    while (t > row) { t -= row + 1; ++row; }
    tm = row;
    tn = t;
  } else {
    tm = blockIdx.x / p.tiles_n;
    tn = blockIdx.x - tm * p.tiles_n;
  }
  const int64_t m0 = (int64_t)tm * DT, n0 = (int64_t)tn * DT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int WS = DT / 16;           // 8 x 8 sub-tiles per wave side
  double acc[WS][WS];
#pragma unroll
  for (int i = 0; i < WS; ++i)
#pragma unroll
    for (int j = 0; j < WS; ++j) acc[i][j] = 0.0;
  const int blk = (lane >> 2) & 3, bi = blk >> 1, bj = blk & 1, q4 = lane & 3, kq = lane >> 4;
  const int arow = wm * (DT / 2) + 4 * bi + q4;     // fragment row of sub-tile 0
  const int bcol = wn * (DT / 2) + 4 * bj + q4;     // fragment column of sub-tile 0

  double ra[DT / 16], rb[DT / 16];
  const int nk = (int)((p.K + DK - 1) / DK);
  if (nk > 0) {
    dg_load<DT>(p, m0, n0, 0, ra, rb, tid);
    dg_store<DT>(p, As[0], Bs[0], ra, rb, tid);
  }
  __syncthreads();
  for (int s = 0; s < nk; ++s) {
    const int buf = s & 1;
    const bool more = s + 1 < nk;
    if (more) dg_load<DT>(p, m0, n0, (int64_t)(s + 1) * DK, ra, rb, tid);
#pragma unroll
    for (int kk = 0; kk < DK; kk += 4) {
      double af[WS], bfv[WS];
#pragma unroll
      for (int i = 0; i < WS; ++i) af[i] = As[buf][kk + kq][arow + 8 * i];
#pragma unroll
      for (int j = 0; j < WS; ++j) bfv[j] = Bs[buf][kk + kq][bcol + 8 * j];
#pragma unroll
      for (int i = 0; i < WS; ++i)
#pragma unroll
        for (int j = 0; j < WS; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_4x4x4f64(af[i], bfv[j], acc[i][j], 0, 0, 0);
    }
    if (more) dg_store<DT>(p, As[buf ^ 1], Bs[buf ^ 1], ra, rb, tid);
    __syncthreads();
  }
  // lane l holds row 4 bi + l / 16, column 4 bj + l % 4 of each 8 x 8 sub-tile; C is
  // read a sub-tile row at a time, every read before the stores (clamped addresses)
  const int64_t r0 = m0 + wm * (DT / 2) + 4 * bi + kq;
  const int64_t c0 = n0 + wn * (DT / 2) + 4 * bj + q4;
#pragma unroll
  for (int i = 0; i < WS; ++i) {
    const int64_t row = r0 + 8 * i;
    double cv[WS];
#pragma unroll
    for (int j = 0; j < WS; ++j)
      cv[j] = p.beta != 0.0 ? p.C[min(row, p.M - 1) * p.ldc + min(c0 + 8 * j, p.N - 1)] : 0.0;
#pragma unroll
    for (int j = 0; j < WS; ++j) cv[j] = p.beta * cv[j] + p.alpha * acc[i][j];
#pragma unroll
    for (int j = 0; j < WS; j += 2) asm volatile("" : "+v"(cv[j]), "+v"(cv[j + 1]));
    if (row < p.M) {
#pragma unroll
      for (int j = 0; j < WS; ++j)
        if (c0 + 8 * j < p.N) p.C[row * p.ldc + c0 + 8 * j] = cv[j];
    }
  }
}

// The same product for 32 x 32 tiles and K <= 128 (the factorization's next-panel update,
// a chain of short launches where every K step of k_dgemm would wait for its own loads):
// the operands of every K step are fetched at the start, so that the loads overlap, then
// staged through LDS one step at a time and multiplied in k_dgemm's order; C is read at
// the start as well.
constexpr int PF_STEPS = 8;
__global__ __launch_bounds__(256) void k_dgemm32_short(DgemmArgs p) {
  constexpr int DT = 32, WS = 2;
  __shared__ double As[2][DK][DT + DPAD];
  __shared__ double Bs[2][DK][DT + DPAD];
  const int tm = blockIdx.x / p.tiles_n, tn = blockIdx.x - tm * p.tiles_n;
  const int64_t m0 = (int64_t)tm * DT, n0 = (int64_t)tn * DT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int blk = (lane >> 2) & 3, bi = blk >> 1, bj = blk & 1, q4 = lane & 3, kq = lane >> 4;
  const int arow = wm * (DT / 2) + 4 * bi + q4;
  const int bcol = wn * (DT / 2) + 4 * bj + q4;
  const int nk = (int)((p.K + DK - 1) / DK);        // <= PF_STEPS
  double ra[PF_STEPS][2], rb[PF_STEPS][2];
#pragma unroll
  for (int s = 0; s < PF_STEPS; ++s)
    if (s < nk) dg_load<DT>(p, m0, n0, (int64_t)s * DK, ra[s], rb[s], tid);
  // C's values too (clamped addresses; values outside the matrix are discarded)
  const int64_t r0 = m0 + wm * (DT / 2) + 4 * bi + kq;
  const int64_t c0 = n0 + wn * (DT / 2) + 4 * bj + q4;
  double cv[WS][WS];
#pragma unroll
  for (int i = 0; i < WS; ++i)
#pragma unroll
    for (int j = 0; j < WS; ++j)
      cv[i][j] = p.beta != 0.0 ? p.C[min(r0 + 8 * i, p.M - 1) * p.ldc + min(c0 + 8 * j, p.N - 1)] : 0.0;
  double acc[WS][WS];
#pragma unroll
  for (int i = 0; i < WS; ++i)
#pragma unroll
    for (int j = 0; j < WS; ++j) acc[i][j] = 0.0;
  // slot s & 1 was last read in step s - 2, before every wave passed the barrier of s - 1
#pragma unroll
  for (int s = 0; s < PF_STEPS; ++s) {
    if (s >= nk) break;
    dg_store<DT>(p, As[s & 1], Bs[s & 1], ra[s], rb[s], tid);
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < DK; kk += 4) {
      double af[WS], bfv[WS];
#pragma unroll
      for (int i = 0; i < WS; ++i) af[i] = As[s & 1][kk + kq][arow + 8 * i];
#pragma unroll
      for (int j = 0; j < WS; ++j) bfv[j] = Bs[s & 1][kk + kq][bcol + 8 * j];
#pragma unroll
      for (int i = 0; i < WS; ++i)
#pragma unroll
        for (int j = 0; j < WS; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_4x4x4f64(af[i], bfv[j], acc[i][j], 0, 0, 0);
    }
  }
#pragma unroll
  for (int i = 0; i < WS; ++i) {
    const int64_t row = r0 + 8 * i;
#pragma unroll
    for (int j = 0; j < WS; ++j) cv[i][j] = p.beta * cv[i][j] + p.alpha * acc[i][j];
#pragma unroll
    for (int j = 0; j < WS; j += 2) asm volatile("" : "+v"(cv[i][j]), "+v"(cv[i][j + 1]));
    if (row < p.M) {
#pragma unroll
      for (int j = 0; j < WS; ++j)
        if (c0 + 8 * j < p.N) p.C[row * p.ldc + c0 + 8 * j] = cv[i][j];
    }
  }
}

// ------------------------------------------------------------------ fp64 GEMM, LDS ring
// C = beta C + alpha A op(B) for row-major A (M x K, rows 16-byte aligned) and B (K x N,
// or with BT op(B)(k, n) = B[n ldb + k], rows 16-byte aligned), K a multiple of 16: the
// trailing updates of the rounding and of the Cholesky factorization (BT, LOWER: only the
// tiles on or below the diagonal, a diagonal tile computed and stored in full).  Tile
// 128 x 128, 8 waves of
// 32 x 64 built from 8 x 8 sub-tiles of the 2 x 2 block arrangement above; two
// work-groups per CU (four waves per SIMD).  The waves copy each K step of 16 straight
// from global memory into LDS (A in 16-byte pieces, rows clamped to M; B one dword per
// lane, columns clamped to N element by element), without a pass through registers,
// into two slots: the copy of step s + 1 runs while step s is multiplied.
//   A slot: row r at byte 128 r, k stored at position k ^ 2 (r & 7)
//   B slot: k-row kr at byte 1024 kr, column n stored at position n ^ 8 (kr & 3)
// so that the 8 rows (A, one k) and 8 columns (B, one k) that a group of 16 lanes
// reads fall on distinct banks (A pairs k = 2c, 2c + 1 stay together for the 16-byte
// copies).
constexpr int RT = 128, RK = 16, RST = 2;
constexpr int RA_BYTES = RT * RK * 8;               // A part of a slot
constexpr int RSLOT = 2 * RA_BYTES;
constexpr int RWAVES = 8;
constexpr int RA_PER = RA_BYTES / 1024 / RWAVES;     // 16-byte copies per wave and step (2)
constexpr int RB_PER = RA_BYTES / 256 / RWAVES;      // dword copies per wave and step (8)
static_assert(RA_PER == 2 && RB_PER == 8, "copy layout below assumes 8 waves");


template <bool BT, bool LOWER>
__global__ __launch_bounds__(64 * RWAVES, 4) void k_dgemm_ring(DgemmArgs p) {
  __shared__ __attribute__((aligned(16))) char ring[RST * RSLOT];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;          // 32-row group, 64-column half
  // work-group -> tile: contiguous ranges per XCD (ids are dealt round-robin to 8), then
  // groups of 8 tile-rows walked column by column (LOWER: the lower tiles row by row)
  int tm, tn;
  {
    const int nb = gridDim.x, b = blockIdx.x;
    const int per = nb / 8, rem = nb % 8;
    const int xcd = b % 8, idx = b / 8;
    const int t = (xcd < rem) ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
    if (LOWER) {
      // t = tm (tm + 1) / 2 + tn, tn <= tm
      int r = (int)((sqrt(8.0 * (double)t + 1.0) - 1.0) * 0.5);
      while ((r + 1) * (r + 2) / 2 <= t) ++r;
      while (r * (r + 1) / 2 > t) --r;
      tm = r;
      tn = t - r * (r + 1) / 2;
    } else {
      const int tiles_m = (int)((p.M + RT - 1) / RT);
      const int g = t / (8 * p.tiles_n);
      const int first = g * 8;
      const int gs = min(8, tiles_m - first);
      const int in = t - g * 8 * p.tiles_n;
      tm = first + in % gs;
      tn = in / gs;
    }
  }
  const int64_t m0 = (int64_t)tm * RT, n0 = (int64_t)tn * RT;
  const int nst = (int)(p.K / RK);

  // A copy i (i = 0, 1) of this wave: rows 8 (2 wave + i) + lane / 8, k pair c ^ (r & 7)
  // at chunk c = lane % 8.  B copy i: k-row 2 wave + i / 4, columns 32 (i % 4) + 0..31,
  // column n at position n ^ 8 (k-row & 3); offsets clamp at the last column.
  uint32_t ga[2], gb[2];
  // clamp limit of this wave's first B k-row (the last column of the matrix); the second
  // k-row's is ldb further
  const uint32_t gl0 = (uint32_t)((2 * wave * p.ldb + (p.N - 1 - n0)) * 8 + 4 * (lane & 1));
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int r = 8 * (2 * wave + i) + (lane >> 3), c = lane & 7;
    const int64_t gr = min(m0 + r, p.M - 1) - m0;
    ga[i] = (uint32_t)((gr * p.lda + 2 * (c ^ (r & 7))) * 8);
    if (BT) {
      // op(B) rows n (B's rows) are copied like A's rows, clamped to N
      const int64_t gn = min(n0 + r, p.N - 1) - n0;
      gb[i] = (uint32_t)((gn * p.ldb + 2 * (c ^ (r & 7))) * 8);
    } else {
      const int kr = 2 * wave + i;
      const int nl = (lane >> 1) ^ (8 * (kr & 3));
      gb[i] = (uint32_t)((kr * p.ldb + nl) * 8 + 4 * (lane & 1));
    }
  }
  const uint32_t ring_lds = (uint32_t)(uintptr_t)(lds_void*)ring;
  const char* srcA = reinterpret_cast<const char*>(p.A + m0 * p.lda);
  const char* srcB = reinterpret_cast<const char*>(BT ? p.B + n0 * p.ldb : p.B + n0);
  const int64_t stepA = RK * 8, stepB = BT ? (int64_t)RK * 8 : (int64_t)RK * p.ldb * 8;
  const bool bx4 = p.b16 && n0 + RT <= p.N;
  auto issue = [&](int s) {
    const uint32_t slot = ring_lds + (uint32_t)((s & 1) * RSLOT);
    const char* a = srcA + s * stepA;
    const char* b = srcB + s * stepB;
#pragma unroll
    for (int i = 0; i < 2; ++i) lds_copy16(a, ga[i], slot + (2 * wave + i) * 1024);
    if (BT) {
#pragma unroll
      for (int i = 0; i < 2; ++i) lds_copy16(b, gb[i], slot + RA_BYTES + (2 * wave + i) * 1024);
    } else if (bx4) {
      // interior column tile: whole k-rows of B in 16-byte pieces (column pairs stay
      // together under the swizzle)
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int kr = 2 * wave + i;
        const uint32_t off = (uint32_t)((kr * p.ldb + ((2 * lane) ^ (8 * (kr & 3)))) * 8);
        lds_copy16(b, off, slot + RA_BYTES + kr * 1024);
      }
    } else {
      // the clamped offsets are formed here at every step (opaque copies of the bases
      // keep the compiler from holding all eight in registers)
      uint32_t b0 = gb[0], b1 = gb[1], l0 = gl0;
      asm volatile("" : "+v"(b0), "+v"(b1), "+v"(l0));
      const uint32_t l1 = l0 + (uint32_t)(p.ldb * 8);
#pragma unroll
      for (int i = 0; i < 8; ++i)
        lds_copy4(b, min((i < 4 ? b0 : b1) + 256 * (i & 3), i < 4 ? l0 : l1),
                  slot + RA_BYTES + (8 * wave + i) * 256);
    }
  };
  auto barrier = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // fragment read offsets: A sub-tile i adds 1024 i, k group t uses xa[t]; B sub-tile j
  // uses xb[j % 4] + 256 (j / 4), k group t adds 4096 t
  const int blk = (lane >> 2) & 3, bi = blk >> 1, bj = blk & 1, q4 = lane & 3, kq = lane >> 4;
  const int ra7 = 4 * bi + q4;                      // fragment row mod 8
  const uint32_t base_a = (uint32_t)((wm * 32 + ra7) * 128);
  uint32_t xa[4], xb[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) xa[t] = base_a + 8 * ((4 * t + kq) ^ (2 * ra7));
  if (BT) {
    // op(B) slot laid out like A's: column n at byte 128 n, k at position k ^ 2 (n & 7);
    // sub-tile j adds 1024 j (8 columns), k group t uses xb[t]
    const int rb7 = 4 * bj + q4;
    const uint32_t base_b = (uint32_t)(RA_BYTES + (wn * 64 + rb7) * 128);
#pragma unroll
    for (int t = 0; t < 4; ++t) xb[t] = base_b + 8 * ((4 * t + kq) ^ (2 * rb7));
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      xb[j] = (uint32_t)(RA_BYTES + kq * 1024 + (wn * 64 + 4 * bj + q4) * 8 + 64 * (j ^ kq));
  }

  double acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0;

  if (nst > 0) issue(0);
  for (int s = 0; s < nst; ++s) {
    // step s landed (own copies, then everyone's); step s - 1 read by every wave
    __builtin_amdgcn_s_waitcnt(0x0F70);               // vmcnt(0): lgkmcnt, expcnt untouched
    barrier();
    if (s + 1 < nst) issue(s + 1);
    const char* slot = ring + (s & 1) * RSLOT;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      double af[4], bfv[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const double*>(slot + xa[t] + 1024 * i);
      if (BT) {
#pragma unroll
        for (int j = 0; j < 8; ++j) bfv[j] = *reinterpret_cast<const double*>(slot + xb[t] + 1024 * j);
      } else {
#pragma unroll
        for (int j = 0; j < 8; ++j)
          bfv[j] = *reinterpret_cast<const double*>(slot + xb[j & 3] + 256 * (j >> 2) + 4096 * t);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f64_4x4x4f64(af[i], bfv[j], acc[i][j], 0, 0, 0);
    }
  }
  // lane l holds row 4 bi + l / 16, column 4 bj + l % 4 of each 8 x 8 sub-tile.  C is
  // read a sub-tile row (8 values) at a time, all reads before the stores (clamped
  // addresses; values outside the matrix are discarded).
  const int64_t r0 = m0 + wm * 32 + 4 * bi + kq;
  const int64_t c0 = n0 + wn * 64 + 4 * bj + q4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t row = r0 + 8 * i;
    double cv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      cv[j] = p.beta != 0.0 ? p.C[min(row, p.M - 1) * p.ldc + min(c0 + 8 * j, p.N - 1)] : 0.0;
#pragma unroll
    for (int j = 0; j < 8; ++j) cv[j] = p.beta * cv[j] + p.alpha * acc[i][j];
    // formed before the first store: otherwise each value is computed inside its store's
    // branch, behind a wait for every earlier store
#pragma unroll
    for (int j = 0; j < 8; j += 2) asm volatile("" : "+v"(cv[j]), "+v"(cv[j + 1]));
    if (row < p.M) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (c0 + 8 * j < p.N) p.C[row * p.ldc + c0 + 8 * j] = cv[j];
    }
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

// out[r * ld_out + c] = code[r][c] - zero[r] as bf16 (small integers, exact) for r < rows,
// c < cols; every other entry of the rows_out x ld_out plane is 0.  ld_out is a multiple
// of 16; one thread per 16-column group (one packed code word), two 16-byte stores.
__global__ __launch_bounds__(256) void k_dequant(const uint32_t* __restrict__ codes,
                                                 const float* __restrict__ zero, int64_t rows,
                                                 int64_t cols, u16* __restrict__ out,
                                                 int64_t ld_out, int64_t rows_out) {
  const int64_t nw = (cols + 15) / 16;     // packed words per code row
  const int64_t gw = ld_out / 16;          // 16-column groups per output row
  const int64_t total = rows_out * gw;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * 256) {
    const int64_t r = e / gw, w = e - r * gw;
    uint32_t h[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) h[k] = 0;
    if (r < rows && w < nw) {
      const uint32_t word = codes[r * nw + w];
      const float z = zero[r];
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const float v = (float)((word >> (2 * k)) & 3u) - z;   // small integer, exact in bf16
        h[k] = (w * 16 + k < cols) ? (__float_as_uint(v) >> 16) : 0u;
      }
    }
    u16* dst = out + r * ld_out + w * 16;
    *reinterpret_cast<uint4*>(dst) = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16),
                                                h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    *reinterpret_cast<uint4*>(dst + 8) = make_uint4(h[8] | (h[9] << 16), h[10] | (h[11] << 16),
                                                    h[12] | (h[13] << 16), h[14] | (h[15] << 16));
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

// Lower Cholesky factor in place, in panels of CHOL_PANEL columns: inside a panel each
// 64-column block column is one k_chol_block launch (left-looking over the panel's earlier
// columns, the diagonal block factored in every work-group, the rows below solved through
// the block's inverse); after a panel the trailing matrix right of it receives one
// rank-CHOL_PANEL update.  Entries above the diagonal inside the trailing matrix pick up
// finite values that are never read.
#ifndef FQ_CHOL_PANEL
#define FQ_CHOL_PANEL 128
#endif
constexpr int64_t CHOL_PANEL = FQ_CHOL_PANEL;

namespace {
// Auxiliary stream and events of the look-ahead factorization, one set per device, made on
// first use (default priority).  The mutex also keeps the event records and waits of one
// factorization from interleaving with another's.
struct CholAux {
  hipStream_t s2 = nullptr;
  hipEvent_t chain = nullptr, upd = nullptr;
  bool ok = false, init = false;
};
std::mutex g_chol_mu;
CholAux g_chol_aux[64];

CholAux* chol_aux() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  CholAux& a = g_chol_aux[dev];
  if (!a.init) {
    a.init = true;
    a.ok = hipStreamCreateWithFlags(&a.s2, hipStreamNonBlocking) == hipSuccess &&
           hipEventCreateWithFlags(&a.chain, hipEventDisableTiming) == hipSuccess &&
           hipEventCreateWithFlags(&a.upd, hipEventDisableTiming) == hipSuccess;
  }
  return a.ok ? &a : nullptr;
}
}  // namespace

hipError_t q_cholesky(double* A, int64_t K, double* Lslots, int* flags, hipStream_t s) {
  std::lock_guard<std::mutex> lock(g_chol_mu);
  // under the kernel timer every part runs on the caller's stream (timed intervals must
  // not overlap)
  CholAux* aux = prof_enabled() ? nullptr : chol_aux();
  bool pending = false;            // a trailing update is in flight on the auxiliary stream
  int64_t nblk = 0, kp0 = 0;       // blocks launched; the previous block's column and width
  int kpb = 0;
  for (int64_t j0 = 0; j0 < K; j0 += CHOL_PANEL) {
    const int64_t jb = std::min<int64_t>(CHOL_PANEL, K - j0);
    for (int64_t k0 = j0; k0 < j0 + jb; k0 += CB) {
      const int kb = (int)std::min<int64_t>(CB, j0 + jb - k0);
      // one work-group per slab of 64 rows below, at most 255 (more slabs are dealt round
      // robin): every work-group factors the diagonal block, so more than one round of
      // work-groups per compute unit would repeat that latency
      const int64_t below = K - k0 - kb;
      const unsigned grid = (unsigned)(1 + std::min<int64_t>((below + CB - 1) / CB, 255));
      double* Lout = Lslots + (nblk & 1) * CB * CB;
      const double* Lprev = nblk > 0 ? Lslots + ((nblk - 1) & 1) * CB * CB : nullptr;
      prof_begin(s, "chol_block");
      hipLaunchKernelGGL(k_chol_block, dim3(grid), dim3(256), 0, s, A, K, K, j0, k0, kb, Lout,
                         Lprev, kp0, kpb, flags);
      prof_end(s);
      ++nblk;
      kp0 = k0;
      kpb = kb;
    }
    // rank-jb update of the trailing matrix right of the panel, in two parts (look-ahead):
    // (a) the next panel's columns, on this stream, which the next panel's factorization
    //     needs; (b) everything right of the next panel, on the auxiliary stream, beside
    //     the next panel's factorization (which touches only its own columns).  (a) of the
    //     next panel waits for (b) of this one, which updated the same columns.
    const int64_t j1 = j0 + jb;
    const int64_t rest = K - j1;
    if (rest <= 0) continue;
    const int64_t jb1 = std::min<int64_t>(CHOL_PANEL, rest);
    const int64_t j2 = j1 + jb1, rest2 = K - j2;
    hipError_t e;
    if (aux && pending) {
      if ((e = hipStreamWaitEvent(s, aux->upd, 0)) != hipSuccess) return e;
      pending = false;
    }
    // (a): rows j1.., columns [j1, j2) (a full rectangle: the upper triangle of the next
    // diagonal block is never read), on 32 x 32 tiles while 64 x 64 ones would leave
    // compute units idle (it is on the chain of dependent launches)
    const double* Pa = A + j1 * K + j0;
    const int tile_a = ((rest + 63) / 64) * ((jb1 + 63) / 64) < 256 ? 32 : 64;
    e = dgemm(rest, jb1, jb, -1.0, 1.0, Pa, K, Pa, K, true, A + j1 * K + j1, K, false, s,
              "chol_syrk", tile_a);
    if (e != hipSuccess) return e;
    if (rest2 <= 0) continue;
    // (b): rows j2.., columns [j2, K), tiles on or below the diagonal (the LDS-ring kernel
    // where its layout rules hold and the matrix is large enough to fill the device)
    const double* Pb = A + j2 * K + j0;
    const int tile_b = rest2 >= 384 ? 0 : 64;
    hipStream_t sb = s;
    if (aux) {
      if ((e = hipEventRecord(aux->chain, s)) != hipSuccess) return e;
      if ((e = hipStreamWaitEvent(aux->s2, aux->chain, 0)) != hipSuccess) return e;
      sb = aux->s2;
    }
    e = dgemm(rest2, rest2, jb, -1.0, 1.0, Pb, K, Pb, K, true, A + j2 * K + j2, K, true, sb,
              "chol_syrk", tile_b);
    if (e != hipSuccess) return e;
    if (aux) {
      if ((e = hipEventRecord(aux->upd, aux->s2)) != hipSuccess) return e;
      pending = true;
    }
  }
  if (aux && pending) {
    hipError_t e = hipStreamWaitEvent(s, aux->upd, 0);
    if (e != hipSuccess) return e;
  }
  if (nblk > 0) {
    prof_begin(s, "chol_block");
    hipLaunchKernelGGL(k_chol_last, dim3(1), dim3(256), 0, s, A, K,
                       Lslots + ((nblk - 1) & 1) * CB * CB, kp0, kpb);
    prof_end(s);
  }
  return last_launch_error();
}

hipError_t q_reverse_upper(const double* A, int64_t K, double* R, double* inv_rdiag,
                           hipStream_t s) {
  prof_begin(s, "q_reverse");
  hipLaunchKernelGGL(k_rev_diag, dim3(grid_for(K, 256)), dim3(256), 0, s, A, K, inv_rdiag);
  hipLaunchKernelGGL(k_reverse_upper, dim3(grid_for(K, 1)), dim3(256), 0, s, A, K, inv_rdiag, R);
  prof_end(s);
  return last_launch_error();
}

hipError_t q_clip_grid(const float* D, int64_t rows, int64_t cols, int bits, QuantScratch& w,
                       float* scale, float* zero, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  prof_begin(s, "q_clip_grid");
  hipLaunchKernelGGL(k_clip_grid, dim3(rows), dim3(256), 0, s, D, cols, (1 << bits) - 1, w.scal,
                     w.Y, scale, zero, w.scale64, w.zero64);
  prof_end(s);
  return last_launch_error();
}

hipError_t q_gptq_block(const float* D, int64_t rows, int64_t cols, int i1, int i2, int o1,
                        int cw, int64_t ld_res, int bits, QuantScratch& w, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  prof_begin(s, "gptq_block");
  hipLaunchKernelGGL(k_gptq_block, dim3(grid_for(rows, GROWS, 1 << 30)), dim3(GTH), 0, s, D, rows,
                     cols, i1, i2 - i1, (int64_t)(i1 - o1), cw, ld_res, (1 << bits) - 1, w.scal,
                     w.dead, w.R, w.scale64, w.zero64, w.Y, w.codes8, w.res);
  prof_end(s);
  return last_launch_error();
}

hipError_t dgemm(int64_t M, int64_t N, int64_t K, double alpha, double beta, const double* A,
                 int64_t lda, const double* B, int64_t ldb, bool b_trans, double* C, int64_t ldc,
                 bool lower_only, hipStream_t s, const char* name, int tile) {
  if (M <= 0 || N <= 0) return hipSuccess;
  DgemmArgs p;
  p.M = M; p.N = N; p.K = K < 0 ? 0 : K;
  p.alpha = alpha; p.beta = beta;
  p.A = A; p.lda = lda; p.B = B; p.ldb = ldb; p.C = C; p.ldc = ldc;
  p.b_trans = (int)b_trans;
  p.lower_only = (int)lower_only;
  p.b16 = ((reinterpret_cast<uintptr_t>(B) & 15) == 0) && ldb % 2 == 0;
  // row-major operands, K a multiple of 16, 16-byte aligned A rows and 32-bit copy
  // offsets: the LDS-ring kernel
  // b_trans: op(B) rows are B's rows, copied in 16-byte pieces like A's (16-byte aligned);
  // lower_only: square C, tiles on or below the diagonal
  const bool ring_ok = K > 0 && K % RK == 0 && (!lower_only || (b_trans && M == N)) &&
                       (reinterpret_cast<uintptr_t>(A) & 15) == 0 && lda % 2 == 0 &&
                       (b_trans ? ((reinterpret_cast<uintptr_t>(B) & 15) == 0 && ldb % 2 == 0 &&
                                   (int64_t)(RT - 1) * ldb * 8 + RK * 8 < ((int64_t)1 << 31))
                                : ((reinterpret_cast<uintptr_t>(B) & 7) == 0 &&
                                   (int64_t)(RK - 1) * ldb * 8 + RT * 8 < ((int64_t)1 << 31))) &&
                       (int64_t)(RT - 1) * lda * 8 + RK * 8 < ((int64_t)1 << 31);
  if (ring_ok && tile == 0) {
    const int64_t tm_ = (M + RT - 1) / RT;
    p.tiles_n = (int)((N + RT - 1) / RT);
    const int64_t g = lower_only ? tm_ * (tm_ + 1) / 2 : tm_ * p.tiles_n;
    prof_begin(s, name);
    if (!b_trans)
      hipLaunchKernelGGL((k_dgemm_ring<false, false>), dim3((unsigned)g), dim3(64 * RWAVES), 0, s, p);
    else if (!lower_only)
      hipLaunchKernelGGL((k_dgemm_ring<true, false>), dim3((unsigned)g), dim3(64 * RWAVES), 0, s, p);
    else
      hipLaunchKernelGGL((k_dgemm_ring<true, true>), dim3((unsigned)g), dim3(64 * RWAVES), 0, s, p);
    prof_end(s);
    return last_launch_error();
  }
  const int DT = tile == 128 ? 128 : tile == 32 ? 32 : 64;
  const int tiles_m = (int)((M + DT - 1) / DT), tiles_n = (int)((N + DT - 1) / DT);
  p.tiles_n = tiles_n;
  const int64_t grid = lower_only ? (int64_t)tiles_m * (tiles_m + 1) / 2 : (int64_t)tiles_m * tiles_n;
  prof_begin(s, name);
  if (DT == 128) hipLaunchKernelGGL(k_dgemm<128>, dim3((unsigned)grid), dim3(256), 0, s, p);
  else if (DT == 32 && !lower_only && p.K <= (int64_t)DK * PF_STEPS)
    hipLaunchKernelGGL(k_dgemm32_short, dim3((unsigned)grid), dim3(256), 0, s, p);
  else if (DT == 32) hipLaunchKernelGGL(k_dgemm<32>, dim3((unsigned)grid), dim3(256), 0, s, p);
  else hipLaunchKernelGGL(k_dgemm<64>, dim3((unsigned)grid), dim3(256), 0, s, p);
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
                        u16* out, int64_t ld_out, int64_t rows_out, hipStream_t s) {
  if (rows_out < rows) rows_out = rows;
  if (ld_out % 16 != 0 || ld_out < cols) return hipErrorInvalidValue;
  const int64_t nw = rows_out * (ld_out / 16);
  if (nw <= 0) return hipSuccess;
  prof_begin(s, "dequant");
  hipLaunchKernelGGL(k_dequant, dim3(grid_for(nw, 256)), dim3(256), 0, s, codes, zero, rows, cols,
                     out, ld_out, rows_out);
  prof_end(s);
  return last_launch_error();
}

}  // namespace fq
