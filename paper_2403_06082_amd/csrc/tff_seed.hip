// Rotation factors of a frame drawn on the device from a 64-bit seed (Sec. 2.2 and the
// appendix on constructing TFFs take a random rotation; the storage appendix keeps only
// (k, rho, d) and what regenerates the rotation).  The paper names no generator; the
// recipe here:
//  * Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11): key = (seed mod 2^32,
//    seed div 2^32), counter = (p mod 2^32, p div 2^32, f, 0) for pair p of factor f;
//  * u1 from output words (x0, x1), u2 from (x2, x3): u = (2^21 x_odd + floor(x_even /
//    2^11) + 1/2) / 2^53, in (0, 1);
//  * Box-Muller: entries 2p, 2p + 1 of the row-major n x n matrix G are
//    sqrt(-2 ln u1) cos(2 pi u2) and sqrt(-2 ln u1) sin(2 pi u2);
//  * the factor is Q of G = Q R with R's diagonal made positive (Householder QR in fp64,
//    then the signs of R's diagonal moved into Q): a Haar-distributed orthogonal matrix.
#include "fq_internal.h"

#include <cmath>

namespace fq {
namespace {

constexpr int ST = 256;

// 10 rounds of Philox4x32 on c with key (k0, k1)
__device__ __forceinline__ void philox10(uint32_t (&c)[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = (uint32_t)p1;
    c[2] = n2;
    c[3] = (uint32_t)p0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

__device__ __forceinline__ double unit53(uint32_t lo, uint32_t hi) {
  const uint64_t m = ((uint64_t)hi << 21) | (lo >> 11);
  return ((double)m + 0.5) * 0x1p-53;
}

// G (n x n, row-major, fp64) of factor f.  One thread per pair of entries.
__global__ __launch_bounds__(ST) void k_seeded_gauss(uint32_t k0, uint32_t k1, uint32_t f,
                                                     int64_t n, double* __restrict__ G) {
  const int64_t total = n * n, npair = (total + 1) / 2;
  for (int64_t p = (int64_t)blockIdx.x * ST + threadIdx.x; p < npair;
       p += (int64_t)gridDim.x * ST) {
    uint32_t c[4] = {(uint32_t)p, (uint32_t)((uint64_t)p >> 32), f, 0u};
    philox10(c, k0, k1);
    const double u1 = unit53(c[0], c[1]), u2 = unit53(c[2], c[3]);
    const double rad = sqrt(-2.0 * log(u1));
    const double th = 2.0 * M_PI * u2;
    G[2 * p] = rad * cos(th);
    if (2 * p + 1 < total) G[2 * p + 1] = rad * sin(th);
  }
}

__device__ __forceinline__ double block_sum(double v, double* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int w = ST / 2; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  const double s = red[0];
  __syncthreads();
  return s;
}

// One work-group: A (n x n, row-major) = G is reduced by Householder reflections
// H_j = I - beta_j v_j v_j^T (v_j kept in column j of V, zero above row j; R_jj = alpha_j),
// then Q = H_0 H_1 ... H_{n-1} is formed in A's storage, applied from the right end to the
// identity, and out = Q diag(sign(alpha)) in fp32.  A thread owns columns tid, tid + 256,
// ...; the reflector of a step sits in LDS.
__global__ __launch_bounds__(ST) void k_haar_qr(double* __restrict__ A, int n,
                                                double* __restrict__ V,
                                                double* __restrict__ ab,
                                                float* __restrict__ out) {
  extern __shared__ double vs[];          // n doubles
  __shared__ double red[ST];
  double* alpha = ab;
  double* beta = ab + n;
  const int tid = threadIdx.x;
  for (int j = 0; j < n; ++j) {
    double s = 0.0;
    for (int r = j + tid; r < n; r += ST) {
      const double x = A[(int64_t)r * n + j];
      s = fma(x, x, s);
    }
    const double nrm2 = block_sum(s, red);
    const double x0 = A[(int64_t)j * n + j];
    const double nrm = sqrt(nrm2);
    const double al = nrm == 0.0 ? 0.0 : (x0 >= 0.0 ? -nrm : nrm);
    const double vj = x0 - al;
    const double vtv = nrm2 - x0 * x0 + vj * vj;
    const double be = vtv > 0.0 ? 2.0 / vtv : 0.0;
    for (int r = j + tid; r < n; r += ST) {
      const double v = r == j ? vj : A[(int64_t)r * n + j];
      vs[r] = v;
      V[(int64_t)r * n + j] = v;
    }
    if (tid == 0) {
      alpha[j] = al;
      beta[j] = be;
    }
    __syncthreads();
    for (int c = j + 1 + tid; c < n; c += ST) {
      double d = 0.0;
      for (int r = j; r < n; ++r) d = fma(vs[r], A[(int64_t)r * n + c], d);
      const double t = be * d;
      for (int r = j; r < n; ++r) A[(int64_t)r * n + c] -= t * vs[r];
    }
    __syncthreads();
  }
  for (int64_t e = tid; e < (int64_t)n * n; e += ST) {
    const int64_t r = e / n, c = e - r * n;
    A[e] = r == c ? 1.0 : 0.0;
  }
  __syncthreads();
  for (int j = n - 1; j >= 0; --j) {
    for (int r = j + tid; r < n; r += ST) vs[r] = V[(int64_t)r * n + j];
    __syncthreads();
    const double be = beta[j];
    for (int c = j + tid; c < n; c += ST) {
      double d = 0.0;
      for (int r = j; r < n; ++r) d = fma(vs[r], A[(int64_t)r * n + c], d);
      const double t = be * d;
      for (int r = j; r < n; ++r) A[(int64_t)r * n + c] -= t * vs[r];
    }
    __syncthreads();
  }
  for (int64_t e = tid; e < (int64_t)n * n; e += ST) {
    const int64_t c = e % n;
    const double sg = alpha[c] < 0.0 ? -1.0 : 1.0;
    out[e] = (float)(A[e] * sg);
  }
}

}  // namespace

hipError_t tff_seeded_factor(uint64_t seed, int f, int n, double* G, double* V, double* ab,
                             float* out, hipStream_t s) {
  const int64_t npair = ((int64_t)n * n + 1) / 2;
  int64_t g = (npair + ST - 1) / ST;
  if (g > 65536) g = 65536;
  prof_begin(s, "tff_seed");
  hipLaunchKernelGGL(k_seeded_gauss, dim3((unsigned)(g > 0 ? g : 1)), dim3(ST), 0, s,
                     (uint32_t)(seed & 0xFFFFFFFFull), (uint32_t)(seed >> 32), (uint32_t)f,
                     (int64_t)n, G);
  hipLaunchKernelGGL(k_haar_qr, dim3(1), dim3(ST), (size_t)n * sizeof(double), s, G, n, V, ab,
                     out);
  prof_end(s);
  return last_launch_error();
}

}  // namespace fq
