// Diagonal Wiener filter at synthesis: the per-row dot products of the gains
//   g_i = (D H~ D^^T)_ii / (D^ H~ D^^T)_ii,  D^ = diag(scale) Q',  Q' = codes - zero,
// from E = Q' H~ (formed beforehand on the bf16 MFMA engine): with D^ H~ = diag(scale) E,
// g_i = (D_i . E_i) / (scale_i (Q'_i . E_i)).  One work-group per row, fp64 sums.
#include "fq_internal.h"

namespace fq {
namespace {

constexpr int WT = 256;

__device__ __forceinline__ double shfl_xor_d(double v, int m) {
  const long long b = __double_as_longlong(v);
  const int lo = __shfl_xor((int)(b & 0xffffffffll), m, 64);
  const int hi = __shfl_xor((int)(b >> 32), m, 64);
  return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

// D: K_out x K_in fp32 (row stride K_in); E: same; Q: bf16 plane, row stride ldq.
__global__ __launch_bounds__(WT) void k_wiener_rows(const float* __restrict__ D,
                                                    const float* __restrict__ E,
                                                    const u16* __restrict__ Q, int64_t ldq,
                                                    int64_t K_in, const float* scale,
                                                    float* __restrict__ gain, float* scale_out) {
  __shared__ double sn[WT / 64], sd[WT / 64];
  const int64_t i = blockIdx.x;
  const float* d = D + i * K_in;
  const float* e = E + i * K_in;
  const u16* q = Q + i * ldq;
  double num = 0.0, den = 0.0;
  for (int64_t j = threadIdx.x; j < K_in; j += WT) {
    const double ev = (double)e[j];
    num = fma((double)d[j], ev, num);
    den = fma((double)__uint_as_float((uint32_t)q[j] << 16), ev, den);
  }
  for (int m = 32; m > 0; m >>= 1) {
    num += shfl_xor_d(num, m);
    den += shfl_xor_d(den, m);
  }
  if ((threadIdx.x & 63) == 0) {
    sn[threadIdx.x >> 6] = num;
    sd[threadIdx.x >> 6] = den;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double n = 0.0, dd = 0.0;
    for (int w = 0; w < WT / 64; ++w) {
      n += sn[w];
      dd += sd[w];
    }
    const double s = (double)scale[i];
    const double g = (dd != 0.0) ? n / (s * dd) : 1.0;
    gain[i] = (float)g;
    if (scale_out) scale_out[i] = (float)(g * s);
  }
}

}  // namespace

hipError_t wiener_rows(const float* D, const float* E, const u16* Q, int64_t ldq, int64_t K_out,
                       int64_t K_in, const float* scale, float* gain, float* scale_out,
                       hipStream_t s) {
  if (K_out <= 0) return hipSuccess;
  prof_begin(s, "wiener_rows");
  hipLaunchKernelGGL(k_wiener_rows, dim3((unsigned)K_out), dim3(WT), 0, s, D, E, Q, ldq, K_in,
                     scale, gain, scale_out);
  prof_end(s);
  return last_launch_error();
}

}  // namespace fq
