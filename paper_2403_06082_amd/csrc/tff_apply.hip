// Tight fusion frames applied from their construction instead of a dense d x K matrix
// (Sec. 2.2 "Constructing TFFs" and the appendix "Synopsis of Construction of Tight Fusion
// Frames"; the appendix "Computational Complexity during Inference" counts the cost of
// this route).
//
// The frame is P = (R1 (x) R2) T / sqrt(k) (a Parseval frame), with
//  - T's column block s (rho columns, s < k) the realification of subspace s of a complex
//    (k, rho/2, d/2) frame: row c of the base frame F (c < rho/2) is 1 on the complex
//    coordinates [c m, (c + 1) m), m = d / rho (spectral tetris when d / rho is an integer),
//    modulated by w^(j s), w = exp(2 pi i / k); complex coordinate j is the real pair
//    (2j, 2j+1), complex column c the real pair (2c, 2c+1);
//  - R1 (x) R2 the rotation: a vector of length d read row-major as a d1 x d2 matrix M is
//    mapped to R1 M R2^T.
// Analysis (u = P^T x): z = complex form of R1^T M R2, then
//   u[s rho + 2c] + i u[s rho + 2c + 1] = k^(-1/2) sum_{j < m} conj(w^((c m + j) s)) z[c m + j],
// a length-k DFT of each zero-padded m-block.  Synthesis (y = P v) is its adjoint:
//   z[c m + j] = k^(-1/2) sum_{s < k} w^((c m + j) s) (v[s rho + 2c] + i v[s rho + 2c + 1]),
// then y = R1 Z R2^T.  Work per vector: d (d1 + d2) + 2 d k FMAs instead of d k rho.
#include "fq_internal.h"

#include <algorithm>
#include <cmath>

namespace fq {
namespace {

constexpr int TT = 256;
constexpr int RT = 1024;       // threads of a rotation work-group

template <typename T>
__device__ __forceinline__ float ld_f32(const T* p);
template <>
__device__ __forceinline__ float ld_f32<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ld_f32<uint16_t>(const uint16_t* p) {   // bf16
  return __uint_as_float((uint32_t)*p << 16);
}
template <>
__device__ __forceinline__ float ld_f32<_Float16>(const _Float16* p) { return (float)*p; }

// tws[t] = exp(2 pi i t / k) for t < k, into LDS (fp32 sincospif of 2t/k: phase error
// below 4e-7 rad)
__device__ __forceinline__ void load_twiddles(float2* tws, int k) {
  for (int t = threadIdx.x; t < k; t += TT) {
    float sn, cs;
    sincospif(2.0f * (float)t / (float)k, &sn, &cs);
    tws[t] = make_float2(cs, sn);
  }
}

// out[t] = A M[t] R on the d1 x d2 row-major view of each vector, with A(a, i) = L[a][i]
// (L[i][a] when TL).  grid (n * d1): a work-group owns row a of the result for one vector:
// first z = row a of A M (d2 values, LDS), then z R.  Each dot product is split over
// G = 1024 / d2 threads (1 when d2 > 1024) whose partials meet in LDS in a fixed order; the
// loads of M and R are contiguous across lanes, those of L uniform.  in rows at stride
// ldin, out rows at stride ldout.  Dynamic LDS: (d2 + G d2) floats.
template <typename XT, bool TL>
__global__ __launch_bounds__(RT) void k_rotate(const XT* __restrict__ in, int64_t ldin,
                                               const float* __restrict__ L,
                                               const float* __restrict__ R, int d1, int d2,
                                               float* __restrict__ out, int64_t ldout) {
  extern __shared__ float rsh[];
  const int64_t t = blockIdx.x / d1;
  const int a = (int)(blockIdx.x - t * d1);
  const int G = d2 < RT ? RT / d2 : 1;
  float* z = rsh;
  float* red = rsh + d2;
  const XT* x = in + t * ldin;
  for (int e = threadIdx.x; e < G * d2; e += RT) {
    const int g = e / d2, j = e - g * d2;
    float acc = 0.f;
#pragma unroll 8
    for (int i = g; i < d1; i += G) {
      const float l = TL ? L[(int64_t)i * d1 + a] : L[(int64_t)a * d1 + i];
      acc = fmaf(l, ld_f32<XT>(x + (int64_t)i * d2 + j), acc);
    }
    red[e] = acc;
  }
  __syncthreads();
  for (int j = threadIdx.x; j < d2; j += RT) {
    float acc = 0.f;
    for (int g = 0; g < G; ++g) acc += red[g * d2 + j];
    z[j] = acc;
  }
  __syncthreads();
  float* o = out + t * ldout + (int64_t)a * d2;
  for (int e = threadIdx.x; e < G * d2; e += RT) {
    const int g = e / d2, b = e - g * d2;
    float acc = 0.f;
#pragma unroll 8
    for (int j = g; j < d2; j += G) acc = fmaf(z[j], R[(int64_t)j * d2 + b], acc);
    red[e] = acc;
  }
  __syncthreads();
  for (int b = threadIdx.x; b < d2; b += RT) {
    float acc = 0.f;
    for (int g = 0; g < G; ++g) acc += red[g * d2 + b];
    o[b] = acc;
  }
}

// Rt = R^T for a d2 x d2 matrix, through 32 x 32 LDS tiles.  grid (ceil(d2/32)^2).
__global__ __launch_bounds__(TT) void k_transpose(const float* __restrict__ R, int d2,
                                                  float* __restrict__ Rt) {
  __shared__ float tile[32][33];
  const int nb = (d2 + 31) / 32;
  const int bi = blockIdx.x / nb, bj = blockIdx.x - bi * nb;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;       // 8 rows per pass
  for (int r = ty; r < 32; r += 8) {
    const int i = bi * 32 + r, j = bj * 32 + tx;
    tile[r][tx] = (i < d2 && j < d2) ? R[(int64_t)i * d2 + j] : 0.f;
  }
  __syncthreads();
  for (int r = ty; r < 32; r += 8) {
    const int i = bj * 32 + r, j = bi * 32 + tx;
    if (i < d2 && j < d2) Rt[(int64_t)i * d2 + j] = tile[tx][r];
  }
}

// Analysis DFT step.  grid (n * ceil(k / 16), rho / 2): work-group (t, s-block, c); its
// 256 threads are 16 values of s times 16 groups of the m terms, whose partials meet in LDS
// in a fixed order.  Twiddles and the m-block of z sit in LDS (dynamic, (k + m) float2).
// Work-group (t, 0, 0) also zeroes U[t][k rho .. ldu).
__global__ __launch_bounds__(TT) void k_tff_analysis(const float* __restrict__ y, int64_t d,
                                                     int k, int rho, int m, float scale,
                                                     float* __restrict__ U, int64_t ldu) {
  extern __shared__ float2 sh[];
  __shared__ float2 red[16][16];
  const int nsb = (k + 15) / 16;
  const int64_t t = blockIdx.x / nsb;
  const int sb = (int)(blockIdx.x - t * nsb);
  const int c = blockIdx.y;
  float2* tws = sh;
  float2* zs = sh + k;
  load_twiddles(tws, k);
  const float2* yz = reinterpret_cast<const float2*>(y + t * d) + (int64_t)c * m;
  for (int i = threadIdx.x; i < m; i += TT) zs[i] = yz[i];
  __syncthreads();
  const int sl = threadIdx.x & 15, g = threadIdx.x >> 4;
  const int s = sb * 16 + sl;
  const int per = (m + 15) / 16;
  const int j0 = g * per, j1 = min(m, j0 + per);
  float re = 0.f, im = 0.f;
  if (s < k && j0 < j1) {
    int idx = (int)((((int64_t)c * m + j0) % k) * s % k);
#pragma unroll 4
    for (int j = j0; j < j1; ++j) {
      const float2 w = tws[idx], z = zs[j];
      re = fmaf(w.x, z.x, fmaf(w.y, z.y, re));       // conj(w) z
      im = fmaf(w.x, z.y, fmaf(-w.y, z.x, im));
      idx += s;
      if (idx >= k) idx -= k;
    }
  }
  red[g][sl] = make_float2(re, im);
  __syncthreads();
  if (threadIdx.x < 16 && s < k) {
    float sr = 0.f, si = 0.f;
    for (int q = 0; q < 16; ++q) { sr += red[q][sl].x; si += red[q][sl].y; }
    *reinterpret_cast<float2*>(U + t * ldu + (int64_t)s * rho + 2 * c) =
        make_float2(scale * sr, scale * si);
  }
  if (c == 0 && sb == 0)
    for (int64_t j = (int64_t)k * rho + threadIdx.x; j < ldu; j += TT) U[t * ldu + j] = 0.f;
}

// Synthesis DFT step.  grid (n * ceil(m / 16), rho / 2): work-group (t, j-block, c); its
// 256 threads are 16 values of j times 16 groups of the k terms, whose partials meet in LDS
// in a fixed order.  Twiddles and the k values of column pair c sit in LDS (dynamic, 2k
// float2).  Z contiguous (d per vector).
__global__ __launch_bounds__(TT) void k_tff_synthesis(const float* __restrict__ V, int64_t ldv,
                                                      int k, int rho, int m, int64_t d,
                                                      float scale, float* __restrict__ Z) {
  extern __shared__ float2 sh[];
  __shared__ float2 red[16][16];
  const int njb = (m + 15) / 16;
  const int64_t t = blockIdx.x / njb;
  const int jb = (int)(blockIdx.x - t * njb);
  const int c = blockIdx.y;
  float2* tws = sh;
  float2* nus = sh + k;
  load_twiddles(tws, k);
  for (int i = threadIdx.x; i < k; i += TT)
    nus[i] = *reinterpret_cast<const float2*>(V + t * ldv + (int64_t)i * rho + 2 * c);
  __syncthreads();
  const int jl = threadIdx.x & 15, g = threadIdx.x >> 4;
  const int j = jb * 16 + jl;
  const int per = (k + 15) / 16;
  const int s0 = g * per, s1 = min(k, s0 + per);
  const int64_t jj = (int64_t)c * m + j;
  float re = 0.f, im = 0.f;
  if (j < m && s0 < s1) {
    const int step = (int)(jj % k);
    int idx = (int)((int64_t)step * s0 % k);
#pragma unroll 4
    for (int s = s0; s < s1; ++s) {
      const float2 w = tws[idx], v = nus[s];
      re = fmaf(w.x, v.x, fmaf(-w.y, v.y, re));      // w v
      im = fmaf(w.x, v.y, fmaf(w.y, v.x, im));
      idx += step;
      if (idx >= k) idx -= k;
    }
  }
  red[g][jl] = make_float2(re, im);
  __syncthreads();
  if (threadIdx.x < 16 && j < m) {
    float sr = 0.f, si = 0.f;
    for (int q = 0; q < 16; ++q) { sr += red[q][jl].x; si += red[q][jl].y; }
    *reinterpret_cast<float2*>(Z + t * d + 2 * jj) = make_float2(scale * sr, scale * si);
  }
}

unsigned blocks_for(int64_t total) { return (unsigned)((total + TT - 1) / TT); }

size_t rot_lds(int d2) { return (size_t)(d2 + (d2 < RT ? RT / d2 : 1) * d2) * sizeof(float); }

// Columns c0 .. c0 + nc - 1 of T / sqrt(k) as rows of Z (nc x d, complex pairs): column
// s rho + 2c + e is zero outside the m-block c, where complex coordinate c m + j holds
// k^(-1/2) w^((c m + j) s) (e = 0) or i k^(-1/2) w^((c m + j) s) (e = 1).  One thread per
// complex coordinate; the phase index (c m + j) s mod k is exact in 64-bit integers.
__global__ __launch_bounds__(TT) void k_tff_columns(int64_t c0, int64_t nc, int64_t d, int k,
                                                    int rho, int m, float scale,
                                                    float* __restrict__ Z) {
  const int64_t dc = d / 2;
  const int64_t e = (int64_t)blockIdx.x * TT + threadIdx.x;
  if (e >= nc * dc) return;
  const int64_t r = e / dc, j = e - r * dc;
  const int64_t col = c0 + r;
  const int64_t sidx = col / rho;
  const int within = (int)(col - sidx * rho), c = within >> 1, odd = within & 1;
  float2 v = make_float2(0.f, 0.f);
  if (j / m == c) {
    const int64_t t = (j % k) * (sidx % k) % k;
    float sn, cs;
    sincospif(2.0f * (float)t / (float)k, &sn, &cs);
    v = odd ? make_float2(-sn * scale, cs * scale) : make_float2(cs * scale, sn * scale);
  }
  *reinterpret_cast<float2*>(Z + r * d + 2 * j) = v;
}

// P[i][c0 + r] = Pt[r][i] for r < nc, i < d: 32 x 32 tiles through LDS.
// grid (ceil(nc / 32) * ceil(d / 32)).
__global__ __launch_bounds__(TT) void k_scatter_columns(const float* __restrict__ Pt, int64_t nc,
                                                        int64_t d, float* __restrict__ P,
                                                        int64_t ldp, int64_t c0) {
  __shared__ float tile[32][33];
  const int64_t nbi = (d + 31) / 32;
  const int64_t br = blockIdx.x / nbi, bi = blockIdx.x - br * nbi;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int q = ty; q < 32; q += 8) {
    const int64_t r = br * 32 + q, i = bi * 32 + tx;
    tile[q][tx] = (r < nc && i < d) ? Pt[r * d + i] : 0.f;
  }
  __syncthreads();
  for (int q = ty; q < 32; q += 8) {
    const int64_t i = bi * 32 + q, r = br * 32 + tx;
    if (i < d && r < nc) P[i * ldp + c0 + r] = tile[tx][q];
  }
}

}  // namespace

hipError_t tff_analysis(const void* X, int xt, int64_t ldx, int64_t n, const TffDev& F,
                        float* y, float* U, int64_t ldu, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const dim3 gr((unsigned)(n * F.d1));
  const size_t lds = rot_lds(F.d2);
  prof_begin(s, "tff_rotate");
  if (xt == 0)
    hipLaunchKernelGGL((k_rotate<float, true>), gr, dim3(RT), lds, s, (const float*)X, ldx, F.R1, F.R2, F.d1, F.d2, y, F.d);
  else if (xt == 1)
    hipLaunchKernelGGL((k_rotate<_Float16, true>), gr, dim3(RT), lds, s, (const _Float16*)X, ldx, F.R1, F.R2, F.d1, F.d2, y, F.d);
  else
    hipLaunchKernelGGL((k_rotate<uint16_t, true>), gr, dim3(RT), lds, s, (const uint16_t*)X, ldx, F.R1, F.R2, F.d1, F.d2, y, F.d);
  prof_end(s);
  prof_begin(s, "tff_dft");
  const dim3 ga((unsigned)(n * ((F.k + 15) / 16)), (unsigned)(F.rho / 2));
  hipLaunchKernelGGL(k_tff_analysis, ga, dim3(TT), (size_t)(F.k + F.m) * sizeof(float2), s, y, F.d,
                     (int)F.k, (int)F.rho, (int)F.m, (float)(1.0 / std::sqrt((double)F.k)), U, ldu);
  prof_end(s);
  return last_launch_error();
}

hipError_t tff_transpose_r2(const TffDev& F, float* R2t, hipStream_t s) {
  const int nb = (F.d2 + 31) / 32;
  prof_begin(s, "tff_rotate");
  hipLaunchKernelGGL(k_transpose, dim3((unsigned)(nb * nb)), dim3(TT), 0, s, F.R2, F.d2, R2t);
  prof_end(s);
  return last_launch_error();
}

hipError_t tff_synthesis(const float* V, int64_t ldv, int64_t n, const TffDev& F,
                         const float* R2t, float* z, float* Y, int64_t ldy, hipStream_t s) {
  if (n == 0) return hipSuccess;
  prof_begin(s, "tff_dft");
  const dim3 gs((unsigned)(n * ((F.m + 15) / 16)), (unsigned)(F.rho / 2));
  hipLaunchKernelGGL(k_tff_synthesis, gs, dim3(TT), (size_t)(2 * F.k) * sizeof(float2), s, V, ldv,
                     (int)F.k, (int)F.rho, (int)F.m, F.d, (float)(1.0 / std::sqrt((double)F.k)), z);
  prof_end(s);
  const dim3 gr((unsigned)(n * F.d1));
  prof_begin(s, "tff_rotate");
  hipLaunchKernelGGL((k_rotate<float, false>), gr, dim3(RT), rot_lds(F.d2), s,
                     (const float*)z, F.d, F.R1, R2t, F.d1, F.d2, Y, ldy);
  prof_end(s);
  return last_launch_error();
}

hipError_t tff_materialize(const TffDev& F, const float* R2t, float* Z, float* Pt, int64_t nc_max,
                           float* P, int64_t ldp, hipStream_t s) {
  const int64_t K = F.k * F.rho;
  const float scale = (float)(1.0 / std::sqrt((double)F.k));
  for (int64_t c0 = 0; c0 < K; c0 += nc_max) {
    const int64_t nc = std::min(nc_max, K - c0);
    prof_begin(s, "tff_columns");
    hipLaunchKernelGGL(k_tff_columns, dim3(blocks_for(nc * (F.d / 2))), dim3(TT), 0, s, c0, nc, F.d,
                       (int)F.k, (int)F.rho, (int)F.m, scale, Z);
    prof_end(s);
    prof_begin(s, "tff_rotate");
    hipLaunchKernelGGL((k_rotate<float, false>), dim3((unsigned)(nc * F.d1)), dim3(RT), rot_lds(F.d2), s,
                       (const float*)Z, F.d, F.R1, R2t, F.d1, F.d2, Pt, F.d);
    prof_end(s);
    prof_begin(s, "tff_columns");
    const int64_t g = ((nc + 31) / 32) * ((F.d + 31) / 32);
    hipLaunchKernelGGL(k_scatter_columns, dim3((unsigned)g), dim3(TT), 0, s, Pt, nc, F.d, P, ldp, c0);
    prof_end(s);
  }
  return last_launch_error();
}

}  // namespace fq
