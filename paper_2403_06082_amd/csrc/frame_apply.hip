// Layer outputs straight from the stored codes and the two frames: Y = X Theta^T with
// Theta^ = P_out diag(scale) (q - zero) P_in^T (appendix "Computational Complexity during
// Inference"), taken in the order of Sec. 3 "Inference Procedure" (analysis operator on
// the inputs, the quantized D^, synthesis operator):
//   U = X P_in            (tokens x K_in)
//   V = U (q - zero)^T S  (tokens x K_out; the 2-bit codes decoded on the fly)
//   Y = V P_out^T         (tokens x d_out)
// for small token counts (decode, small batches), where every step streams its operand
// from HBM once: P_in (d_in x K_in fp32), the packed codes, P_out (d_out x K_out fp32).
// Tokens go through in blocks of at most 8; all arithmetic is fp32 with fp32
// accumulation (the split-K partials of U are summed in fp64).
#include "fq_internal.h"

#include <algorithm>

namespace fq {
namespace {

constexpr int AT = 256;        // threads per work-group in every kernel here

// Work-group barrier for LDS traffic only: waits for this wave's LDS operations, not for
// its global loads (a fenced __syncthreads would also drain every load in flight).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <typename T>
__device__ __forceinline__ float to_f32(T v);
template <>
__device__ __forceinline__ float to_f32<float>(float v) { return v; }
template <>
__device__ __forceinline__ float to_f32<uint16_t>(uint16_t v) {   // bf16
  return __uint_as_float((uint32_t)v << 16);
}
template <>
__device__ __forceinline__ float to_f32<_Float16>(_Float16 v) { return (float)v; }

// ---- step 1: part[s][t][j] = sum over k in split s of X[t][k] P_in[k][j]
// grid (ceil(K_in / (4 AT)), ksplit); a thread owns 4 consecutive columns.
template <typename XT, int NT, bool VEC>
__global__ __launch_bounds__(AT) void k_apply_in(const XT* __restrict__ X, int64_t ldx, int nt,
                                                 int64_t d_in, const float* __restrict__ P,
                                                 int64_t K_in, int kper,
                                                 float* __restrict__ part) {
  __shared__ float xs[NT][256];
  const int s = blockIdx.y;
  const int64_t k0 = (int64_t)s * kper;
  const int kn = (int)min((int64_t)kper, d_in - k0);
  for (int e = threadIdx.x; e < NT * kper; e += AT) {
    const int t = e / kper, k = e % kper;
    xs[t][k] = (t < nt && k < kn) ? to_f32<XT>(X[t * ldx + k0 + k]) : 0.f;
  }
  __syncthreads();
  const int64_t j = ((int64_t)blockIdx.x * AT + threadIdx.x) * 4;
  if (j >= K_in) return;
  float acc[NT][4];
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q) acc[t][q] = 0.f;
  const float* p = P + k0 * K_in + j;
  for (int k = 0; k < kn; ++k, p += K_in) {
    float v[4];
    if (VEC) {
      const float4 w = *reinterpret_cast<const float4*>(p);
      v[0] = w.x; v[1] = w.y; v[2] = w.z; v[3] = w.w;
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = (j + q < K_in) ? p[q] : 0.f;
    }
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const float x = xs[t][k];
#pragma unroll
      for (int q = 0; q < 4; ++q) acc[t][q] = fmaf(x, v[q], acc[t][q]);
    }
  }
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (j + q < K_in) part[((int64_t)s * NT + t) * K_in + j + q] = acc[t][q];
}

// U[t][j] = sum over the splits (fp64), zero for t >= nt; U has ldu >= K_in columns,
// columns [K_in, ldu) zero.  grid (ldu / 64, NT): a work-group owns 64 columns of one
// token; its 4 waves sum every 4th split and combine through LDS in a fixed order.
__global__ __launch_bounds__(AT) void k_apply_in_reduce(const float* __restrict__ part, int nt_blk,
                                                        int nt, int ksplit, int64_t K_in,
                                                        int64_t ldu, float* __restrict__ U) {
  __shared__ double red[AT / 64][64];
  const int lane = threadIdx.x & 63, g = threadIdx.x >> 6;
  const int t = blockIdx.y;
  const int64_t j = (int64_t)blockIdx.x * 64 + lane;
  double acc = 0.0;
  if (t < nt && j < K_in) {
    const float* p = part + (int64_t)t * K_in + j;
    const int64_t step = (int64_t)nt_blk * K_in;
#pragma unroll 8
    for (int s = g; s < ksplit; s += AT / 64) acc += p[s * step];
  }
  red[g][lane] = acc;
  __syncthreads();
  if (g == 0 && j < ldu)
    U[(int64_t)t * ldu + j] = (float)(red[0][lane] + red[1][lane] + red[2][lane] + red[3][lane]);
}

// ---- step 2: V[t][i] = scale_i (sum_j U[t][j] q_ij - zero_i sum_j U[t][j])
// (the same sum as sum_j U[t][j] (q_ij - zero_i); both forms have error bounds of the
// same size, since |q|, |q - zero| <= 3).  A work-group owns 16 rows (4 per wave); U goes
// through LDS UCH(NT) columns at a time (at most 32 KB), and the work-group sums each token's U
// while staging it.  A lane takes code words w = lane, lane + 64, ... of its wave's 4
// rows; the first chunk's words are loaded right after its U, each later chunk's words one
// chunk ahead, and LDS-only barriers keep them in flight meanwhile.  A word is spread
// into bytes, (word >> 2b) & 0x03030303 holding the codes of columns b, b+4, b+8, b+12,
// and each byte converts to float in one instruction.  In LDS, group g (4 columns) of
// word w sits at group (g + w/2) mod 4 of the word's 16 columns, so that 8 lanes reading
// the same group of consecutive words cover all banks.  BITS = 4: 8 codes per word,
// (word >> 4b) & 0x0F0F0F0F holds the codes of columns 2g + b (byte g), U sits in LDS in
// column order (a word's 8 columns are 32 bytes, so 8 lanes on consecutive words cover
// all banks without the rotation).
template <int NT, int BITS>
__global__ __launch_bounds__(AT) void k_apply_codes(const float* __restrict__ U, int64_t ldu,
                                                    const uint32_t* codes,   // not restrict: its loads must stay before the barriers
                                                    int64_t K_out, int64_t nwords,
                                                    const float* __restrict__ scale,
                                                    const float* __restrict__ zero,
                                                    float* __restrict__ V) {
  // columns per chunk (at most 32 KB of LDS; 2048 for up to 4 tokens keeps the code words
  // of two chunks in registers)
  constexpr int UCH = NT <= 4 ? 2048 : 8192 / NT;
  constexpr int CPW = BITS == 2 ? 16 : 8;    // codes per word
  constexpr int WPL = UCH / (CPW * 64);      // code words per lane and row in a chunk
  constexpr int SPT = UCH / (4 * AT);        // staging rounds per token
  __shared__ __attribute__((aligned(16))) float us[NT][UCH];
  __shared__ float usum_w[AT / 64][NT];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row0 = (int64_t)blockIdx.x * 16 + wave * 4;
  float acc[4][NT], tsum[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    tsum[t] = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[r][t] = 0.f;
  }
  const uint32_t* crow[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) crow[r] = codes + min(row0 + r, K_out - 1) * nwords;
  // code words of a chunk: 4 rows x WPL words per lane (clamped loads, unconditional; with
  // 4-bit codes the padded U row can reach one word past a code row, whose columns carry
  // U = 0, so the index is clamped into the row)
  auto load_words = [&](uint32_t (&dst)[4][WPL], int64_t c0) {
    const int nw = (int)(min((int64_t)UCH, ldu - c0) / CPW);
#pragma unroll
    for (int k = 0; k < WPL; ++k) {
      const int w = lane + 64 * k;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        dst[r][k] = crow[r][min(c0 / CPW + min(w, nw - 1), nwords - 1)];
    }
  };
  uint32_t wd[4][WPL], wn[4][WPL] = {};
  for (int64_t c0 = 0; c0 < ldu; c0 += UCH) {
    const int cn = (int)min((int64_t)UCH, ldu - c0);        // multiple of 16
    const int nw = cn / CPW;
    lds_barrier();                          // the previous chunk's reads of us are done
    float4 uv[NT][SPT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int m = 0; m < SPT; ++m) {
        const int c = (m * AT + (int)threadIdx.x) * 4;   // unconditional load, clamped
        uv[t][m] = *reinterpret_cast<const float4*>(U + t * ldu + c0 + min(c, cn - 4));
      }
    // the first chunk's words are loaded after its U, so that storing U into LDS waits for
    // U alone; later chunks' words were loaded one chunk ahead
    if (c0 == 0) load_words(wd, 0);
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int m = 0; m < SPT; ++m) {
        const int c = (m * AT + (int)threadIdx.x) * 4;
        const uint32_t keep = c < cn ? 0xffffffffu : 0u;      // a mask, not a branch: the
        const float4 u4 = uv[t][m];                            // load stays unconditional
        const float4 v = make_float4(__uint_as_float(__float_as_uint(u4.x) & keep),
                                     __uint_as_float(__float_as_uint(u4.y) & keep),
                                     __uint_as_float(__float_as_uint(u4.z) & keep),
                                     __uint_as_float(__float_as_uint(u4.w) & keep));
        tsum[t] += (v.x + v.y) + (v.z + v.w);
        if constexpr (BITS == 2) {
          const int w = c >> 4, g = (c >> 2) & 3;
          *reinterpret_cast<float4*>(&us[t][16 * w + 4 * ((g + (w >> 1)) & 3)]) = v;
        } else {
          *reinterpret_cast<float4*>(&us[t][c]) = v;
        }
      }
    lds_barrier();
    if (c0 + UCH < ldu) load_words(wn, c0 + UCH);   // in flight during this chunk's work
#pragma unroll
    for (int k = 0; k < WPL; ++k) {
      const int w = lane + 64 * k;
      if (w >= nw) break;
      if constexpr (BITS == 4) {
        uint32_t y[4][2];                     // byte g of y[r][b]: code of column 2g + b
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int b = 0; b < 2; ++b) {
            y[r][b] = (wd[r][k] >> (4 * b)) & 0x0F0F0F0Fu;
            asm volatile("" : "+v"(y[r][b]));
          }
#pragma unroll
        for (int h = 0; h < 2; ++h) {          // columns 4h .. 4h + 3 of the word: bytes 2h, 2h + 1
          float q[4][4];
#pragma unroll
          for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int x = 0; x < 4; ++x)
              q[r][x] = (float)((y[r][x & 1] >> (8 * (2 * h + (x >> 1)))) & 0xffu);
#pragma unroll
          for (int t = 0; t < NT; ++t) {
            const float4 v = *reinterpret_cast<const float4*>(&us[t][8 * w + 4 * h]);
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              acc[r][t] = fmaf(v.x, q[r][0], acc[r][t]);
              acc[r][t] = fmaf(v.y, q[r][1], acc[r][t]);
              acc[r][t] = fmaf(v.z, q[r][2], acc[r][t]);
              acc[r][t] = fmaf(v.w, q[r][3], acc[r][t]);
            }
          }
        }
        continue;
      }
      uint32_t y[4][4];                       // byte g of y[r][b]: code of column 4g + b
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          y[r][b] = (wd[r][k] >> (2 * b)) & 0x03030303u;
          asm volatile("" : "+v"(y[r][b]));   // keep the bytes: one conversion per code
        }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float q[4][4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int b = 0; b < 4; ++b) q[r][b] = (float)((y[r][b] >> (8 * g)) & 0xffu);
        const int pg = (g + (w >> 1)) & 3;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const float4 v = *reinterpret_cast<const float4*>(&us[t][16 * w + 4 * pg]);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            acc[r][t] = fmaf(v.x, q[r][0], acc[r][t]);
            acc[r][t] = fmaf(v.y, q[r][1], acc[r][t]);
            acc[r][t] = fmaf(v.z, q[r][2], acc[r][t]);
            acc[r][t] = fmaf(v.w, q[r][3], acc[r][t]);
          }
        }
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int k = 0; k < WPL; ++k) wd[r][k] = wn[r][k];
  }
  // token sums of U over the work-group, row sums over each wave
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      tsum[t] += __shfl_xor(tsum[t], o);
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r][t] += __shfl_xor(acc[r][t], o);
    }
  }
  if (lane == 0)
#pragma unroll
    for (int t = 0; t < NT; ++t) usum_w[wave][t] = tsum[t];
  __syncthreads();
  if (lane == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t i = row0 + r;
      if (i < K_out) {
        const float s = scale[i], z = zero[i];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const float us_t = (usum_w[0][t] + usum_w[1][t]) + (usum_w[2][t] + usum_w[3][t]);
          V[t * K_out + i] = s * fmaf(-z, us_t, acc[r][t]);
        }
      }
    }
  }
}

// ---- rounded activations (appendix "FrameQuant for Activation Quantization?"): per token
// t, Delta_t = max_j |U[t][j]| / qmax and Cq[t][j] = round(U[t][j] / Delta_t) (IEEE fp32
// divisions, ties to even; Delta_t = 0 gives a zero row).  One 1024-thread work-group per
// token.
// CPW > 0 stores each CPW-column code word's bytes in the order of the spread code words
// (NB = CPW / 4 dwords per word): column CPW w + NB g + b at byte CPW w + 4b + g (columns
// [K, ldc) zero); CPW = 0 stores column j at byte j.
// csum (optional) receives sum_j Cq[t][j].
constexpr int QT = 1024;       // threads per token in the activation rounding kernel

template <int CPW>
__global__ __launch_bounds__(QT) void k_act_quantize(const float* __restrict__ U, int64_t ldu,
                                                     int64_t K, float qmax,
                                                     int8_t* __restrict__ Cq, int64_t ldc,
                                                     float* __restrict__ delta,
                                                     int* __restrict__ csum) {
  __shared__ float wmax[QT / 64];
  __shared__ int wsum[QT / 64];
  const int64_t t = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float* u = U + t * ldu;
  float mx = 0.f;
#pragma unroll 4
  for (int64_t j = threadIdx.x; j < K; j += QT) mx = fmaxf(mx, fabsf(u[j]));
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  if (lane == 0) wmax[wave] = mx;
  __syncthreads();
  mx = 0.f;
#pragma unroll
  for (int w = 0; w < QT / 64; ++w) mx = fmaxf(mx, wmax[w]);
  const float dl = mx / qmax;
  int sum = 0;
#pragma unroll 4
  for (int64_t j = threadIdx.x; j < ldc; j += QT) {
    int q = 0;
    if (j < K && dl > 0.f) q = (int)rintf(u[j] / dl);
    sum += q;
    int64_t dst = j;
    if (CPW > 0) {
      constexpr int NB = CPW > 0 ? CPW / 4 : 1;
      const int r = (int)(j % CPW);
      dst = (j - r) + 4 * (r % NB) + r / NB;
    }
    Cq[t * ldc + dst] = (int8_t)q;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  if (lane == 0) wsum[wave] = sum;
  __syncthreads();
  if (threadIdx.x == 0) {
    delta[t] = dl;
    if (csum) {
      int total = 0;
      for (int w = 0; w < QT / 64; ++w) total += wsum[w];
      csum[t] = total;
    }
  }
}

template <int B> struct CqWord;                         // one code word's Cq bytes
template <> struct CqWord<2> { typedef uint4 type; };   // 16 columns
template <> struct CqWord<4> { typedef uint2 type; };   // 8 columns
__device__ __forceinline__ uint32_t dw(const uint4& d, int b) {
  return b == 0 ? d.x : b == 1 ? d.y : b == 2 ? d.z : d.w;
}
__device__ __forceinline__ uint32_t dw(const uint2& d, int b) { return b == 0 ? d.x : d.y; }

// V[t][i] = scale_i Delta_t (sum_j Cq[t][j] q_ij - zero_i sum_j Cq[t][j]) for BITS-bit codes
// (2 or 4), the dot product exact in int32 (|sum| <= (2^BITS - 1) * 127 * K_in) and
// converted to float at the end.  Same work split as k_apply_codes: 16 rows per
// work-group, 4 per wave, lanes over code words; Cq (layout of k_act_quantize with
// CPW = 32 / BITS, ldc = CPW nwords bytes) goes through LDS CW words at a time, and each
// word's spread codes meet the matching NB = CPW / 4 dwords of Cq in NB v_dot4 per row and
// token.
template <int NT, int BITS>
__global__ __launch_bounds__(AT) void k_apply_codes_i8(const int8_t* __restrict__ Cq,
                                                       int64_t ldc,
                                                       const float* __restrict__ delta,
                                                       const int* __restrict__ csum,
                                                       const uint32_t* codes, int64_t K_out,
                                                       int64_t nwords,
                                                       const float* __restrict__ scale,
                                                       const float* __restrict__ zero,
                                                       float* __restrict__ V) {
  typedef typename CqWord<BITS>::type WT;
  constexpr int CPW = 32 / BITS, NB = CPW / 4;
  constexpr uint32_t MASK = BITS == 2 ? 0x03030303u : 0x0F0F0F0Fu;
  constexpr int CW = NT >= 8 ? 128 : 256;    // words per chunk (NT * CW * CPW bytes <= 16 KB)
  constexpr int WPL = CW / 64;               // code words per lane and row in a chunk
  __shared__ WT cs[NT][CW];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t row0 = (int64_t)blockIdx.x * 16 + wave * 4;
  int acc[4][NT];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[r][t] = 0;
  const uint32_t* crow[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) crow[r] = codes + min(row0 + r, K_out - 1) * nwords;
  auto load_words = [&](uint32_t (&dst)[4][WPL], int64_t w0) {
    const int nw = (int)min((int64_t)CW, nwords - w0);
#pragma unroll
    for (int k = 0; k < WPL; ++k) {
      const int w = lane + 64 * k;
#pragma unroll
      for (int r = 0; r < 4; ++r) dst[r][k] = crow[r][w0 + min(w, nw - 1)];
    }
  };
  uint32_t wd[4][WPL], wn[4][WPL] = {};
  const WT* src = reinterpret_cast<const WT*>(Cq);
  const int64_t ldq = ldc / CPW;             // words per token row
  for (int64_t w0 = 0; w0 < nwords; w0 += CW) {
    const int nw = (int)min((int64_t)CW, nwords - w0);
    lds_barrier();                          // the previous chunk's reads of cs are done
    WT cv[NT * CW / AT];
#pragma unroll
    for (int e = 0; e < NT * CW / AT; ++e) {
      const int f = e * AT + (int)threadIdx.x, t = f / CW, w = f - t * CW;
      cv[e] = src[t * ldq + w0 + min(w, nw - 1)];
    }
    if (w0 == 0) load_words(wd, 0);
#pragma unroll
    for (int e = 0; e < NT * CW / AT; ++e) {
      const int f = e * AT + (int)threadIdx.x, t = f / CW, w = f - t * CW;
      cs[t][w] = cv[e];
    }
    lds_barrier();
    if (w0 + CW < nwords) load_words(wn, w0 + CW);   // in flight during this chunk's work
#pragma unroll
    for (int k = 0; k < WPL; ++k) {
      const int w = lane + 64 * k;
      if (w >= nw) break;
      uint32_t y[4][NB];                    // byte g of y[r][b]: code of column NB g + b
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int b = 0; b < NB; ++b) y[r][b] = (wd[r][k] >> (BITS * b)) & MASK;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const WT d = cs[t][w];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int b = 0; b < NB; ++b)
            acc[r][t] = __builtin_amdgcn_sdot4((int)y[r][b], (int)dw(d, b), acc[r][t], false);
      }
    }
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int k = 0; k < WPL; ++k) wd[r][k] = wn[r][k];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1)
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[r][t] += __shfl_xor(acc[r][t], o);
  if (lane == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int64_t i = row0 + r;
      if (i < K_out) {
        const float sc = scale[i], z = zero[i];
#pragma unroll
        for (int t = 0; t < NT; ++t)
          V[t * K_out + i] = sc * delta[t] * fmaf(-z, (float)csum[t], (float)acc[r][t]);
      }
    }
  }
}

// ---- step 3: Y[t][o] = sum_i V[t][i] P_out[o][i]
// A work-group owns R output rows; a thread owns 4 consecutive columns of every 4 AT-wide
// chunk of P_out's rows (each V element is read once per work-group).
template <int NT, int R, bool VEC>
__global__ __launch_bounds__(AT) void k_apply_out(const float* __restrict__ V, int nt,
                                                  const float* __restrict__ P, int64_t K_out,
                                                  int64_t d_out, float* __restrict__ Y,
                                                  int64_t ldy) {
  __shared__ float red[AT / 64][R][NT];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t o0 = (int64_t)blockIdx.x * R;
  float acc[R][NT];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[r][t] = 0.f;
  const float* prow[R];
#pragma unroll
  for (int r = 0; r < R; ++r) prow[r] = P + min(o0 + r, d_out - 1) * K_out;
  for (int64_t i = (int64_t)threadIdx.x * 4; i < K_out; i += AT * 4) {
    float v[NT][4];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (VEC) {
        const float4 w = *reinterpret_cast<const float4*>(V + t * K_out + i);
        v[t][0] = w.x; v[t][1] = w.y; v[t][2] = w.z; v[t][3] = w.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) v[t][q] = (i + q < K_out) ? V[t * K_out + i + q] : 0.f;
      }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
      float p[4];
      if (VEC) {
        const float4 w = *reinterpret_cast<const float4*>(prow[r] + i);
        p[0] = w.x; p[1] = w.y; p[2] = w.z; p[3] = w.w;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) p[q] = (i + q < K_out) ? prow[r][i + q] : 0.f;
      }
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[r][t] = fmaf(v[t][q], p[q], acc[r][t]);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1)
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int t = 0; t < NT; ++t) acc[r][t] += __shfl_xor(acc[r][t], o);
  if (lane == 0)
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int t = 0; t < NT; ++t) red[wave][r][t] = acc[r][t];
  __syncthreads();
  if (threadIdx.x < R * NT) {
    const int r = threadIdx.x / NT, t = threadIdx.x % NT;
    const int64_t o = o0 + r;
    if (o < d_out && t < nt) {
      float sum = 0.f;
#pragma unroll
      for (int w = 0; w < AT / 64; ++w) sum += red[w][r][t];
      Y[t * ldy + o] = sum;
    }
  }
}

int64_t rup16(int64_t x) { return (x + 15) / 16 * 16; }

// splits of d_in for step 1: about 64 (enough work-groups to fill the CUs), at least 32
// rows each, at most 256 rows each (the LDS copy of the tokens' X slice)
int apply_ksplit(int64_t d_in) {
  int64_t ks = 64;
  while (ks > 1 && d_in / ks < 32) ks >>= 1;
  if ((d_in + ks - 1) / ks > 256) ks = (d_in + 255) / 256;
  return (int)ks;
}

template <int NT>
hipError_t apply_block(const void* X, int xt, int64_t ldx, int nt, int64_t d_in,
                       const uint32_t* codes, int bits, const float* scale, const float* zero,
                       int64_t K_out, int64_t K_in, const float* P_out, int64_t d_out,
                       const float* P_in, float* Y, const ApplyScratch& w, hipStream_t s) {
  const int ks = apply_ksplit(d_in);
  const int kper = (int)((d_in + ks - 1) / ks);
  const int ks_eff = (int)((d_in + kper - 1) / kper);
  const int64_t ldu = rup16(K_in);
  const bool vin = (K_in % 4 == 0) && ((reinterpret_cast<uintptr_t>(P_in) & 15) == 0);
  const bool vout = (K_out % 4 == 0) && ((reinterpret_cast<uintptr_t>(P_out) & 15) == 0);
  const dim3 gin((unsigned)((K_in + 4 * AT - 1) / (4 * AT)), (unsigned)ks_eff);
  prof_begin(s, "apply_in");
#define FQ_APPLY_IN(XT)                                                                          \
  if (vin) hipLaunchKernelGGL((k_apply_in<XT, NT, true>), gin, dim3(AT), 0, s,                    \
                              (const XT*)X, ldx, nt, d_in, P_in, K_in, kper, w.part);            \
  else hipLaunchKernelGGL((k_apply_in<XT, NT, false>), gin, dim3(AT), 0, s,                       \
                          (const XT*)X, ldx, nt, d_in, P_in, K_in, kper, w.part);
  if (xt == 0) { FQ_APPLY_IN(float) }
  else if (xt == 1) { FQ_APPLY_IN(_Float16) }
  else { FQ_APPLY_IN(uint16_t) }
#undef FQ_APPLY_IN
  hipLaunchKernelGGL(k_apply_in_reduce, dim3((unsigned)(ldu / 64 + (ldu % 64 != 0)), NT), dim3(AT), 0, s,
                     w.part, NT, nt, ks_eff, K_in, ldu, w.U);
  prof_end(s);
  const int cpw = bits == 2 ? 16 : 8;
  if (hipError_t e = apply_codes(w.U, ldu, nt, codes, K_out, (K_in + cpw - 1) / cpw, scale, zero, w.V, s, bits); e != hipSuccess)
    return e;
  prof_begin(s, "apply_out");
  constexpr int R = NT >= 4 ? 8 : 4;
  const dim3 gout((unsigned)((d_out + R - 1) / R));
  if (vout)
    hipLaunchKernelGGL((k_apply_out<NT, R, true>), gout, dim3(AT), 0, s, w.V, nt, P_out, K_out, d_out, Y, d_out);
  else
    hipLaunchKernelGGL((k_apply_out<NT, R, false>), gout, dim3(AT), 0, s, w.V, nt, P_out, K_out, d_out, Y, d_out);
  prof_end(s);
  return last_launch_error();
}

}  // namespace

hipError_t apply_codes(const float* U, int64_t ldu, int nt, const uint32_t* codes,
                       int64_t K_out, int64_t nwords, const float* scale, const float* zero,
                       float* V, hipStream_t s, int bits) {
  if (bits != 2 && bits != 4) return hipErrorInvalidValue;
  const dim3 g((unsigned)((K_out + 15) / 16));
  prof_begin(s, "apply_codes");
#define FQ_CODES(N, B)                                                                           \
  hipLaunchKernelGGL((k_apply_codes<N, B>), g, dim3(AT), 0, s, U, ldu, codes, K_out, nwords, scale, zero, V);
#define FQ_CODES_NT(B)                                                                           \
  if (nt == 1) { FQ_CODES(1, B) }                                                                \
  else if (nt == 2) { FQ_CODES(2, B) }                                                           \
  else if (nt <= 4) { FQ_CODES(4, B) }                                                           \
  else { FQ_CODES(8, B) }
  if (bits == 2) { FQ_CODES_NT(2) } else { FQ_CODES_NT(4) }
#undef FQ_CODES_NT
#undef FQ_CODES
  prof_end(s);
  return last_launch_error();
}

hipError_t act_quantize(const float* U, int64_t ldu, int64_t n, int64_t K, int bits,
                        int8_t* Cq, int64_t ldc, int perm_cpw, float* delta, int* csum,
                        hipStream_t s) {
  if (n == 0) return hipSuccess;
  const float qmax = (float)((1 << (bits - 1)) - 1);
  const dim3 g((unsigned)n);
  prof_begin(s, "act_quantize");
  if (perm_cpw == 16)
    hipLaunchKernelGGL(k_act_quantize<16>, g, dim3(QT), 0, s, U, ldu, K, qmax, Cq, ldc, delta, csum);
  else if (perm_cpw == 8)
    hipLaunchKernelGGL(k_act_quantize<8>, g, dim3(QT), 0, s, U, ldu, K, qmax, Cq, ldc, delta, csum);
  else
    hipLaunchKernelGGL(k_act_quantize<0>, g, dim3(QT), 0, s, U, ldu, K, qmax, Cq, ldc, delta, csum);
  prof_end(s);
  return last_launch_error();
}

hipError_t apply_codes_i8(const int8_t* Cq, int64_t ldc, const float* delta, const int* csum,
                          int nt, int bits, const uint32_t* codes, int64_t K_out, int64_t nwords,
                          const float* scale, const float* zero, float* V, hipStream_t s) {
  const dim3 g((unsigned)((K_out + 15) / 16));
  prof_begin(s, "apply_codes");
#define FQ_CODES_I8(N, B) \
  hipLaunchKernelGGL((k_apply_codes_i8<N, B>), g, dim3(AT), 0, s, Cq, ldc, delta, csum, codes, K_out, nwords, scale, zero, V);
#define FQ_CODES_I8_NT(B)                 \
  if (nt == 1) { FQ_CODES_I8(1, B) }      \
  else if (nt == 2) { FQ_CODES_I8(2, B) } \
  else if (nt <= 4) { FQ_CODES_I8(4, B) } \
  else { FQ_CODES_I8(8, B) }
  if (bits == 4) { FQ_CODES_I8_NT(4) }
  else { FQ_CODES_I8_NT(2) }
#undef FQ_CODES_I8_NT
#undef FQ_CODES_I8
  prof_end(s);
  return last_launch_error();
}

size_t apply_scratch_floats(int64_t d_in, int64_t K_out, int64_t K_in, ApplyScratch* w,
                            float* base) {
  const int ks = apply_ksplit(d_in);
  const int64_t kper = (d_in + ks - 1) / ks;
  const int64_t ks_eff = (d_in + kper - 1) / kper;
  size_t off = 0;
  auto take = [&](size_t n) {
    float* p = base ? base + off : nullptr;
    off += (n + 63) / 64 * 64;
    return p;
  };
  ApplyScratch l{};
  l.part = take((size_t)ks_eff * APPLY_NT * K_in);
  l.U = take((size_t)APPLY_NT * rup16(K_in));
  l.V = take((size_t)APPLY_NT * K_out);
  if (w) *w = l;
  return off;
}

hipError_t frame_apply(const void* X, int xt, int64_t n, int64_t ldx, int64_t d_in,
                       const uint32_t* codes, int bits, const float* scale, const float* zero,
                       int64_t K_out, int64_t K_in, const float* P_out, int64_t d_out,
                       const float* P_in, float* Y, const ApplyScratch& w, hipStream_t s) {
  const int esz = xt == 0 ? 4 : 2;
  for (int64_t t0 = 0; t0 < n; t0 += APPLY_NT) {
    const int nt = (int)std::min<int64_t>(APPLY_NT, n - t0);
    const void* Xb = static_cast<const char*>(X) + t0 * ldx * esz;
    float* Yb = Y + t0 * d_out;
    hipError_t e;
    if (nt == 1)
      e = apply_block<1>(Xb, xt, ldx, nt, d_in, codes, bits, scale, zero, K_out, K_in, P_out, d_out, P_in, Yb, w, s);
    else if (nt == 2)
      e = apply_block<2>(Xb, xt, ldx, nt, d_in, codes, bits, scale, zero, K_out, K_in, P_out, d_out, P_in, Yb, w, s);
    else if (nt <= 4)
      e = apply_block<4>(Xb, xt, ldx, nt, d_in, codes, bits, scale, zero, K_out, K_in, P_out, d_out, P_in, Yb, w, s);
    else
      e = apply_block<8>(Xb, xt, ldx, nt, d_in, codes, bits, scale, zero, K_out, K_in, P_out, d_out, P_in, Yb, w, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace fq
