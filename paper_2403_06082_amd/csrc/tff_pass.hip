// The analysis D = P_out^T W P_in, H~ = P_in^T H P_in and the synthesis
// W^ = P_out diag(scale)(Q - zero) P_in^T with both frames applied from their
// construction P = (R1 (x) R2) T / sqrt(k) (Sec. 2.2 and the appendix on constructing
// TFFs; the appendix on inference cost counts this route), for whole weight matrices.
//
// Every two-sided product is two passes of a one-sided row transform with a transpose
// between them: D^T = (W P_in)^T P_out, so D is the transposed row analysis (by P_out) of
// the transposed row analysis (by P_in) of W.  A row transform has two parts:
//  - the rotation R1^T M R2 (analysis) or R1 M R2^T (synthesis) of each row read as a
//    d1 x d2 matrix M: two batched small products on fp32 MFMA (k_rot_step);
//  - the DFT part, which acts on the rho/2 blocks of 2m real coordinates separately:
//    block c of an analysed row is y_c F_c with F_c the real 2m x 2k matrix
//      F_c[2j][2s] = F_c[2j+1][2s+1] = cos(phi) / sqrt(k),
//      F_c[2j][2s+1] = -sin(phi) / sqrt(k),  F_c[2j+1][2s] = sin(phi) / sqrt(k),
//      phi = 2 pi ((c m + j) s mod k) / k,
//    (conj(w^((cm+j)s)) times the complex coordinate, realified), and a synthesised row is
//    v_c F_c^T.  All rows of all blocks are one batch of rho/2 MFMA products (bf16 pairs,
//    fp32 accumulation), 2 d k multiply-adds per row instead of the dense d k rho.
// Block c of an analysed row fills frame columns s rho + 2c + e (e = 0, 1).  The analysis
// writes that order straight from the product's epilogue (a row map); on the synthesis
// side the gathers below move between frame order and the block order of the products.
#include "fq_internal.h"

#include <cmath>

namespace fq {
namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int TT = 256;
constexpr int RB = 64;       // rotation output tile (RB x RB per wave)
constexpr int RK = 16;       // rotation k step

template <typename T>
__device__ __forceinline__ float ldx_f32(const T* p);
template <>
__device__ __forceinline__ float ldx_f32<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ldx_f32<uint16_t>(const uint16_t* p) {   // bf16
  return __uint_as_float((uint32_t)*p << 16);
}
template <>
__device__ __forceinline__ float ldx_f32<_Float16>(const _Float16* p) { return (float)*p; }

__device__ __forceinline__ uint32_t rne_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

struct RotOut {
  float* f; int64_t ldf;               // fp32 rows (row t at f + t ldf)
  u16* hi; u16* lo; int64_t ldp;       // bf16 pair rows in block layout (row t at + t ldp)
  int bw, pb;                          // block layout: coordinate p sits at (p / bw) pb + p % bw
};

// 4 consecutive elements at p as floats (16 bytes for fp32, 8 for the 16-bit types)
template <typename T>
__device__ __forceinline__ float4 ld4_f32(const T* p);
template <>
__device__ __forceinline__ float4 ld4_f32<float>(const float* p) {
  return *reinterpret_cast<const float4*>(p);
}
template <>
__device__ __forceinline__ float4 ld4_f32<uint16_t>(const uint16_t* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
}
template <>
__device__ __forceinline__ float4 ld4_f32<_Float16>(const _Float16* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  const _Float16* h = reinterpret_cast<const _Float16*>(&u);
  return make_float4((float)h[0], (float)h[1], (float)h[2], (float)h[3]);
}

typedef float RotTile[RK][RB + 4];

// Stage the RK x RB tile T(k, q) = base[q ld + k] (KC) or base[k ld + q] (!KC), k0 <= k <
// k0 + RK, q0 <= q < q0 + RB, into L[k - k0][q - q0]; entries with k >= kext or q >= qext
// are 0.  The tile is 256 runs of 4 elements contiguous in memory; thread r of nthr takes
// runs r, r + nthr, ...  A run is one 16- (8-) byte load when vec (rows aligned) and it
// lies inside the extents, else element by element.
template <typename T, bool KC>
__device__ __forceinline__ void stage_tile(const T* __restrict__ base, int64_t ld, int k0, int kext,
                                           int q0, int qext, bool vec, RotTile& L, int r,
                                           int nthr) {
  for (int u = r; u < 256; u += nthr) {
    if (KC) {
      const int q = u >> 2, kq = (u & 3) * 4;
      const int gq = q0 + q, gk = k0 + kq;
      const T* src = base + (int64_t)gq * ld + gk;
      if (vec && gq < qext && gk + 3 < kext) {
        const float4 v = ld4_f32<T>(src);
        L[kq][q] = v.x; L[kq + 1][q] = v.y; L[kq + 2][q] = v.z; L[kq + 3][q] = v.w;
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c)
          L[kq + c][q] = (gq < qext && gk + c < kext) ? ldx_f32<T>(src + c) : 0.f;
      }
    } else {
      const int k = u >> 4, qq = (u & 15) * 4;
      const int gk = k0 + k, gq = q0 + qq;
      const T* src = base + (int64_t)gk * ld + gq;
      if (vec && gk < kext && gq + 3 < qext) {
        *reinterpret_cast<float4*>(&L[k][qq]) = ld4_f32<T>(src);
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c)
          L[k][qq + c] = (gk < kext && gq + c < qext) ? ldx_f32<T>(src + c) : 0.f;
      }
    }
  }
}

// One factor of the rotation for n vectors, each read as a d1 x d2 row-major matrix X_t:
// XL: C_t = X_t S (S d2 x d2), else C_t = S X_t (S d1 x d1); S(a, b) = S[b][a] when ST.
// A work-group of 4 waves owns one 64 x 64 output tile for 4 consecutive vectors (one per
// wave) and stages the tile of S they share once per k step of 16.  Each wave forms its
// tile as 2 x 2 blocks of v_mfma_f32_32x32x2_f32 (fp32 operands and sums).  grid
// (ceil(n/4) * ceil(d1/64) * ceil(d2/64)).  vx / vs: rows of X / S allow 4-element loads.
// OUT 0: fp32 rows; OUT 1: bf16 (hi, lo) rows in block layout.
template <typename XT, bool XL, bool ST, int OUT>
__global__ __launch_bounds__(256) void k_rot_step(const XT* __restrict__ X, int64_t ldx, int64_t n,
                                                  const float* __restrict__ S, int d1, int d2,
                                                  int vx, int vs, RotOut o) {
  __shared__ __attribute__((aligned(16))) RotTile Sh;
  __shared__ __attribute__((aligned(16))) RotTile Xw[4];
  const int tr = (d1 + RB - 1) / RB, tc = (d2 + RB - 1) / RB;
  const int64_t blk = blockIdx.x;
  const int64_t tg = blk / (tr * tc);
  const int rem = (int)(blk - tg * (tr * tc));
  const int i0 = (rem / tc) * RB, j0 = (rem % tc) * RB;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lo = lane & 31, hi = lane >> 5;
  const int64_t t = tg * 4 + wave;
  const bool live = t < n;
  const int Kd = XL ? d2 : d1;
  const XT* x = X + (live ? t : 0) * ldx;
  floatx16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[a][b][v] = 0.f;
  RotTile& Xt = Xw[wave];
  for (int k0 = 0; k0 < Kd; k0 += RK) {
    // shared operand: B = S (XL) with q = j, or A = S (!XL) with q = i
    if (XL) {
      if (ST) stage_tile<float, true>(S, d2, k0, Kd, j0, d2, vs, Sh, tid, 256);
      else stage_tile<float, false>(S, d2, k0, Kd, j0, d2, vs, Sh, tid, 256);
    } else {
      if (ST) stage_tile<float, false>(S, d1, k0, Kd, i0, d1, vs, Sh, tid, 256);
      else stage_tile<float, true>(S, d1, k0, Kd, i0, d1, vs, Sh, tid, 256);
    }
    // this wave's vector: A = X_t (XL, contiguous in k) or B = X_t (!XL, contiguous in j)
    if (XL) stage_tile<XT, true>(x, d2, k0, Kd, i0, live ? d1 : 0, vx, Xt, lane, 64);
    else stage_tile<XT, false>(x, d2, k0, Kd, j0, live ? d2 : 0, vx, Xt, lane, 64);
    __syncthreads();
    const RotTile& As = XL ? Xt : Sh;
    const RotTile& Bs = XL ? Sh : Xt;
    // lane l supplies A(32 a + l % 32, kk + l / 32) and B(kk + l / 32, 32 b + l % 32)
#pragma unroll
    for (int kk = 0; kk < RK; kk += 2) {
      const float a0 = As[kk + hi][lo], a1 = As[kk + hi][32 + lo];
      const float b0 = Bs[kk + hi][lo], b1 = Bs[kk + hi][32 + lo];
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
    }
    __syncthreads();
  }
  if (!live) return;
  // 32 x 32 accumulator layout: value v of lane l is row 8 (v / 4) + 4 (l / 32) + v % 4,
  // column l % 32 of its block
#pragma unroll
  for (int a = 0; a < 2; ++a) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int i = i0 + 32 * a + 8 * (v >> 2) + 4 * hi + (v & 3);
      if (i >= d1) continue;
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        const int j = j0 + 32 * b + lo;
        if (j >= d2) continue;
        const float val = acc[a][b][v];
        const int64_t p = (int64_t)i * d2 + j;
        if (OUT == 0) {
          o.f[t * o.ldf + p] = val;
        } else {
          const int64_t c = p / o.bw;
          const int64_t idx = t * o.ldp + c * o.pb + (p - c * o.bw);
          const uint32_t h = rne_bf16(val);
          o.hi[idx] = (u16)h;
          o.lo[idx] = (u16)rne_bf16(val - __uint_as_float(h << 16));
        }
      }
    }
  }
}

// Block-layout pad columns [bw, pb) of every block of n rows set to 0 (both planes).
__global__ __launch_bounds__(TT) void k_zero_pads(u16* hi, u16* lo, int64_t n, int64_t ldp,
                                                  int nb, int bw, int pb) {
  const int w = pb - bw;
  const int64_t total = n * nb * w;
  for (int64_t e = (int64_t)blockIdx.x * TT + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * TT) {
    const int64_t r = e / ((int64_t)nb * w);
    const int64_t q = e - r * nb * w;
    const int64_t c = q / w, x = q - c * w;
    const int64_t idx = r * ldp + c * pb + bw + x;
    hi[idx] = 0;
    if (lo) lo[idx] = 0;
  }
}

// F_c for c < rho/2 as bf16 (hi, lo) planes [c][pm][pk] (rows 2j + e, columns 2s + e'),
// zero outside 2m x 2k.  One thread per 2 x 2 entry block (c, j, s): one phase, four
// entries, 32-bit stores (pm and pk are even).
// colscale (may be NULL): frame vector q = s rho + 2c + e (column 2s + e of block c) scaled
// by colscale[q], i.e. the blocks of P diag(colscale)
__global__ __launch_bounds__(TT) void k_dft_blocks(int k, int m, int nb, int pm, int pk,
                                                   float scale, const float* __restrict__ colscale,
                                                   int rho, u16* __restrict__ hi,
                                                   u16* __restrict__ lo) {
  // grid (ceil(hk / TT), hm, nb): slot sx, coordinate pair j, block c (no index division)
  const int hk = pk / 2;
  const int sx = (int)(blockIdx.x * TT + threadIdx.x);
  const int j = (int)blockIdx.y;
  const int64_t c = blockIdx.z;
  if (sx >= hk) return;
  {
    float cs = 0.f, sn = 0.f;
    if (j < m && sx < k) {
      // (c m + j) mod k < k and sx < k <= 3968: the product fits 32 bits
      const int base = (int)((c * m + j) % k);
      const int64_t ph = (int)((uint32_t)(base * sx) % (uint32_t)k);
      sincospif(2.0f * (float)ph / (float)k, &sn, &cs);
      cs *= scale;
      sn *= scale;
    }
    // rows 2j (x) and 2j + 1 (y); columns 2s (re) and 2s + 1 (im)
    float a0 = 1.f, a1 = 1.f;
    if (colscale && sx < k) {
      a0 = colscale[(int64_t)sx * rho + 2 * c];
      a1 = colscale[(int64_t)sx * rho + 2 * c + 1];
    }
    const float v00 = cs * a0, v01 = -sn * a1, v10 = sn * a0, v11 = cs * a1;
    auto pair = [](float a, float b, uint32_t& h, uint32_t& l) {
      const uint32_t ha = rne_bf16(a), hb = rne_bf16(b);
      h = ha | (hb << 16);
      l = rne_bf16(a - __uint_as_float(ha << 16)) | (rne_bf16(b - __uint_as_float(hb << 16)) << 16);
    };
    uint32_t h0, l0, h1, l1;
    pair(v00, v01, h0, l0);
    pair(v10, v11, h1, l1);
    const int64_t r0 = (c * pm + 2 * j) * pk + 2 * sx;
    *reinterpret_cast<uint32_t*>(hi + r0) = h0;
    *reinterpret_cast<uint32_t*>(lo + r0) = l0;
    *reinterpret_cast<uint32_t*>(hi + r0 + pk) = h1;
    *reinterpret_cast<uint32_t*>(lo + r0 + pk) = l1;
  }
}

// V[t][c pk + p] = scale[q] M[q][t], q = (p/2) rho + 2c + (p&1), as bf16 (hi, lo) for
// p < 2k, t < n; 0 for p in [2k, pk).  M is K x n (rows q at stride ldm); scale may be
// NULL (1).  A work-group takes 64 p by 32 t through LDS and writes each row t of both
// planes as 128-byte pieces (four bf16 a thread).  grid (ceil(pk/64) * ceil(n/32), rho/2).
__global__ __launch_bounds__(TT) void k_gather(const float* __restrict__ M, int64_t ldm, int64_t n,
                                               const float* __restrict__ scale, int k2, int pk,
                                               int rho, u16* __restrict__ hi,
                                               u16* __restrict__ lo, int64_t ldv) {
  __shared__ float tile[64][33];
  const int c = blockIdx.y;
  const int npb = (pk + 63) / 64;
  const int64_t tb = blockIdx.x / npb;
  const int pbk = (int)(blockIdx.x - tb * npb);
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int q = ty; q < 64; q += 8) {
    const int p = pbk * 64 + q;
    const int64_t t = tb * 32 + tx;
    float v = 0.f;
    if (p < k2 && t < n) {
      const int64_t row = (int64_t)(p >> 1) * rho + 2 * c + (p & 1);
      v = M[row * ldm + t];
      if (scale) v *= scale[row];
    }
    tile[q][tx] = v;
  }
  __syncthreads();
  // thread: p quad pq = tid % 16 of rows t = tid / 16 and tid / 16 + 16
  const int pq = threadIdx.x & 15;
  const int p = pbk * 64 + 4 * pq;
  if (p >= pk) return;
  for (int tl = threadIdx.x >> 4; tl < 32; tl += TT / 16) {
    const int64_t t = tb * 32 + tl;
    if (t >= n) break;
    uint32_t h[4], l[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float v = tile[4 * pq + u][tl];
      h[u] = rne_bf16(v);
      l[u] = rne_bf16(v - __uint_as_float(h[u] << 16));
    }
    const int64_t idx = t * ldv + (int64_t)c * pk + p;
    *reinterpret_cast<uint2*>(hi + idx) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    *reinterpret_cast<uint2*>(lo + idx) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
  }
}

// The codes read down their columns: V[t][c pk + 2s + e] = code(q, t) - zero[q] as bf16
// (small integers, exact), q = s rho + 2c + e, for the code matrix's columns t < cols and
// s < k; 0 for s in [k, pk / 2).  codes: rows x ceil(cols / cpw) words, cpw = floor(32 / bits)
// codes a word, row-major.  A work-group takes 32 columns t and 32 pair slots s of one block
// c: the 64 code rows through LDS, then rows of V in 128-byte pieces.
// grid (ceil(cols / 32), ceil(pk / 64), rho / 2).
template <int BITS>
__global__ __launch_bounds__(TT) void k_dequant_gather_t(const uint32_t* __restrict__ codes,
                                                         const float* __restrict__ zero,
                                                         int64_t cols, int k, int pk, int rho,
                                                         u16* __restrict__ V, int64_t ldv) {
  constexpr int CPW = 32 / BITS;
  constexpr uint32_t MASK = (1u << BITS) - 1u;
  __shared__ float tile[64][33];
  const int64_t nw = (cols + CPW - 1) / CPW;
  const int64_t t0 = (int64_t)blockIdx.x * 32;
  const int s0 = blockIdx.y * 32, c = blockIdx.z;
  const int tid = threadIdx.x;
  {  // code row i: slot s0 + i / 2, e = i % 2; this thread's 8 columns of it, which lie
     // in at most two words (a word holds at least 8 codes)
    const int i = tid >> 2, tq = (tid & 3) * 8;
    const int sx = s0 + (i >> 1);
    const bool in = sx < k;
    const int64_t q = in ? (int64_t)sx * rho + 2 * c + (i & 1) : 0;
    const uint32_t* row = codes + q * nw;
    const float z = in ? zero[q] : 0.f;
    const int64_t ta = t0 + tq, wa = ta / CPW;
    const uint32_t w0 = (in && ta < cols) ? row[wa] : 0u;
    const uint32_t w1 = (in && wa + 1 < nw) ? row[wa + 1] : 0u;
    const int off = (int)(ta - wa * CPW);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int pos = off + u;                       // code position from word wa
      const uint32_t w = pos < CPW ? (w0 >> (BITS * pos)) : (w1 >> (BITS * (pos - CPW)));
      tile[i][tq + u] = (in && ta + u < cols) ? (float)(w & MASK) - z : 0.f;
    }
  }
  __syncthreads();
  const int sl = tid & 31;
  if (s0 + sl >= pk / 2) return;
  for (int tl = tid >> 5; tl < 32; tl += TT / 32) {
    const int64_t t = t0 + tl;
    if (t >= cols) break;
    const uint32_t v = (__float_as_uint(tile[2 * sl][tl]) >> 16) |
                       (__float_as_uint(tile[2 * sl + 1][tl]) & 0xFFFF0000u);
    *reinterpret_cast<uint32_t*>(V + t * ldv + (int64_t)c * pk + 2 * (s0 + sl)) = v;
  }
}

// X = (X + X^T) / 2 in place (n x n at stride ld): work-group (bi, bj), bi <= bj, owns the
// tiles (bi, bj) and (bj, bi).  grid (T, T), T = ceil(n / 32); bi > bj return at once.
__global__ __launch_bounds__(TT) void k_sym_average(float* __restrict__ X, int64_t n, int64_t ld) {
  __shared__ float a[32][33], b[32][33];
  const int64_t bi = blockIdx.x, bj = blockIdx.y;
  if (bi > bj) return;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
  for (int q = ty; q < 32; q += 8) {
    const int64_t i = bi * 32 + q, j = bj * 32 + tx;
    a[q][tx] = (i < n && j < n) ? X[i * ld + j] : 0.f;
    const int64_t i2 = bj * 32 + q, j2 = bi * 32 + tx;
    b[q][tx] = (i2 < n && j2 < n) ? X[i2 * ld + j2] : 0.f;
  }
  __syncthreads();
  for (int q = ty; q < 32; q += 8) {
    const int64_t i = bi * 32 + q, j = bj * 32 + tx;
    if (i < n && j < n) X[i * ld + j] = 0.5f * (a[q][tx] + b[tx][q]);
    const int64_t i2 = bj * 32 + q, j2 = bi * 32 + tx;
    if (i2 < n && j2 < n) X[i2 * ld + j2] = 0.5f * (b[q][tx] + a[tx][q]);
  }
}

// ---- both rotation factors of a row in one work-group.
// out_t = A X_t B with X_t the d1 x d2 view of row t; analysis: A = R1^T, B = R2; synthesis:
// A = R1, B = R2^T.  A work-group of NW waves takes nv consecutive rows and one block of
// BJ = 16 NW output columns; wave w forms the 16 columns [16 w, 16 w + 16) of the block for
// every output row, with v_mfma_f32_16x16x4_f32 on 16 x 16 tiles:
//  step A  T = X_t B[:, cols], K = d2.  Inside a chunk of 16 k values, at step s lane l
//          supplies k = kc + 4 (l / 16) + s (a permutation of the k order, the same for both
//          operands), so each lane reads its operands for four steps as one 16-byte run.
//  step B  out[:, cols] = A T, K = d1.  The accumulator of tile mt of step A holds, in lane
//          l and value v, T[16 mt + 4 (l / 16) + v][col l % 16]: in the same k order this is
//          exactly the B operand of step B at step v, so T stays in registers.
// X_t, B[:, block] (transposed) and A sit in LDS with k contiguous; the next row's X is
// fetched into registers while the current one is multiplied.  The output block goes
// through LDS (the space of X_t) and leaves in runs of 8 consecutive elements per lane.
#ifndef FR_ROWS
#define FR_ROWS 4
#endif
constexpr int FR_NV = FR_ROWS;   // rows per work-group
constexpr int FR_MAXQ = 16;      // pieces of 4 elements of a row per thread

__host__ __device__ constexpr int fr_pad16(int x) { return (x + 15) / 16 * 16; }
__host__ __device__ inline int fr_waves(int d2) { return fr_pad16(d2) >= 128 ? 8 : 4; }
__host__ __device__ inline int fr_mt(int d1) {    // 16-row tiles of d1 (5 -> 6, 7 -> 8)
  const int m = fr_pad16(d1) / 16;
  return m == 5 ? 6 : (m == 7 ? 8 : m);
}

// LDS floats of the fused kernel for d1 x d2
__host__ __device__ inline int64_t fr_lds_floats(int d1, int d2) {
  const int64_t m = 16 * fr_mt(d1), k = fr_pad16(d2), bj = 16 * fr_waves(d2);
  const int64_t pxo = (k > bj ? k : bj) + 4;
  return m * pxo + bj * (k + 4) + m * (m + 4);
}

typedef float floatx4 __attribute__((ext_vector_type(4)));

// a row's pieces held raw while in flight (16 bytes for fp32, 8 for the 16-bit types);
// converted to fp32 when stored to LDS
template <typename XT> struct FrRaw { typedef uint2 T; };
template <> struct FrRaw<float> { typedef float4 T; };
__device__ __forceinline__ float4 fr_cvt(float4 v, const float*) { return v; }
__device__ __forceinline__ float4 fr_cvt(uint2 u, const uint16_t*) {   // bf16
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
}
__device__ __forceinline__ float4 fr_cvt(uint2 u, const _Float16*) {
  const _Float16* h = reinterpret_cast<const _Float16*>(&u);
  return make_float4((float)h[0], (float)h[1], (float)h[2], (float)h[3]);
}

template <typename XT, bool SYN, int OUT, int MT, int NQ, int NW>
__global__ __launch_bounds__(64 * NW) void k_rot_fused(const XT* __restrict__ X, int64_t ldx,
                                                       int64_t n, const float* __restrict__ R1,
                                                       const float* __restrict__ R2, int d1,
                                                       int d2, int vout, int nv, RotOut o) {
  extern __shared__ __attribute__((aligned(16))) float fr_lds[];
  constexpr int M = 16 * MT;                   // d1 padded
  constexpr int BJ = 16 * NW;                  // output columns per work-group
  constexpr int NT = 64 * NW;                  // threads
  const int K2 = fr_pad16(d2);                 // d2 padded (k of step A)
  const int PX = K2 + 4, PA = M + 4;           // row pitches (floats): 16-byte reads of 16
  constexpr int PO = BJ + 4;                   // rows at one k fall on distinct banks
  const int PXO = (K2 > BJ ? K2 : BJ) + 4;
  float* Xs = fr_lds;                          // [M][PX]   X_t (i, k); later [M][PO] output
  float* Bs = Xs + M * PXO;                    // [BJ][PX]  B[k][jb BJ + j] at (j, k)
  float* As = Bs + BJ * PX;                    // [M][PA]   A[i][k]
  const int njb = (d2 + BJ - 1) / BJ;
  const int jb = (int)(blockIdx.x % njb);
  const int64_t t0 = (int64_t)(blockIdx.x / njb) * nv;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int c = lane & 15, g = lane >> 4;

  // resident operands: A (d1 x d1) and the block's columns of B, zero padded
  for (int e = tid; e < M * M; e += NT) {
    const int i = e / M, k = e - i * M;
    float v = 0.f;
    if (i < d1 && k < d1) v = SYN ? R1[(int64_t)i * d1 + k] : R1[(int64_t)k * d1 + i];
    As[i * PA + k] = v;
  }
  for (int e = tid; e < BJ * K2; e += NT) {
    const int j = e / K2, k = e - j * K2;
    const int jj = jb * BJ + j;
    float v = 0.f;
    if (jj < d2 && k < d2) v = SYN ? R2[(int64_t)jj * d2 + k] : R2[(int64_t)k * d2 + jj];
    Bs[j * PX + k] = v;
  }

  // the row's d1 x d2 values in pieces of 4 (d2 % 4 == 0, so a piece stays in one row of
  // the view): piece e = tid + NT q covers elements 4 e .. 4 e + 3, i.e.
  // (i, k) = (4 e / d2, 4 e mod d2); its LDS offset is computed once
  typedef typename FrRaw<XT>::T Raw;
  const int qrow = d2 / 4;
  const int nq = d1 * qrow;
  int loff[NQ];
  {
    int i = tid / qrow, r = tid - (tid / qrow) * qrow;
    const int di = NT / qrow, dr = NT - (NT / qrow) * qrow;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      loff[q] = i * PX + 4 * r;
      i += di;
      r += dr;
      if (r >= qrow) { r -= qrow; ++i; }
    }
  }
  Raw pre[NQ];
  auto fetch = [&](int64_t t) {
    const Raw* x = reinterpret_cast<const Raw*>(X + t * ldx);
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      if (tid + NT * q < nq) pre[q] = x[tid + NT * q];
  };
  if (t0 < n) fetch(t0);

  // zero padding of X_t: rows d1 .. M once (the output block, staged in the same space,
  // covers rows < d1 only when BJ <= K2); columns d2 .. K2 of rows < d1 before every row
  const bool stage_fits = BJ <= K2;
  for (int e = tid; e < (M - d1) * K2; e += NT) Xs[d1 * PX + (e / K2) * PX + e % K2] = 0.f;
  const int kpad = K2 - d2;

  for (int v = 0; v < nv; ++v) {
    const int64_t t = t0 + v;
    if (t >= n) break;
    __syncthreads();                 // the previous row's output has left the LDS
    if (!stage_fits) {
      for (int e = tid; e < M * K2; e += NT) {
        const int i = e / K2, k = e - i * K2;
        if (i >= d1 || k >= d2) Xs[i * PX + k] = 0.f;
      }
    } else if (kpad > 0) {
      for (int e = tid; e < d1 * kpad; e += NT) Xs[(e / kpad) * PX + d2 + e % kpad] = 0.f;
    }
#pragma unroll
    for (int q = 0; q < NQ; ++q)
      if (tid + NT * q < nq)
        *reinterpret_cast<float4*>(&Xs[loff[q]]) = fr_cvt(pre[q], (const XT*)nullptr);
    __syncthreads();
    if (v + 1 < nv && t + 1 < n) fetch(t + 1);

    // step A: T[:, 16 w + c] for all M rows; the MT accumulators interleave
    floatx4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int kc = 0; kc < K2; kc += 16) {
      const float4 bv = *reinterpret_cast<const float4*>(&Bs[(16 * w + c) * PX + kc + 4 * g]);
      float4 av[MT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        av[mt] = *reinterpret_cast<const float4*>(&Xs[(16 * mt + c) * PX + kc + 4 * g]);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt].x, bv.x, acc[mt], 0, 0, 0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt].y, bv.y, acc[mt], 0, 0, 0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt].z, bv.z, acc[mt], 0, 0, 0);
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt].w, bv.w, acc[mt], 0, 0, 0);
    }
    __syncthreads();                 // every wave is done with X_t
    // step B: out[:, 16 w + c] = A T, the accumulators of step A as the B operand
    floatx4 res[MT];
#pragma unroll
    for (int it = 0; it < MT; ++it) res[it] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float4 av[MT];
#pragma unroll
      for (int it = 0; it < MT; ++it)
        av[it] = *reinterpret_cast<const float4*>(&As[(16 * it + c) * PA + 16 * mt + 4 * g]);
#pragma unroll
      for (int it = 0; it < MT; ++it) res[it] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[it].x, acc[mt][0], res[it], 0, 0, 0);
#pragma unroll
      for (int it = 0; it < MT; ++it) res[it] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[it].y, acc[mt][1], res[it], 0, 0, 0);
#pragma unroll
      for (int it = 0; it < MT; ++it) res[it] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[it].z, acc[mt][2], res[it], 0, 0, 0);
#pragma unroll
      for (int it = 0; it < MT; ++it) res[it] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[it].w, acc[mt][3], res[it], 0, 0, 0);
    }
    // lane l, value r of tile it: output row 16 it + 4 g + r, block column 16 w + c
    float* Os = Xs;
#pragma unroll
    for (int it = 0; it < MT; ++it)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (16 * it + 4 * g + r < d1) Os[(16 * it + 4 * g + r) * PO + 16 * w + c] = res[it][r];
    __syncthreads();
    // the block's rows (< d1) in runs of 8 columns: run u = (row, 8 j8) of d1 x BJ / 8
    const int jbase = jb * BJ;
    const int ncol = min(BJ, d2 - jbase);
    for (int u = tid; u < d1 * (BJ / 8); u += NT) {
      const int ii = u / (BJ / 8), j8 = (u - ii * (BJ / 8)) * 8;
      if (j8 >= ncol) continue;
      const float4 v0 = *reinterpret_cast<const float4*>(&Os[ii * PO + j8]);
      const float4 v1 = *reinterpret_cast<const float4*>(&Os[ii * PO + j8 + 4]);
      const float vv[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
      const int64_t p0 = (int64_t)ii * d2 + jbase + j8;
      if (OUT == 0) {
        float* dst = o.f + t * o.ldf + p0;
        if (vout && j8 + 8 <= ncol) {
          *reinterpret_cast<float4*>(dst) = v0;
          *reinterpret_cast<float4*>(dst + 4) = v1;
        } else {
          for (int e = 0; e < 8 && j8 + e < ncol; ++e) dst[e] = vv[e];
        }
      } else {
        const int64_t cb = (uint32_t)p0 / (uint32_t)o.bw, pin = p0 - cb * o.bw;   // p0 < 2^31
        const int64_t idx = t * o.ldp + cb * o.pb + pin;
        if (vout && j8 + 8 <= ncol && pin + 8 <= o.bw) {
          uint32_t h[4], l[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t ha = rne_bf16(vv[2 * e]), hb = rne_bf16(vv[2 * e + 1]);
            h[e] = ha | (hb << 16);
            l[e] = rne_bf16(vv[2 * e] - __uint_as_float(ha << 16)) |
                   (rne_bf16(vv[2 * e + 1] - __uint_as_float(hb << 16)) << 16);
          }
          *reinterpret_cast<uint4*>(o.hi + idx) = make_uint4(h[0], h[1], h[2], h[3]);
          *reinterpret_cast<uint4*>(o.lo + idx) = make_uint4(l[0], l[1], l[2], l[3]);
        } else {
          for (int e = 0; e < 8 && j8 + e < ncol; ++e) {
            const int64_t pe = p0 + e, ce = (uint32_t)pe / (uint32_t)o.bw;
            const int64_t ie = t * o.ldp + ce * o.pb + (pe - ce * o.bw);
            const uint32_t hh = rne_bf16(vv[e]);
            o.hi[ie] = (u16)hh;
            o.lo[ie] = (u16)rne_bf16(vv[e] - __uint_as_float(hh << 16));
          }
        }
      }
    }
  }
}

template <typename XT, bool SYN, int OUT>
void launch_rot_fused(const XT* X, int64_t ldx, int64_t n, const TffDev& F, const RotOut& o,
                      hipStream_t s) {
  const int MT = fr_mt(F.d1), NW = fr_waves(F.d2);
  const int njb = (F.d2 + 16 * NW - 1) / (16 * NW);
  const size_t lds = (size_t)fr_lds_floats(F.d1, F.d2) * sizeof(float);
  // rows per work-group: at least FR_NV (the resident factors serve them all), and as
  // many as fill the device's work-group slots in one round when that takes fewer row
  // times than rounds of FR_NV rows (e.g. 4512 rows of the 11008-wide frame: one round of
  // 18 rows instead of five of 4).  On a side stream, which shares its compute units with
  // the caller's other work, FR_NV, so that many short work-groups balance the load.
  static int n_cu = 0;
  if (n_cu <= 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n_cu <= 0)
      n_cu = 1;
  }
  const int64_t per_cu = std::max<int64_t>(1, std::min<int64_t>((int64_t)(160 * 1024) / (int64_t)lds, 32 / NW));
  const int64_t groups = std::max<int64_t>(1, (int64_t)n_cu * per_cu / njb);   // row groups at once
  const int nv = is_side_stream(s) ? FR_NV
                                    : (int)std::max<int64_t>(FR_NV, std::min<int64_t>((n + groups - 1) / groups, 64));
  const dim3 g((unsigned)(njb * ((n + nv - 1) / nv))), b((unsigned)(64 * NW));
  const bool small = (int64_t)F.d1 * (F.d2 / 4) <= 64 * NW * 4;
  // 16-byte output runs: 8-element runs start 16-byte aligned in every destination row
  int vout;
  if (OUT == 0)
    vout = (F.d2 % 8 == 0 && o.ldf % 4 == 0 && (reinterpret_cast<uintptr_t>(o.f) & 15) == 0);
  else
    vout = (F.d2 % 8 == 0 && o.bw % 8 == 0 && o.pb % 8 == 0 && o.ldp % 8 == 0 &&
            (reinterpret_cast<uintptr_t>(o.hi) & 15) == 0 &&
            (reinterpret_cast<uintptr_t>(o.lo) & 15) == 0);
  // dynamic LDS beyond 64 KB needs the kernel's limit raised (once per instantiation)
#define FR_LAUNCH(m, q, nw) { \
      static const hipError_t attr = hipFuncSetAttribute( \
          reinterpret_cast<const void*>(k_rot_fused<XT, SYN, OUT, m, q, nw>), \
          hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024); \
      (void)attr; \
      hipLaunchKernelGGL((k_rot_fused<XT, SYN, OUT, m, q, nw>), g, b, lds, s, X, ldx, n, F.R1, F.R2, F.d1, F.d2, vout, nv, o); }
#define FR_CASE(m) case m: \
      if (NW == 4) { if (small) FR_LAUNCH(m, 4, 4) else FR_LAUNCH(m, FR_MAXQ, 4) } \
      else { if (small) FR_LAUNCH(m, 4, 8) else FR_LAUNCH(m, 8, 8) } \
      break;
  switch (MT) {
    FR_CASE(1) FR_CASE(2) FR_CASE(3) FR_CASE(4) FR_CASE(6) FR_CASE(8)
    default: break;
  }
#undef FR_CASE
#undef FR_LAUNCH
}

// the fused kernel applies when d1 <= 128, d2 % 4 == 0, rows are aligned for 4-element
// loads, a row fits the register prefetch and the operands fit in LDS
bool rot_fused_ok(const TffDev& F, const void* X, int esz, int64_t ldx) {
  const int NW = fr_waves(F.d2);
  const int maxq = NW == 4 ? FR_MAXQ : 8;
  return F.d1 <= 128 && F.d2 % 4 == 0 && ldx % 4 == 0 &&
         (reinterpret_cast<uintptr_t>(X) % (4 * esz)) == 0 &&
         (int64_t)F.d1 * (F.d2 / 4) <= (int64_t)64 * NW * maxq &&
         fr_lds_floats(F.d1, F.d2) * 4 <= 160 * 1024;
}

unsigned grid_1d(int64_t total) {
  const int64_t g = (total + TT - 1) / TT;
  return (unsigned)(g < 65536 ? (g > 0 ? g : 1) : 65536);
}

// The two rotation factors of n rows.  Analysis: tmp = X R2, then R1^T tmp into `o`;
// synthesis: tmp = X R2^T, then R1 tmp into `o`.  xt: 0 f32, 1 f16, 2 bf16 (first factor
// only; tmp is fp32).
template <int OUT>
hipError_t rotate_rows(const void* X, int xt, int64_t ldx, int64_t n, const TffDev& F, bool synth,
                       float* tmp, const RotOut& o, hipStream_t s, const char* name) {
  const int64_t tiles = (int64_t)((F.d1 + RB - 1) / RB) * ((F.d2 + RB - 1) / RB);
  const dim3 g((unsigned)((n + 3) / 4 * tiles)), b(256);
  RotOut ot{};
  ot.f = tmp; ot.ldf = F.d;
  auto al = [](const void* p, int bytes) { return ((uintptr_t)p % bytes) == 0; };
  const int esz = xt == 0 ? 4 : 2;
  const int vx = (F.d2 % 4 == 0 && ldx % 4 == 0 && al(X, 4 * esz)) ? 1 : 0;
  const int vt = (F.d2 % 4 == 0 && al(tmp, 16)) ? 1 : 0;      // tmp rows are d floats
  const int vs2 = (F.d2 % 4 == 0 && al(F.R2, 16)) ? 1 : 0;
  const int vs1 = (F.d1 % 4 == 0 && al(F.R1, 16)) ? 1 : 0;
  prof_begin(s, name);
  // the pass analyses into the block layout and synthesises into fp32 rows
  if (rot_fused_ok(F, X, esz, ldx) && synth == (OUT == 0)) {
    if constexpr (OUT == 0) {
      launch_rot_fused<float, true, 0>((const float*)X, ldx, n, F, o, s);
    } else {
      if (xt == 0)
        launch_rot_fused<float, false, OUT>((const float*)X, ldx, n, F, o, s);
      else if (xt == 1)
        launch_rot_fused<_Float16, false, OUT>((const _Float16*)X, ldx, n, F, o, s);
      else
        launch_rot_fused<uint16_t, false, OUT>((const uint16_t*)X, ldx, n, F, o, s);
    }
    prof_end(s);
    return last_launch_error();
  }
  if (synth) {
    hipLaunchKernelGGL((k_rot_step<float, true, true, 0>), g, b, 0, s, (const float*)X, ldx, n, F.R2, F.d1, F.d2, vx, vs2, ot);
    hipLaunchKernelGGL((k_rot_step<float, false, false, OUT>), g, b, 0, s, (const float*)tmp, F.d, n, F.R1, F.d1, F.d2, vt, vs1, o);
  } else {
    if (xt == 0)
      hipLaunchKernelGGL((k_rot_step<float, true, false, 0>), g, b, 0, s, (const float*)X, ldx, n, F.R2, F.d1, F.d2, vx, vs2, ot);
    else if (xt == 1)
      hipLaunchKernelGGL((k_rot_step<_Float16, true, false, 0>), g, b, 0, s, (const _Float16*)X, ldx, n, F.R2, F.d1, F.d2, vx, vs2, ot);
    else
      hipLaunchKernelGGL((k_rot_step<uint16_t, true, false, 0>), g, b, 0, s, (const uint16_t*)X, ldx, n, F.R2, F.d1, F.d2, vx, vs2, ot);
    hipLaunchKernelGGL((k_rot_step<float, false, true, OUT>), g, b, 0, s, (const float*)tmp, F.d, n, F.R1, F.d1, F.d2, vt, vs1, o);
  }
  prof_end(s);
  return last_launch_error();
}

}  // namespace

TffPassGeom tff_pass_geom(const TffDev& F) {
  TffPassGeom g;
  g.nb = F.rho / 2;
  g.m2 = 2 * F.m;
  g.pm = (g.m2 + 31) / 32 * 32;
  g.k2 = 2 * F.k;
  g.pk = (g.k2 + 31) / 32 * 32;
  return g;
}

hipError_t tff_dft_blocks(const TffDev& F, u16* hi, u16* lo, hipStream_t s, const float* colscale) {
  const TffPassGeom g = tff_pass_geom(F);
  prof_begin(s, "tffp_blocks");
  hipLaunchKernelGGL(k_dft_blocks, dim3((unsigned)((g.pk / 2 + TT - 1) / TT), (unsigned)(g.pm / 2), (unsigned)g.nb), dim3(TT), 0, s, (int)F.k,
                     (int)F.m, (int)g.nb, (int)g.pm, (int)g.pk,
                     (float)(1.0 / std::sqrt((double)F.k)), colscale, (int)F.rho, hi, lo);
  prof_end(s);
  return last_launch_error();
}

hipError_t tff_rows_analysis_t(const void* X, int xt, int64_t ldx, int64_t n, const TffDev& F,
                               const u16* Fhi, const u16* Flo, float* tmp, u16* Yhi, u16* Ylo,
                               float* O, float* out, int64_t ldout, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const TffPassGeom g = tff_pass_geom(F);
  const int64_t ldy = g.nb * g.pm;
  RotOut o{};
  o.hi = Yhi; o.lo = Ylo; o.ldp = ldy; o.bw = (int)g.m2; o.pb = (int)g.pm;
  hipError_t e;
  if (g.pm > g.m2) {
    prof_begin(s, "tffp_gather");
    hipLaunchKernelGGL(k_zero_pads, dim3(grid_1d(n * g.nb * (g.pm - g.m2))), dim3(TT), 0, s, Yhi, Ylo,
                       n, ldy, (int)g.nb, (int)g.m2, (int)g.pm);
    prof_end(s);
  }
  if ((e = rotate_rows<1>(X, xt, ldx, n, F, false, tmp, o, s, "tffp_rotate_an")) != hipSuccess)
    return e;
  // block c of every analysed row t, in frame order: out[(p/2) rho + 2c + (p&1)][t] =
  // sum_j F_c[j][p] Y[t][c pm + j], i.e. F_c^T Y_c^T per block (A = F_c read M-major,
  // B = Y read K-major), the rows placed in frame order by the epilogue's row map
  GemmDesc d;
  d.M = (int)g.k2; d.N = (int)n; d.K = (int)g.pm;
  d.a[0] = Fhi; d.a[1] = Flo; d.lda = g.pk; d.a_kmajor = false;
  d.b[0] = Yhi; d.b[1] = Ylo; d.ldb = ldy; d.b_kmajor = true;
  d.npass = 3;
  d.pa[0] = 0; d.pb[0] = 0; d.pa[1] = 0; d.pb[1] = 1; d.pa[2] = 1; d.pb[2] = 0;
  d.epi = EPI_F32; d.c = out; d.ldc = ldout; d.rowmap = (int)F.rho;
  d.batch = (int)g.nb; d.bsa = g.pm * g.pk; d.bsb = g.pm; d.bsc = 2 * ldout;
  d.name = "tffp_dft_an";
  (void)O;
  return gemm_run(d, nullptr, s);
}

hipError_t tff_gather_rows(const float* M, int64_t ldm, int64_t n, const float* scale,
                           const TffDev& F, u16* hi, u16* lo, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const TffPassGeom g = tff_pass_geom(F);
  prof_begin(s, "tffp_gather");
  hipLaunchKernelGGL(k_gather, dim3((unsigned)(((n + 31) / 32) * ((g.pk + 63) / 64)), (unsigned)g.nb), dim3(TT), 0, s,
                     M, ldm, n, scale, (int)g.k2, (int)g.pk, (int)F.rho, hi, lo, g.nb * g.pk);
  prof_end(s);
  return last_launch_error();
}

hipError_t tff_dequant_gather_t(const uint32_t* codes, int bits, const float* zero, int64_t cols,
                                const TffDev& F, u16* V, hipStream_t s) {
  if (cols == 0) return hipSuccess;
  const TffPassGeom g = tff_pass_geom(F);
  prof_begin(s, "tffp_gather");
  const dim3 grid((unsigned)((cols + 31) / 32), (unsigned)((g.pk / 2 + 31) / 32), (unsigned)g.nb);
  if (bits == 2)
    hipLaunchKernelGGL(k_dequant_gather_t<2>, grid, dim3(TT), 0, s, codes, zero, cols, (int)F.k,
                       (int)g.pk, (int)F.rho, V, g.nb * g.pk);
  else if (bits == 3)
    hipLaunchKernelGGL(k_dequant_gather_t<3>, grid, dim3(TT), 0, s, codes, zero, cols, (int)F.k,
                       (int)g.pk, (int)F.rho, V, g.nb * g.pk);
  else
    hipLaunchKernelGGL(k_dequant_gather_t<4>, grid, dim3(TT), 0, s, codes, zero, cols, (int)F.k,
                       (int)g.pk, (int)F.rho, V, g.nb * g.pk);
  prof_end(s);
  return last_launch_error();
}

hipError_t tff_rows_synthesis(const u16* Vhi, const u16* Vlo, int64_t n, const TffDev& F,
                              const u16* Fhi, const u16* Flo, float* Z, float* tmp, float* out,
                              int64_t ldout, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const TffPassGeom g = tff_pass_geom(F);
  // Z[:, c 2m .. (c+1) 2m) = V_c F_c^T, all blocks in one batch
  GemmDesc d;
  d.M = (int)n; d.N = (int)g.m2; d.K = (int)g.pk;
  d.a[0] = Vhi; d.a[1] = Vlo; d.lda = g.nb * g.pk; d.a_kmajor = true;
  d.b[0] = Fhi; d.b[1] = Flo; d.ldb = g.pk; d.b_kmajor = true;
  if (Vlo) {
    d.npass = 3;
    d.pa[0] = 0; d.pb[0] = 0; d.pa[1] = 0; d.pb[1] = 1; d.pa[2] = 1; d.pb[2] = 0;
  } else {
    d.npass = 2;
    d.pa[0] = 0; d.pb[0] = 0; d.pa[1] = 0; d.pb[1] = 1;
  }
  d.epi = EPI_F32; d.c = Z; d.ldc = F.d;
  d.batch = (int)g.nb; d.bsa = g.pk; d.bsb = g.pm * g.pk; d.bsc = g.m2;
  d.name = "tffp_dft_syn";
  hipError_t e;
  if ((e = gemm_run(d, nullptr, s)) != hipSuccess) return e;
  RotOut o{};
  o.f = out; o.ldf = ldout;
  return rotate_rows<0>(Z, 0, F.d, n, F, true, tmp, o, s, "tffp_rotate_syn");
}

hipError_t sym_average(float* X, int64_t n, int64_t ld, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const unsigned T = (unsigned)((n + 31) / 32);
  prof_begin(s, "tffp_gather");
  hipLaunchKernelGGL(k_sym_average, dim3(T, T), dim3(TT), 0, s, X, n, ld);
  prof_end(s);
  return last_launch_error();
}

}  // namespace fq
