// bf16 / f16 MFMA GEMM engine for gfx950 (CDNA4) and the small elementwise kernels that
// feed it.  Used for the calibration Hessian (H = X^T X, upper tiles, split over tokens),
// the frame analysis (D = P_l^T W P_prev, H~ = P_prev^T H P_prev) and the synthesis
// (W^ = P_l D^ P_prev^T).
//
// Design
//  * Work-group tile 256 x 256, K step 64, 256 threads = 4 wave64s in a 2 x 2 grid; each
//    wave owns a 128 x 128 sub-tile as 4 x 4 v_mfma_f32_32x32x16 (bf16 or f16) blocks.
//  * Both operands are staged through LDS as [row][k] with the 16-byte k-chunks of each
//    row XOR-swizzled (chunk c of row r lives at slot c ^ ((r>>1 ^ r>>3) & 7)), which
//    keeps the MFMA fragment reads conflict-free without padding.  Two stages (128 KiB)
//    double-buffer the global loads: the next stage is fetched into registers while the
//    current one feeds the MFMAs, with one barrier per stage.
//  * An operand stored with M (or N) contiguous is transposed on the way into LDS: each
//    thread loads an 8 x 8 block (eight 16-byte rows) and transposes it in registers
//    with byte permutes, so every global load stays a coalesced 16-byte access.
//  * fp32 operands enter as bf16 (hi, lo) pairs; a "pass" is one (A plane, B plane)
//    product and all passes accumulate into the same fp32 registers.
//  * Work-group ids are remapped so that consecutive tiles land on the same XCD (ids are
//    dealt round-robin over the 8 XCDs), and tiles are walked in groups of 8 tile-rows
//    for L2 reuse.
#include "fq_internal.h"

#include <stdlib.h>

namespace fq {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

namespace {

constexpr int BM = 256, BN = 256, BK = 64, NT = 256;
constexpr int TILE_ELEMS = BM * BK;          // u16 elements per operand per stage

struct KParams {
  int M, N, K;
  const u16* a0; const u16* a1;
  const u16* b0; const u16* b1;
  int64_t lda, ldb;
  int npass;
  int pa0, pa1, pa2, pb0, pb1, pb2;
  float* c; int64_t ldc;
  u16* c_hi; u16* c_lo;
  int ldc_pad;          // EPI_SPLIT: columns [N, ldc_pad) of the output are written as 0
  int aligned_a, aligned_b;
  int tiles_m, tiles_n, ntiles;
  int ksplit, k_per_split;
  float* part;
};

__device__ __forceinline__ int swz(int r) { return ((r >> 1) ^ (r >> 3)) & 7; }

__device__ __forceinline__ uint32_t bf16_rne_bits(float f) {
  uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

// ------------------------------------------------------------------ operand staging
// K-major operand: element (mn, k) at base[mn * ld + k].  Thread t stages chunks
// c = t + 256 i (i < 8): row c >> 3, 16-byte k-chunk c & 7.
__device__ __forceinline__ void load_kmajor(const u16* __restrict__ base, int64_t ld, int mn0,
                                            int k0, int MN, int K, bool aligned, uint4 (&r)[8],
                                            int tid) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = tid + NT * i;
    const int row = c >> 3;
    const int kc = c & 7;
    const int m = mn0 + row;
    const int k = k0 + kc * 8;
    if (m < MN && k + 8 <= K && aligned) {
      r[i] = *reinterpret_cast<const uint4*>(base + (int64_t)m * ld + k);
    } else {
      uint32_t w[4] = {0, 0, 0, 0};
      if (m < MN) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (k + e < K) {
            uint32_t v = base[(int64_t)m * ld + k + e];
            w[e >> 1] |= v << ((e & 1) * 16);
          }
        }
      }
      r[i] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

__device__ __forceinline__ void store_kmajor(u16* sm, const uint4 (&r)[8], int tid) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = tid + NT * i;
    const int row = c >> 3;
    const int kc = c & 7;
    *reinterpret_cast<uint4*>(sm + row * BK + ((kc ^ swz(row)) << 3)) = r[i];
  }
}

// MN-major operand: element (mn, k) at base[k * ld + mn].  Thread t loads the 8 x 8 block
// k in [k0 + 8 kb, +8), mn in [mn0 + 8 mb, +8) with kb = t >> 5, mb = t & 31.
__device__ __forceinline__ void load_mnmajor(const u16* __restrict__ base, int64_t ld, int mn0,
                                             int k0, int MN, int K, bool aligned, uint4 (&r)[8],
                                             int tid) {
  const int kb = tid >> 5;
  const int mb = tid & 31;
  const int m = mn0 + mb * 8;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int k = k0 + kb * 8 + i;
    if (k < K && m + 8 <= MN && aligned) {
      r[i] = *reinterpret_cast<const uint4*>(base + (int64_t)k * ld + m);
    } else {
      uint32_t w[4] = {0, 0, 0, 0};
      if (k < K) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (m + e < MN) {
            uint32_t v = base[(int64_t)k * ld + m + e];
            w[e >> 1] |= v << ((e & 1) * 16);
          }
        }
      }
      r[i] = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
}

__device__ __forceinline__ uint32_t dw(const uint4& v, int i) {
  return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

// Transpose the 8 x 8 block of 16-bit values and store row mb*8 + j, chunk kb.
__device__ __forceinline__ void store_mnmajor(u16* sm, const uint4 (&r)[8], int tid) {
  const int kb = tid >> 5;
  const int mb = tid & 31;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    uint32_t o[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const uint32_t lo = dw(r[2 * kk], j >> 1);
      const uint32_t hi = dw(r[2 * kk + 1], j >> 1);
      // low half of the output dword from row 2kk, high half from row 2kk+1
      o[kk] = (j & 1) ? __builtin_amdgcn_perm(hi, lo, 0x07060302u)
                      : __builtin_amdgcn_perm(hi, lo, 0x05040100u);
    }
    const int row = mb * 8 + j;
    *reinterpret_cast<uint4*>(sm + row * BK + ((kb ^ swz(row)) << 3)) =
        make_uint4(o[0], o[1], o[2], o[3]);
  }
}

template <bool AK, bool BKM>
__device__ __forceinline__ void load_stage(const KParams& p, int s, int nkt, int kbeg, int m0,
                                           int n0, uint4 (&ra)[8], uint4 (&rb)[8], int tid) {
  const int pass = s / nkt;
  const int kt = s - pass * nkt;
  const int pa = pass == 0 ? p.pa0 : (pass == 1 ? p.pa1 : p.pa2);
  const int pb = pass == 0 ? p.pb0 : (pass == 1 ? p.pb1 : p.pb2);
  const u16* A = pa ? p.a1 : p.a0;
  const u16* B = pb ? p.b1 : p.b0;
  const int k0 = kbeg + kt * BK;
  if (AK) load_kmajor(A, p.lda, m0, k0, p.M, p.K, p.aligned_a, ra, tid);
  else load_mnmajor(A, p.lda, m0, k0, p.M, p.K, p.aligned_a, ra, tid);
  if (BKM) load_kmajor(B, p.ldb, n0, k0, p.N, p.K, p.aligned_b, rb, tid);
  else load_mnmajor(B, p.ldb, n0, k0, p.N, p.K, p.aligned_b, rb, tid);
}

template <bool AK, bool BKM>
__device__ __forceinline__ void store_stage(u16* sA, u16* sB, const uint4 (&ra)[8],
                                            const uint4 (&rb)[8], int tid) {
  if (AK) store_kmajor(sA, ra, tid); else store_mnmajor(sA, ra, tid);
  if (BKM) store_kmajor(sB, rb, tid); else store_mnmajor(sB, rb, tid);
}

__device__ __forceinline__ uint4 frag(const u16* sm, int row, int chunk) {
  return *reinterpret_cast<const uint4*>(sm + row * BK + ((chunk ^ swz(row)) << 3));
}

template <bool F16>
__device__ __forceinline__ floatx16 mfma(uint4 a, uint4 b, floatx16 c) {
  if constexpr (F16) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8_t, a),
                                                 __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                  __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  }
}

// Work-group id -> (split, tm, tn).
__device__ __forceinline__ void tile_coords(const KParams& p, bool sym, int& split, int& tm,
                                            int& tn) {
  const int nb = gridDim.x;
  const int b = blockIdx.x;
  // consecutive remapped ids share an XCD (ids are dealt round-robin to 8 XCDs)
  const int per = nb / 8, rem = nb % 8;
  const int xcd = b % 8, idx = b / 8;
  const int bb = (xcd < rem) ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
  split = bb / p.ntiles;
  int t = bb - split * p.ntiles;
  if (sym) {
    int row = 0, cnt = p.tiles_n;
    while (t >= cnt) { t -= cnt; ++row; --cnt; }
    tm = row;
    tn = row + t;
  } else {
    const int G = 8;
    const int per_group = G * p.tiles_n;
    const int g = t / per_group;
    const int first = g * G;
    const int gs = min(G, p.tiles_m - first);
    const int in = t - g * per_group;
    tm = first + in % gs;
    tn = in / gs;
  }
}

// Byte offsets, fixed for the whole tile, of a thread's global loads relative to the
// stage base (operand origin of the tile at the stage's first k), of its LDS stores and
// of its MFMA fragment reads.
template <bool KM>
__device__ __forceinline__ void load_offsets(int64_t ld, uint32_t (&g)[8], uint32_t (&st)[8],
                                             int tid) {
  if (KM) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int c = tid + NT * i;
      const int row = c >> 3, kc = c & 7;
      g[i] = (uint32_t)(((int64_t)row * ld + kc * 8) * 2);
      st[i] = (uint32_t)((row * BK + ((kc ^ swz(row)) << 3)) * 2);
    }
  } else {
    const int kb = tid >> 5, mb = tid & 31;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      g[i] = (uint32_t)(((int64_t)(kb * 8 + i) * ld + mb * 8) * 2);
      const int row = mb * 8 + i;   // store row of output vector i after the transpose
      st[i] = (uint32_t)((row * BK + ((kb ^ swz(row)) << 3)) * 2);
    }
  }
}

__device__ __forceinline__ void fast_load(const char* base, const uint32_t (&g)[8], uint4 (&r)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = *reinterpret_cast<const uint4*>(base + g[i]);
}

template <bool KM>
__device__ __forceinline__ void fast_store(char* sm, const uint32_t (&st)[8], const uint4 (&r)[8]) {
  if (KM) {
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<uint4*>(sm + st[i]) = r[i];
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      uint32_t o[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const uint32_t lo = dw(r[2 * kk], j >> 1);
        const uint32_t hi = dw(r[2 * kk + 1], j >> 1);
        o[kk] = (j & 1) ? __builtin_amdgcn_perm(hi, lo, 0x07060302u)
                        : __builtin_amdgcn_perm(hi, lo, 0x05040100u);
      }
      *reinterpret_cast<uint4*>(sm + st[j]) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
}

template <bool AK, bool BKM, bool F16, int EPI>
__global__ __launch_bounds__(NT, 1) void k_gemm(KParams p) {
  __shared__ __attribute__((aligned(16))) u16 smem[2 * 2 * TILE_ELEMS];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr bool SYM = (EPI == EPI_SYM || EPI == EPI_PARTIAL);

  int split, tm, tn;
  tile_coords(p, SYM, split, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  int kbeg = 0, kend = p.K;
  if (EPI == EPI_PARTIAL) {
    kbeg = split * p.k_per_split;
    kend = min(p.K, kbeg + p.k_per_split);
  }
  const int nkt = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
  const int nstage = nkt * p.npass;
  // interior tiles with 16-byte aligned operands take the check-free loaders for every
  // full K step
  const bool interior = (m0 + BM <= p.M) && (n0 + BN <= p.N) && p.aligned_a && p.aligned_b;

  uint32_t ga[8], gb[8], sa[8], sb[8];
  load_offsets<AK>(p.lda, ga, sa, tid);
  load_offsets<BKM>(p.ldb, gb, sb, tid);
  // fragment offsets (bytes) for the 4 row blocks x 4 k16 sub-steps of each operand
  uint32_t fa[4][4], fb[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int chunk = kk * 2 + (lane >> 5);
      const int ra = wm * 128 + i * 32 + (lane & 31);
      const int rb = wn * 128 + i * 32 + (lane & 31);
      fa[i][kk] = (uint32_t)((ra * BK + ((chunk ^ swz(ra)) << 3)) * 2);
      fb[i][kk] = (uint32_t)((rb * BK + ((chunk ^ swz(rb)) << 3)) * 2);
    }

  floatx16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // stage s -> (pass, k0); the stage's operand origins
  auto stage_k0 = [&](int s, int& pass) {
    pass = s / nkt;
    return kbeg + (s - pass * nkt) * BK;
  };
  auto origin = [&](int pass, int k0, const char*& A, const char*& B) {
    const int pa = pass == 0 ? p.pa0 : (pass == 1 ? p.pa1 : p.pa2);
    const int pb = pass == 0 ? p.pb0 : (pass == 1 ? p.pb1 : p.pb2);
    const u16* a = pa ? p.a1 : p.a0;
    const u16* b = pb ? p.b1 : p.b0;
    A = reinterpret_cast<const char*>(AK ? a + (int64_t)m0 * p.lda + k0 : a + (int64_t)k0 * p.lda + m0);
    B = reinterpret_cast<const char*>(BKM ? b + (int64_t)n0 * p.ldb + k0 : b + (int64_t)k0 * p.ldb + n0);
  };

  uint4 ra[8], rb[8];
  auto fetch = [&](int s) {
    int pass;
    const int k0 = stage_k0(s, pass);
    if (interior && k0 + BK <= kend) {
      const char* A;
      const char* B;
      origin(pass, k0, A, B);
      fast_load(A, ga, ra);
      fast_load(B, gb, rb);
    } else {
      load_stage<AK, BKM>(p, s, nkt, kbeg, m0, n0, ra, rb, tid);
    }
  };
  auto put = [&](int s, char* sA, char* sB) {
    int pass;
    const int k0 = stage_k0(s, pass);
    if (interior && k0 + BK <= kend) {
      fast_store<AK>(sA, sa, ra);
      fast_store<BKM>(sB, sb, rb);
    } else {
      store_stage<AK, BKM>(reinterpret_cast<u16*>(sA), reinterpret_cast<u16*>(sB), ra, rb, tid);
    }
  };

  char* sm = reinterpret_cast<char*>(smem);
  constexpr int OPB = TILE_ELEMS * 2;      // bytes per operand per stage
  if (nstage > 0) {
    fetch(0);
    put(0, sm, sm + OPB);
  }
  __syncthreads();

  for (int s = 0; s < nstage; ++s) {
    const int buf = s & 1;
    const char* sA = sm + buf * 2 * OPB;
    const char* sB = sA + OPB;
    const bool more = (s + 1) < nstage;
    if (more) fetch(s + 1);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      uint4 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) af[i] = *reinterpret_cast<const uint4*>(sA + fa[i][kk]);
#pragma unroll
      for (int j = 0; j < 4; ++j) bfr[j] = *reinterpret_cast<const uint4*>(sB + fb[j][kk]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma<F16>(af[i], bfr[j], acc[i][j]);
    }
    if (more) {
      char* nA = sm + (buf ^ 1) * 2 * OPB;
      put(s + 1, nA, nA + OPB);
    }
    __syncthreads();
  }

  // ---------------------------------------------------------------- epilogue
  // 32x32 accumulator layout: value v of lane l is row 8*(v/4) + 4*(l/32) + v%4,
  // column l%32 of its 32 x 32 block.
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int rl = wm * 128 + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
        const int cl = wn * 128 + j * 32 + (lane & 31);
        const int row = m0 + rl, col = n0 + cl;
        const float x = acc[i][j][v];
        if (EPI == EPI_PARTIAL) {
          float* dst = p.part + (int64_t)split * p.ntiles * (BM * BN);
          // tile-major: tile index of (tm, tn) in the upper triangle
          const int tidx = tm * p.tiles_n - (tm * (tm - 1)) / 2 + (tn - tm);
          dst[(int64_t)tidx * (BM * BN) + rl * BN + cl] = x;
        } else if (EPI == EPI_SPLIT) {
          if (row < p.M && col < p.ldc_pad) {
            const bool in = col < p.N;
            const uint32_t h = in ? bf16_rne_bits(x) : 0u;
            const uint32_t l = in ? bf16_rne_bits(x - __uint_as_float(h << 16)) : 0u;
            p.c_hi[(int64_t)row * p.ldc + col] = (u16)h;
            p.c_lo[(int64_t)row * p.ldc + col] = (u16)l;
          }
        } else if (row < p.M && col < p.N) {
          if (EPI == EPI_F32) {
            p.c[(int64_t)row * p.ldc + col] = x;
          } else {  // EPI_SYM
            if (row <= col) {
              p.c[(int64_t)row * p.ldc + col] = x;
              p.c[(int64_t)col * p.ldc + row] = x;
            }
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------------ async GEMM
// Global tiles go straight to LDS with global_load_lds_dwordx4 (no register staging)
// through a 5-stage ring of 256 x 32 tiles (all 160 KiB of LDS) fetched four stages ahead; one barrier per
// stage.  K must be a multiple of 32 (operand planes are zero-padded in K).
//  * K-major operand (X(r, k) at x[r * ld + k]): LDS rows r of 4 chunks of 8 k-values,
//    chunk c stored in slot c ^ ((r >> 2) & 3); fragments are plain 16-byte reads.
//    Rows beyond M (N) are read from the last valid row; their results are discarded.
//  * M/N-major operand (X(r, k) at x[k * ld + r]): LDS rows k of 32 chunks of 8 r-values,
//    chunk x stored in slot x ^ (4 (k & 3)); fragments come from two
//    ds_read_b64_tr_b16 per MFMA operand (inside a group of 16 lanes, lane j supplies
//    4 values of k-row j / 4 and lane i receives the 4 k-values of column i).  Requires
//    M (N) to be a multiple of 8; columns beyond are read from the last valid chunk.
// All fragment reads are bank-conflict free.
constexpr int ABK = 32, ANST = 5;
constexpr int ATILE = BM * ABK;                  // u16 elements per operand per stage

struct AParams {
  int M, N, K;
  const u16* a0; const u16* a1;
  const u16* b0; const u16* b1;
  int64_t lda, ldb;
  int npass;
  int pa0, pa1, pa2, pb0, pb1, pb2;
  float* c; int64_t ldc;
  u16* c_hi; u16* c_lo;
  int ldc_pad;          // EPI_SPLIT: columns [N, ldc_pad) of the output are written as 0
  int tiles_m, tiles_n, ntiles;
  int ksplit, k_per_split;
  float* part;
  int tile0, tcount;    // this launch covers tiles [tile0, tile0 + tcount) (x ksplit)
  int ra, rb;           // row extents the operand loads are clamped to (see gemm_run)
  int64_t bsa, bsb, bsc;  // element strides of A, B and C between the products of a batch
  int rowmap;             // EPI_F32: row r stored at row (r / 2) rowmap + r % 2 when > 0
};

typedef __attribute__((address_space(3))) void lds_void;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

// s_waitcnt immediate that waits for vmcnt <= n and leaves expcnt / lgkmcnt alone
constexpr unsigned waitcnt_vm(unsigned n) {
  return (n & 15u) | ((n >> 4) << 14) | (7u << 4) | (15u << 8);
}

// One 16-byte-per-lane DMA from global memory (wave-uniform base + per-lane offset) into
// 1 KiB of LDS at lds + 16 * lane.  Issued as inline assembly so that the compiler's wait
// insertion does not treat every later LDS read as dependent on it: completion is
// tracked by the explicit vmcnt waits of the ring.
__device__ __forceinline__ void dma16(const char* base, uint32_t off, char* lds) {
  const uint32_t l = (uint32_t)(uintptr_t)(lds_void*)lds;
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(off), "s"(base), "s"(l)
               : "memory", "m0");
}

// Per-lane DMA byte offsets (relative to the stage origin) of the NI chunks a lane moves
// per operand and stage (NI = 1024 chunks / (64 lanes x waves)).
template <bool MN, int NI>
__device__ __forceinline__ void dma_offsets(int64_t ld, int r0, int R, int wave, int lane,
                                            uint32_t (&g)[NI]) {
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int slot = (wave * NI + i) * 64 + lane;
    if (MN) {
      const int k = slot >> 5;
      const int x = (slot & 31) ^ ((k & 3) << 2);
      const int r = min(r0 + 8 * x, R - 8) - r0;
      g[i] = (uint32_t)(((int64_t)k * ld + r) * 2);
    } else {
      const int row = slot >> 2;
      const int c = (slot & 3) ^ ((row >> 2) & 3);
      const int r = min(r0 + row, R - 1) - r0;
      g[i] = (uint32_t)(((int64_t)r * ld + c * 8) * 2);
    }
  }
}

// Fragment read offsets of the NB row blocks (32 rows each) a wave owns, starting at row
// r0w of the tile.  K-major: f[i][kk] are full byte offsets; M/N-major: f[i][0] is the
// first of the block's transpose reads (the others sit at fixed immediate distances).
template <bool MN, int NB>
__device__ __forceinline__ void frag_offsets(int r0w, int lane, uint32_t (&f)[NB][2]) {
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    if (MN) {
      const int j = lane & 15;
      const int g = lane >> 5;
      const int mb = 16 * ((lane >> 4) & 1);
      const int m = r0w + i * 32 + mb + 4 * (j & 3);
      const int k = 8 * g + (j >> 2);
      const int x = (m >> 3) ^ ((k & 3) << 2);
      f[i][0] = (uint32_t)(k * 512 + x * 16 + (m & 7) * 2);
      f[i][1] = 0;
    } else {
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int chunk = kk * 2 + (lane >> 5);
        const int r = r0w + i * 32 + (lane & 31);
        f[i][kk] = (uint32_t)(r * 64 + ((chunk ^ ((r >> 2) & 3)) << 4));
      }
    }
  }
}

template <bool MN, int NB>
__device__ __forceinline__ uint4 afrag(const char* base, const uint32_t (&f)[NB][2], int i, int kk) {
  if (MN) {
    // k rows 16 kk + 8 g + (0..3) and + 4 .. 7: two transpose reads 4 k-rows apart
    const char* p0 = base + f[i][0] + kk * 16 * 512;
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p0 + 4 * 512));
    uint4 r;
    r.x = ((uint32_t)(uint16_t)lo[0]) | ((uint32_t)(uint16_t)lo[1] << 16);
    r.y = ((uint32_t)(uint16_t)lo[2]) | ((uint32_t)(uint16_t)lo[3] << 16);
    r.z = ((uint32_t)(uint16_t)hi[0]) | ((uint32_t)(uint16_t)hi[1] << 16);
    r.w = ((uint32_t)(uint16_t)hi[2]) | ((uint32_t)(uint16_t)hi[3] << 16);
    return r;
  } else {
    return *reinterpret_cast<const uint4*>(base + f[i][kk]);
  }
}

// WAVES = 4: 2 x 2 waves of 128 x 128.  WAVES = 8: 2 x 4 waves of 128 x 64 (two waves per
// SIMD, so one wave's memory waits overlap the other's MFMAs).
template <bool AMN, bool BMN, bool F16, int EPI, int WAVES>
__global__ __launch_bounds__(64 * WAVES, 1) void k_gemm_async(AParams p) {
  constexpr int NBM = 4;                         // 32-row blocks per wave in m
  constexpr int NBN = WAVES == 4 ? 4 : 2;        // 32-col blocks per wave in n
  constexpr int WN = WAVES == 4 ? 2 : 4;         // waves along n
  constexpr int NI = 1024 / (64 * WAVES);        // DMA chunks per lane per operand and stage
  // one LDS object per ring stage, so that the compiler can tell the DMA writes of the
  // stages in flight from the reads of the stage being consumed
  __shared__ __attribute__((aligned(16))) u16 st0[2 * ATILE];
  __shared__ __attribute__((aligned(16))) u16 st1[2 * ATILE];
  __shared__ __attribute__((aligned(16))) u16 st2[2 * ATILE];
  __shared__ __attribute__((aligned(16))) u16 st3[2 * ATILE];
  __shared__ __attribute__((aligned(16))) u16 st4[2 * ATILE];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  constexpr bool SYM = (EPI == EPI_SYM || EPI == EPI_PARTIAL);

  // work-group id -> (split, tile): each XCD (ids dealt round-robin to 8) takes a
  // contiguous range; symmetric products walk the upper triangle row by row, the others
  // go down groups of 8 tile-rows column by column
  int split, tm, tn, tloc;
  {
    const int nb = gridDim.x, bid = blockIdx.x;
    const int per = nb / 8, rem = nb % 8;
    const int xcd = bid % 8, idx = bid / 8;
    const int bb = (xcd < rem) ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
    split = bb / p.tcount;
    tloc = bb - split * p.tcount;
    int t = p.tile0 + tloc;
    if (SYM) {
      // upper tiles in super-blocks of 8 x 8 tiles (diagonal ones triangular), each walked
      // row by row: the work-groups that run together on an XCD read few distinct
      // operand blocks
      const int nsb = (p.tiles_n + 7) / 8;
      int I = 0, J = 0;
      for (;;) {
        const int nr = min(8, p.tiles_n - 8 * I), nc = min(8, p.tiles_n - 8 * J);
        const int cnt = (I == J) ? nr * (nr + 1) / 2 : nr * nc;
        if (t < cnt || (I == nsb - 1 && J == nsb - 1)) break;
        t -= cnt;
        if (++J == nsb) { ++I; J = I; }
      }
      if (I == J) {
        int r = 0, cnt = min(8, p.tiles_n - 8 * I);
        while (t >= cnt) { t -= cnt; ++r; --cnt; }
        tm = 8 * I + r;
        tn = tm + t;
      } else {
        const int nc = min(8, p.tiles_n - 8 * J);
        tm = 8 * I + t / nc;
        tn = 8 * J + t % nc;
      }
    } else {
      const int G = 8;
      const int g = t / (G * p.tiles_n);
      const int first = g * G;
      const int gs = min(G, p.tiles_m - first);
      const int in = t - g * G * p.tiles_n;
      tm = first + in % gs;
      tn = in / gs;
    }
  }
  const int m0 = tm * BM, n0 = tn * BN;
  int kbeg = 0, kend = p.K;
  if (EPI == EPI_PARTIAL || EPI == EPI_TAIL) {
    kbeg = split * p.k_per_split;
    kend = min(p.K, kbeg + p.k_per_split);
  }
  const int nkt = kend > kbeg ? (kend - kbeg) / ABK : 0;
  const int nstage = nkt * p.npass;

  uint32_t ga[NI], gb[NI];
  dma_offsets<AMN, NI>(p.lda, m0, p.ra, wave, lane, ga);
  dma_offsets<BMN, NI>(p.ldb, n0, p.rb, wave, lane, gb);
  uint32_t fa[NBM][2], fb[NBN][2];
  frag_offsets<AMN, NBM>(wm * 128, lane, fa);
  frag_offsets<BMN, NBN>(wn * 32 * NBN, lane, fb);

  floatx16 acc[NBM][NBN];
#pragma unroll
  for (int i = 0; i < NBM; ++i)
#pragma unroll
    for (int j = 0; j < NBN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  // Operand origins of each pass for this work-group's K range; inside a pass the stage
  // origin advances by a fixed byte step, so the issue path is pointer increments only.
  const int64_t bz = blockIdx.y;                 // product of a batch (0 when unbatched)
  auto a_origin = [&](int sel) {
    const u16* a = (sel ? p.a1 : p.a0) + bz * p.bsa;
    return reinterpret_cast<const char*>(AMN ? a + (int64_t)kbeg * p.lda + m0
                                             : a + (int64_t)m0 * p.lda + kbeg);
  };
  auto b_origin = [&](int sel) {
    const u16* b = (sel ? p.b1 : p.b0) + bz * p.bsb;
    return reinterpret_cast<const char*>(BMN ? b + (int64_t)kbeg * p.ldb + n0
                                             : b + (int64_t)n0 * p.ldb + kbeg);
  };
  const char* const oa1 = a_origin(p.pa1);
  const char* const oa2 = a_origin(p.pa2);
  const char* const ob1 = b_origin(p.pb1);
  const char* const ob2 = b_origin(p.pb2);
  const int64_t astep = AMN ? (int64_t)ABK * p.lda * 2 : (int64_t)ABK * 2;
  const int64_t bstep = BMN ? (int64_t)ABK * p.ldb * 2 : (int64_t)ABK * 2;
  const char* iA = a_origin(p.pa0);
  const char* iB = b_origin(p.pb0);
  int ikt = 0, ipass = 0;
  constexpr int OPB = ATILE * 2;                 // bytes per operand per stage
  // DMA of the next stage in issue order into ring slot dst
  auto issue = [&](char* dst) {
    char* dA = dst + wave * NI * 1024;
    char* dB = dA + OPB;
#pragma unroll
    for (int i = 0; i < NI; ++i) dma16(iA, ga[i], dA + i * 1024);
#pragma unroll
    for (int i = 0; i < NI; ++i) dma16(iB, gb[i], dB + i * 1024);
    iA += astep;
    iB += bstep;
    if (++ikt == nkt) {
      ikt = 0;
      ++ipass;
      iA = ipass == 1 ? oa1 : oa2;
      iB = ipass == 1 ? ob1 : ob2;
    }
  };
  auto load = [&](const char* sA, int kk, uint4 (&af)[NBM], uint4 (&bf)[NBN]) {
    const char* sB = sA + OPB;
#pragma unroll
    for (int i = 0; i < NBM; ++i) af[i] = afrag<AMN, NBM>(sA, fa, i, kk);
#pragma unroll
    for (int j = 0; j < NBN; ++j) bf[j] = afrag<BMN, NBN>(sB, fb, j, kk);
  };
  auto mma = [&](const uint4 (&af)[NBM], const uint4 (&bf)[NBN]) {
#pragma unroll
    for (int i = 0; i < NBM; ++i)
#pragma unroll
      for (int j = 0; j < NBN; ++j) acc[i][j] = mfma<F16>(af[i], bf[j], acc[i][j]);
  };
  // Work-group barrier without a memory fence: the only cross-wave traffic is LDS, made
  // safe by the explicit vmcnt waits (DMA landed) and by register dependencies (reads
  // done); a fenced barrier would wait for every DMA in flight.
  auto barrier = [] {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  // Software pipeline over a 5-slot ring (all of the LDS) with stages s + 1 .. s + 3 in
  // flight while stage s is multiplied; fragments of the next k-slice are read from LDS while the
  // current one is in the matrix cores.
  constexpr unsigned PER = 2 * NI;               // DMA instructions per stage and wave
  uint4 a0[NBM], b0[NBN], a1[NBM], b1[NBN];
  // LDS reads per fragment set and MFMAs per k-slice, for the interleaving hints
  constexpr int NDS = (AMN ? 2 * NBM : NBM) + (BMN ? 2 * NBN : NBN);
  constexpr int NMF = NBM * NBN;
  auto interleave = [] {
#pragma unroll
    for (int i = 0; i < NMF; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                      // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, (NDS + NMF - 1) / NMF, 0);  // LDS reads
    }
  };
  // wait until this wave's DMA of stage t has landed, given the last stage issued
  auto wait_stage = [&](int t, int issued_last) {
    const int ahead = issued_last - t;          // stages issued after t
    if (ahead >= 3) __builtin_amdgcn_s_waitcnt(waitcnt_vm(3 * PER));
    else if (ahead == 2) __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * PER));
    else if (ahead == 1) __builtin_amdgcn_s_waitcnt(waitcnt_vm(PER));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  };
  auto step = [&](int s, const char* cur, const char* nxt, char* refill) {
    load(cur, 1, a1, b1);
    mma(a0, b0);
    interleave();
    if (s + 1 < nstage) {
      wait_stage(s + 1, min(nstage - 1, s + ANST - 2));
      barrier();
      if (s + ANST - 1 < nstage) issue(refill);
      load(nxt, 0, a0, b0);
    }
    mma(a1, b1);
    interleave();
  };

  // steady-state step: stages s + 1 .. s + 3 issued, stage s + 4 exists; straight-line
  // code, so that the wait counts before the MFMAs cover only the reads they need
  auto step_full = [&](const char* cur, const char* nxt, char* refill) {
    load(cur, 1, a1, b1);
    mma(a0, b0);
    interleave();
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * PER));
    barrier();
    issue(refill);
    load(nxt, 0, a0, b0);
    mma(a1, b1);
    interleave();
  };

  char* const r0 = reinterpret_cast<char*>(st0);
  char* const r1 = reinterpret_cast<char*>(st1);
  char* const r2 = reinterpret_cast<char*>(st2);
  char* const r3 = reinterpret_cast<char*>(st3);
  char* const r4 = reinterpret_cast<char*>(st4);
  if (nstage > 0) {
    issue(r0);
    if (nstage > 1) issue(r1);
    if (nstage > 2) issue(r2);
    if (nstage > 3) issue(r3);
    wait_stage(0, min(nstage - 1, ANST - 2));
    barrier();
    load(r0, 0, a0, b0);
  }
  int s0 = 0;
  for (; s0 + 8 < nstage; s0 += 5) {
    step_full(r0, r1, r4);
    step_full(r1, r2, r0);
    step_full(r2, r3, r1);
    step_full(r3, r4, r2);
    step_full(r4, r0, r3);
  }
  for (int s = s0; s < nstage; s += 5) {
    step(s, r0, r1, r4);
    if (s + 1 < nstage) step(s + 1, r1, r2, r0);
    if (s + 2 < nstage) step(s + 2, r2, r3, r1);
    if (s + 3 < nstage) step(s + 3, r3, r4, r2);
    if (s + 4 < nstage) step(s + 4, r4, r0, r3);
  }

  // 32x32 accumulator layout: value v of lane l is row 8*(v/4) + 4*(l/32) + v%4,
  // column l%32 of its 32 x 32 block.
#pragma unroll
  for (int i = 0; i < NBM; ++i) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int rl = wm * 128 + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3);
      const int row = m0 + rl;
      if (EPI != EPI_PARTIAL && EPI != EPI_TAIL && row >= p.M) continue;
#pragma unroll
      for (int j = 0; j < NBN; ++j) {
        const int cl = wn * 32 * NBN + j * 32 + (lane & 31);
        const int col = n0 + cl;
        const float x = acc[i][j][v];
        if (EPI == EPI_PARTIAL) {
          const int tidx = tm * p.tiles_n - (tm * (tm - 1)) / 2 + (tn - tm);
          p.part[((int64_t)split * p.ntiles + tidx) * (BM * BN) + rl * BN + cl] = x;
        } else if (EPI == EPI_TAIL) {
          p.part[((int64_t)split * p.tcount + tloc) * (BM * BN) + rl * BN + cl] = x;
        } else if (EPI == EPI_F32) {
          const int64_t orow = p.rowmap > 0 ? (int64_t)(row >> 1) * p.rowmap + (row & 1) : row;
          if (col < p.N) p.c[bz * p.bsc + orow * p.ldc + col] = x;
        } else if (EPI == EPI_SPLIT) {
          if (col < p.ldc_pad) {
            const bool in = col < p.N;
            const uint32_t h = in ? bf16_rne_bits(x) : 0u;
            const uint32_t l = in ? bf16_rne_bits(x - __uint_as_float(h << 16)) : 0u;
            p.c_hi[(int64_t)row * p.ldc + col] = (u16)h;
            p.c_lo[(int64_t)row * p.ldc + col] = (u16)l;
          }
        } else {  // EPI_SYM
          if (col < p.N && row <= col) {
            p.c[(int64_t)row * p.ldc + col] = x;
            p.c[(int64_t)col * p.ldc + row] = x;
          }
        }
      }
    }
  }
}

// ------------------------------------------------------------------ tail reduction
// Tiles [tile0, tile0 + tcount) of a non-symmetric product computed as ksplit K-slices:
// sum the slices (fp64) and apply the product's epilogue.  One thread per 4 columns.
__global__ __launch_bounds__(256) void k_tail_reduce(const float* __restrict__ part, int ksplit,
                                                     int tile0, int tcount, int tiles_m,
                                                     int tiles_n, int M, int N, int epi,
                                                     float* __restrict__ c, int64_t ldc,
                                                     u16* __restrict__ c_hi,
                                                     u16* __restrict__ c_lo, int ldc_pad) {
  const int tloc = blockIdx.y;
  const int t = tile0 + tloc;
  const int G = 8;
  const int g = t / (G * tiles_n);
  const int first = g * G;
  const int gs = min(G, tiles_m - first);
  const int in = t - g * G * tiles_n;
  const int tm = first + in % gs, tn = in / gs;
  const int e0 = (blockIdx.x * 256 + threadIdx.x) * 4;     // element of the 256 x 256 tile
  if (e0 >= BM * BN) return;
  const int rl = e0 / BN, cl = e0 % BN;
  const int row = tm * BM + rl;
  if (row >= M) return;
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int sp = 0; sp < ksplit; ++sp) {
    const float4 v = *reinterpret_cast<const float4*>(part + ((int64_t)sp * tcount + tloc) * (BM * BN) + e0);
    acc[0] += v.x; acc[1] += v.y; acc[2] += v.z; acc[3] += v.w;
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int col = tn * BN + cl + q;
    const float x = (float)acc[q];
    if (epi == EPI_F32) {
      if (col < N) c[(int64_t)row * ldc + col] = x;
    } else if (col < ldc_pad) {
      const bool inb = col < N;
      const uint32_t h = inb ? bf16_rne_bits(x) : 0u;
      const uint32_t l = inb ? bf16_rne_bits(x - __uint_as_float(h << 16)) : 0u;
      c_hi[(int64_t)row * ldc + col] = (u16)h;
      c_lo[(int64_t)row * ldc + col] = (u16)l;
    }
  }
}

// ------------------------------------------------------------------ split-K reduction
// One work-group per (upper tile, 64 x 64 sub-block).  Sums the partial tiles in fp64,
// adds the old H when accumulating, writes H[i][j] and (through LDS) H[j][i], i <= j.
__global__ __launch_bounds__(256) void k_syrk_reduce(const float* __restrict__ part, int N,
                                                     int tiles, int ntiles, int ksplit,
                                                     float* __restrict__ H, int64_t ldh,
                                                     int accumulate) {
  __shared__ float tr[64][65];
  const int sub = blockIdx.x & 15;
  int t = blockIdx.x >> 4;
  const int sr = sub >> 2, sc = sub & 3;
  int tm = 0, cnt = tiles;
  while (t >= cnt) { t -= cnt; ++tm; --cnt; }
  const int tn = tm + t;
  const int tidx = blockIdx.x >> 4;
  const int i0 = tm * BM + sr * 64, j0 = tn * BN + sc * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  // sums: 4 consecutive columns per thread (16-byte loads), the splits in order, up to
  // sixteen loads in flight at a time
  const int c4 = (threadIdx.x & 15) * 4, rq = threadIdx.x >> 4;
  const int64_t sstride = (int64_t)ntiles * (BM * BN);
  for (int r = rq; r < 64; r += 16) {
    const float* p0 = part + (int64_t)tidx * (BM * BN) + (int64_t)(sr * 64 + r) * BN + sc * 64 + c4;
    double sum[4] = {0.0, 0.0, 0.0, 0.0};
    int s = 0;
    for (; s + 16 <= ksplit; s += 16) {
      float4 v[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) v[q] = *reinterpret_cast<const float4*>(p0 + (s + q) * sstride);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        sum[0] += v[q].x; sum[1] += v[q].y; sum[2] += v[q].z; sum[3] += v[q].w;
      }
    }
    if (s < ksplit) {         // the rest (fewer than 16), all loaded before the sums
      float4 v[16];
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (s + q < ksplit) v[q] = *reinterpret_cast<const float4*>(p0 + (s + q) * sstride);
#pragma unroll
      for (int q = 0; q < 16; ++q)
        if (s + q < ksplit) {
          sum[0] += v[q].x; sum[1] += v[q].y; sum[2] += v[q].z; sum[3] += v[q].w;
        }
    }
    const int i = i0 + r;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int j = j0 + c4 + q;
      float v = 0.f;
      if (i < N && j < N) {
        const int ii = i <= j ? i : j, jj = i <= j ? j : i;
        if (accumulate) sum[q] += (double)H[(int64_t)ii * ldh + jj];
        v = (float)sum[q];
        if (i <= j) H[(int64_t)i * ldh + j] = v;
      }
      tr[r][c4 + q] = v;
    }
  }
  __syncthreads();
  // transposed write: element (i0 + c, j0 + r') -> H[j0 + r'][i0 + c]
  for (int r = ty; r < 64; r += 4) {
    const int j = j0 + r, i = i0 + tx;
    if (i < N && j < N && i <= j) H[(int64_t)j * ldh + i] = tr[tx][r];
  }
}

// ------------------------------------------------------------------ elementwise
template <typename T>
__device__ __forceinline__ float ld_f(const T* p) { return (float)*p; }
template <>
__device__ __forceinline__ float ld_f<u16>(const u16* p) { return __uint_as_float((uint32_t)*p << 16); }

template <typename T>
__global__ void k_split(const T* __restrict__ in, int64_t ld_in, int rows, int cols,
                        const float* __restrict__ col_scale, u16* __restrict__ hi,
                        u16* __restrict__ lo, int64_t ld_out) {
  const int64_t total = (int64_t)rows * cols;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(e / cols), c = (int)(e - (int64_t)r * cols);
    float x = ld_f(in + (int64_t)r * ld_in + c);
    if (col_scale) x *= col_scale[c];
    const uint32_t h = bf16_rne_bits(x);
    const float hf = __uint_as_float(h << 16);
    hi[(int64_t)r * ld_out + c] = (u16)h;
    if (lo) lo[(int64_t)r * ld_out + c] = (u16)bf16_rne_bits(x - hf);
  }
}

// 4-wide variant for fp32 rows with cols % 4 == 0 and 16-byte aligned rows.
__global__ void k_split4(const float* __restrict__ in, int64_t ld_in, int rows, int cols,
                         const float* __restrict__ col_scale, u16* __restrict__ hi,
                         u16* __restrict__ lo, int64_t ld_out) {
  const int c4 = cols >> 2;
  const int64_t total = (int64_t)rows * c4;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(e / c4), c = (int)(e - (int64_t)r * c4) * 4;
    float4 x = *reinterpret_cast<const float4*>(in + (int64_t)r * ld_in + c);
    if (col_scale) {
      const float4 sc = *reinterpret_cast<const float4*>(col_scale + c);
      x.x *= sc.x; x.y *= sc.y; x.z *= sc.z; x.w *= sc.w;
    }
    const float xs[4] = {x.x, x.y, x.z, x.w};
    uint32_t h[4], l[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      h[q] = bf16_rne_bits(xs[q]);
      l[q] = bf16_rne_bits(xs[q] - __uint_as_float(h[q] << 16));
    }
    *reinterpret_cast<uint2*>(hi + (int64_t)r * ld_out + c) =
        make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    if (lo)
      *reinterpret_cast<uint2*>(lo + (int64_t)r * ld_out + c) =
          make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
  }
}

__global__ void k_fill_zero(float* p, int rows, int cols, int64_t ld) {
  const int64_t total = (int64_t)rows * cols;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int r = (int)(e / cols), c = (int)(e - (int64_t)r * cols);
    p[(int64_t)r * ld + c] = 0.f;
  }
}

// out[r * ld_out + c] = bf16 pair of in[r][c] (times col_scale[c]) for c < cols and 0 for
// cols <= c < ld_out (K padding).
// One thread per 4 output columns of a row (ld_out is a multiple of 4), rows across
// blockIdx.y: vector loads where the source row allows them, 8-byte stores per plane.
template <typename T>
__device__ __forceinline__ void ld4(const T* src, float (&x)[4], bool vec) {
  if constexpr (sizeof(T) == 4) {
    if (vec) {
      const float4 v = *reinterpret_cast<const float4*>(src);
      x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
      return;
    }
  } else {
    if (vec) {
      const uint2 v = *reinterpret_cast<const uint2*>(src);
      const T* e = reinterpret_cast<const T*>(&v);
#pragma unroll
      for (int q = 0; q < 4; ++q) x[q] = ld_f(e + q);
      return;
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) x[q] = ld_f(src + q);
}

template <typename T>
__global__ __launch_bounds__(256) void k_split_pad(const T* __restrict__ in, int64_t ld_in,
                                                   int rows, int cols,
                                                   const float* __restrict__ col_scale,
                                                   u16* __restrict__ hi, u16* __restrict__ lo,
                                                   int64_t ld_out, int rows_out) {
  const int64_t c0 = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (c0 >= ld_out) return;
  for (int64_t r = blockIdx.y; r < rows_out; r += gridDim.y) {
    float x[4] = {0.f, 0.f, 0.f, 0.f};
    if (r < rows && c0 < cols) {
      const T* src = in + r * ld_in + c0;
      if (c0 + 4 <= cols) {
        const bool vec = (reinterpret_cast<uintptr_t>(src) & (4 * sizeof(T) - 1)) == 0;
        ld4(src, x, vec);
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) x[q] = (c0 + q < cols) ? ld_f(src + q) : 0.f;
      }
      if (col_scale) {
#pragma unroll
        for (int q = 0; q < 4; ++q) x[q] *= (c0 + q < cols) ? col_scale[c0 + q] : 0.f;
      }
    }
    uint32_t h[4], l[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      h[q] = bf16_rne_bits(x[q]);
      l[q] = bf16_rne_bits(x[q] - __uint_as_float(h[q] << 16));
    }
    *reinterpret_cast<uint2*>(hi + r * ld_out + c0) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    if (lo)
      *reinterpret_cast<uint2*>(lo + r * ld_out + c0) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
  }
}

int grid_for(int64_t n, int per_block) {
  int64_t g = (n + per_block - 1) / per_block;
  if (g > 65536) g = 65536;
  if (g < 1) g = 1;
  return (int)g;
}

template <bool AK, bool BKM, bool F16, int EPI>
void launch(const KParams& p, int grid, hipStream_t s) {
  hipLaunchKernelGGL((k_gemm<AK, BKM, F16, EPI>), dim3(grid), dim3(NT), 0, s, p);
}

template <bool AK, bool BKM, bool F16>
bool dispatch_epi(const KParams& p, int epi, int grid, hipStream_t s) {
  switch (epi) {
    case EPI_F32: launch<AK, BKM, F16, EPI_F32>(p, grid, s); return true;
    case EPI_SPLIT: launch<AK, BKM, F16, EPI_SPLIT>(p, grid, s); return true;
    case EPI_SYM: launch<AK, BKM, F16, EPI_SYM>(p, grid, s); return true;
    case EPI_PARTIAL: launch<AK, BKM, F16, EPI_PARTIAL>(p, grid, s); return true;
  }
  return false;
}


// compute units of the current device (cached per device)
int compute_units() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cache[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

}  // namespace

size_t gemm_tail_bytes() { return (size_t)256 * BM * BN * sizeof(float); }

int64_t gemm_tiles(int64_t M, int64_t N) { return ((M + BM - 1) / BM) * ((N + BN - 1) / BN); }

int gemm_sym_tiles(int N) {
  const int t = (N + BN - 1) / BN;
  return t * (t + 1) / 2;
}

size_t gemm_partial_bytes(int N, int ksplit) {
  return (size_t)gemm_sym_tiles(N) * ksplit * BM * BN * sizeof(float);
}

hipError_t gemm_run(const GemmDesc& d, float* partial, hipStream_t s) {
  if (d.M <= 0 || d.N <= 0 || d.batch <= 0) return hipSuccess;
  if (d.batch > 1 && (d.epi != EPI_F32 || d.batch > 65535 || d.bsa % 8 || d.bsb % 8))
    return hipErrorInvalidValue;
  KParams p{};
  p.M = d.M; p.N = d.N; p.K = d.K;
  p.a0 = d.a[0]; p.a1 = d.a[1] ? d.a[1] : d.a[0];
  p.b0 = d.b[0]; p.b1 = d.b[1] ? d.b[1] : d.b[0];
  p.lda = d.lda; p.ldb = d.ldb;
  p.npass = d.npass;
  p.pa0 = d.pa[0]; p.pa1 = d.pa[1]; p.pa2 = d.pa[2];
  p.pb0 = d.pb[0]; p.pb1 = d.pb[1]; p.pb2 = d.pb[2];
  p.c = d.c; p.ldc = d.ldc; p.c_hi = d.c_hi; p.c_lo = d.c_lo;
  p.ldc_pad = (int)(d.ldc_pad > d.N ? d.ldc_pad : d.N);
  // 16-byte aligned rows; per-thread byte offsets inside a 256-row (or 64-row) stage
  // must fit in 32 bits
  auto al = [](const u16* q, int64_t ld) {
    return ((reinterpret_cast<uintptr_t>(q) & 15) == 0) && (ld % 8 == 0) && ld < (1 << 22);
  };
  p.aligned_a = al(p.a0, d.lda) && al(p.a1, d.lda);
  p.aligned_b = al(p.b0, d.ldb) && al(p.b1, d.ldb);
  p.tiles_m = (d.M + BM - 1) / BM;
  p.tiles_n = (d.N + BN - 1) / BN;
  const bool sym = d.epi == EPI_SYM || d.epi == EPI_PARTIAL;
  p.ntiles = sym ? p.tiles_n * (p.tiles_n + 1) / 2 : p.tiles_m * p.tiles_n;
  p.ksplit = d.epi == EPI_PARTIAL ? d.ksplit : 1;
  const int kt_total = (d.K + BK - 1) / BK;
  const int kt_per = (kt_total + p.ksplit - 1) / p.ksplit;
  p.k_per_split = kt_per * BK;
  p.part = partial;
  const int grid = p.ntiles * p.ksplit;
  // asynchronous path: K a multiple of 32 (of each K-split), 16-byte aligned operands;
  // an M/N-major operand is loaded in 8-element pieces, so its extent must be a multiple
  // of 8 or its rows must hold the extent rounded up to 8 (the extra elements only reach
  // output rows / columns that are never stored)
  const bool kp_ok = (p.k_per_split % ABK == 0) && (d.K % ABK == 0);
  const int m8 = (d.M + 7) / 8 * 8, n8 = (d.N + 7) / 8 * 8;
  const bool mn_ok = (d.a_kmajor || d.M % 8 == 0 || d.lda >= m8) &&
                     (d.b_kmajor || d.N % 8 == 0 || d.ldb >= n8);
  if (kp_ok && mn_ok && p.aligned_a && p.aligned_b) {
    AParams q{};
    q.M = d.M; q.N = d.N; q.K = d.K;
    q.a0 = p.a0; q.a1 = p.a1; q.b0 = p.b0; q.b1 = p.b1; q.lda = d.lda; q.ldb = d.ldb;
    q.npass = d.npass;
    q.pa0 = p.pa0; q.pa1 = p.pa1; q.pa2 = p.pa2; q.pb0 = p.pb0; q.pb1 = p.pb1; q.pb2 = p.pb2;
    q.c = d.c; q.ldc = d.ldc; q.c_hi = d.c_hi; q.c_lo = d.c_lo; q.ldc_pad = p.ldc_pad;
    q.tiles_m = p.tiles_m; q.tiles_n = p.tiles_n; q.ntiles = p.ntiles;
    q.ksplit = p.ksplit; q.k_per_split = p.k_per_split; q.part = partial;
    q.ra = d.a_kmajor ? d.M : m8;
    q.rb = d.b_kmajor ? d.N : n8;
    q.bsa = d.bsa; q.bsb = d.bsb; q.bsc = d.bsc;
    q.rowmap = d.epi == EPI_F32 ? d.rowmap : 0;
    const unsigned nbatch = (unsigned)d.batch;
    prof_begin(s, d.name);
#define FQ_LAUNCH_ASYNC_E(AMN, BMN, F16, E, G)                                                        \
    hipLaunchKernelGGL((k_gemm_async<AMN, BMN, F16, E, 8>), dim3(G, nbatch), dim3(512), 0, s, q);
#define FQ_LAUNCH_ASYNC(AMN, BMN, F16, E, G)                                                           \
    switch (E) {                                                                                        \
      case EPI_F32: FQ_LAUNCH_ASYNC_E(AMN, BMN, F16, EPI_F32, G) break;                                 \
      case EPI_SPLIT: FQ_LAUNCH_ASYNC_E(AMN, BMN, F16, EPI_SPLIT, G) break;                             \
      case EPI_SYM: FQ_LAUNCH_ASYNC_E(AMN, BMN, F16, EPI_SYM, G) break;                                 \
      case EPI_TAIL: FQ_LAUNCH_ASYNC_E(AMN, BMN, F16, EPI_TAIL, G) break;                               \
      default: FQ_LAUNCH_ASYNC_E(AMN, BMN, F16, EPI_PARTIAL, G) break;                                  \
    }
    // 8 waves (2 per SIMD, 128 x 64 wave tiles) measured ahead of 4 waves of 128 x 128
    const bool amn = !d.a_kmajor, bmn = !d.b_kmajor;
    auto launch = [&](int epi, int g) {
      if (amn && bmn) {
        if (d.f16) { FQ_LAUNCH_ASYNC(true, true, true, epi, g) } else { FQ_LAUNCH_ASYNC(true, true, false, epi, g) }
      } else if (amn) {
        if (d.f16) { FQ_LAUNCH_ASYNC(true, false, true, epi, g) } else { FQ_LAUNCH_ASYNC(true, false, false, epi, g) }
      } else if (bmn) {
        if (d.f16) { FQ_LAUNCH_ASYNC(false, true, true, epi, g) } else { FQ_LAUNCH_ASYNC(false, true, false, epi, g) }
      } else {
        if (d.f16) { FQ_LAUNCH_ASYNC(false, false, true, epi, g) } else { FQ_LAUNCH_ASYNC(false, false, false, epi, g) }
      }
    };
    // A short last round of tiles (at most half the compute units busy) is split over K
    // into fp32 partial tiles and reduced with the product's epilogue.
    const int cus = compute_units();
    const int rounds = (p.ntiles + cus - 1) / cus;
    const int tail = p.ntiles - (rounds - 1) * cus;
    const int ksteps = d.K / ABK;
    int ts = (tail > 0) ? cus / tail : 0;
    if (ts > ksteps / 4) ts = ksteps / 4;
    const int kps = ts > 0 ? (ksteps + ts - 1) / ts : 0;   // k-steps per slice
    if (kps > 0) ts = (ksteps + kps - 1) / kps;              // no empty slice
    const bool use_tail = partial && d.batch == 1 && d.rowmap == 0 && rounds >= 2 && tail <= cus / 2 && ts >= 2 &&
                          (d.epi == EPI_F32 || d.epi == EPI_SPLIT) &&
                          (size_t)tail * ts * BM * BN * sizeof(float) <= gemm_tail_bytes();
    if (use_tail) {
      q.tile0 = 0;
      q.tcount = p.ntiles - tail;
      q.ksplit = 1;
      launch(d.epi, q.tcount);
      q.tile0 = p.ntiles - tail;
      q.tcount = tail;
      q.ksplit = ts;
      q.k_per_split = kps * ABK;
      q.part = partial;
      launch(EPI_TAIL, tail * ts);
      hipLaunchKernelGGL(k_tail_reduce, dim3(BM * BN / 1024, tail), dim3(256), 0, s, partial, ts,
                         q.tile0, tail, p.tiles_m, p.tiles_n, d.M, d.N, d.epi, d.c, d.ldc,
                         d.c_hi, d.c_lo, q.ldc_pad);
    } else {
      q.tile0 = 0;
      q.tcount = p.ntiles;
      launch(d.epi, grid);
    }
#undef FQ_LAUNCH_ASYNC_E
#undef FQ_LAUNCH_ASYNC
    prof_end(s);
    return last_launch_error();
  }
  // batches and row maps run on the asynchronous path only
  if (d.batch != 1 || d.rowmap != 0) return hipErrorInvalidValue;
  prof_begin(s, d.name);
  bool ok;
  if (d.a_kmajor && d.b_kmajor) {
    ok = d.f16 ? dispatch_epi<true, true, true>(p, d.epi, grid, s)
               : dispatch_epi<true, true, false>(p, d.epi, grid, s);
  } else if (d.a_kmajor && !d.b_kmajor) {
    ok = d.f16 ? dispatch_epi<true, false, true>(p, d.epi, grid, s)
               : dispatch_epi<true, false, false>(p, d.epi, grid, s);
  } else if (!d.a_kmajor && !d.b_kmajor) {
    ok = d.f16 ? dispatch_epi<false, false, true>(p, d.epi, grid, s)
               : dispatch_epi<false, false, false>(p, d.epi, grid, s);
  } else {
    ok = false;
  }
  prof_end(s);
  if (!ok) return hipErrorInvalidValue;
  return last_launch_error();
}

hipError_t syrk_reduce(const float* partial, int N, int ksplit, float* H, int64_t ldh,
                       int accumulate, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  const int tiles = (N + BN - 1) / BN;
  const int ntiles = tiles * (tiles + 1) / 2;
  prof_begin(s, "syrk_reduce");
  hipLaunchKernelGGL(k_syrk_reduce, dim3(ntiles * 16), dim3(256), 0, s, partial, N, tiles,
                     ntiles, ksplit, H, ldh, accumulate);
  prof_end(s);
  return last_launch_error();
}

hipError_t split_bf16(const void* in, int in_type, int64_t ld_in, int rows, int cols,
                      const float* col_scale, u16* hi, u16* lo, int64_t ld_out, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  prof_begin(s, "split_bf16");
  if (in_type == 0) {
    const bool vec = (cols % 4 == 0) && (ld_in % 4 == 0) && (ld_out % 4 == 0) &&
                     ((reinterpret_cast<uintptr_t>(in) & 15) == 0) &&
                     ((reinterpret_cast<uintptr_t>(hi) & 7) == 0) &&
                     (!lo || (reinterpret_cast<uintptr_t>(lo) & 7) == 0) &&
                     (!col_scale || (reinterpret_cast<uintptr_t>(col_scale) & 15) == 0);
    if (vec) {
      hipLaunchKernelGGL(k_split4, dim3(grid_for((int64_t)rows * cols / 4, 256)), dim3(256), 0, s,
                         (const float*)in, ld_in, rows, cols, col_scale, hi, lo, ld_out);
    } else {
      hipLaunchKernelGGL(k_split<float>, dim3(grid_for((int64_t)rows * cols, 256)), dim3(256), 0,
                         s, (const float*)in, ld_in, rows, cols, col_scale, hi, lo, ld_out);
    }
  } else {
    hipLaunchKernelGGL(k_split<_Float16>, dim3(grid_for((int64_t)rows * cols, 256)), dim3(256),
                       0, s, (const _Float16*)in, ld_in, rows, cols, col_scale, hi, lo, ld_out);
  }
  prof_end(s);
  return last_launch_error();
}

hipError_t split_bf16_pad(const void* in, int in_type, int64_t ld_in, int rows, int cols,
                          const float* col_scale, u16* hi, u16* lo, int64_t ld_out,
                          int rows_out, hipStream_t s) {
  if (rows_out < rows) rows_out = rows;
  if (rows_out <= 0 || ld_out <= 0) return hipSuccess;
  if (ld_out % 4 != 0 || ld_out < cols ||
      (reinterpret_cast<uintptr_t>(hi) & 7) != 0 || (lo && (reinterpret_cast<uintptr_t>(lo) & 7) != 0))
    return hipErrorInvalidValue;
  prof_begin(s, "split_bf16");
  // a few thousand work-groups, each thread walking rows_out / 512 rows
  const dim3 g((unsigned)((ld_out + 1023) / 1024), (unsigned)(rows_out < 512 ? rows_out : 512));
  if (in_type == 0)
    hipLaunchKernelGGL(k_split_pad<float>, g, dim3(256), 0, s, (const float*)in, ld_in, rows, cols,
                       col_scale, hi, lo, ld_out, rows_out);
  else if (in_type == 1)
    hipLaunchKernelGGL(k_split_pad<_Float16>, g, dim3(256), 0, s, (const _Float16*)in, ld_in, rows,
                       cols, col_scale, hi, lo, ld_out, rows_out);
  else
    hipLaunchKernelGGL(k_split_pad<u16>, g, dim3(256), 0, s, (const u16*)in, ld_in, rows, cols,
                       col_scale, hi, lo, ld_out, rows_out);
  prof_end(s);
  return last_launch_error();
}

hipError_t fill_zero_f32(float* p, int rows, int cols, int64_t ld, hipStream_t s) {
  if (rows <= 0 || cols <= 0) return hipSuccess;
  prof_begin(s, "fill_zero");
  hipLaunchKernelGGL(k_fill_zero, dim3(grid_for((int64_t)rows * cols, 256)), dim3(256), 0, s, p,
                     rows, cols, ld);
  prof_end(s);
  return last_launch_error();
}

}  // namespace fq
