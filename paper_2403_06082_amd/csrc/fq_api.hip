// C ABI of libfq: argument validation, workspace layout and the launch sequence of each
// call of the FrameQuant per-layer pass (see include/fq.h for the contract).
#include "fq_internal.h"
#include "../../include/fq.h"

#include <algorithm>
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <string>
#include <vector>
#include <mutex>

namespace fq {

// ---------------------------------------------------------------- errors
static thread_local std::string g_last_error;

static fq_status fail(fq_status st, const char* msg) {
  g_last_error = msg;
  return st;
}

static fq_status hip_fail(hipError_t e, const char* where) {
  std::string m = std::string(where) + ": " + hipGetErrorString(e);
  g_last_error = m;
  return FQ_ERR_HIP;
}

hipError_t last_launch_error() { return hipGetLastError(); }

// kernel of the fp64 update GEMMs: by default the LDS-ring kernel for the updates beyond
// a span (large: K_out x 512 x the rest) and the 64 x 64 kernel for those inside a span
// (K_out x 128 x at most 384); FQ_DGEMM_TILE=64|128 puts every update on the
// register-staged kernel with that tile, for comparison
static int dgemm_tile_from_env() {
  const char* v = getenv("FQ_DGEMM_TILE");
  const int t = v ? atoi(v) : 0;
  return (t == 64 || t == 128) ? t : 0;
}
static int g_dgemm_tile = dgemm_tile_from_env();

// ---------------------------------------------------------------- kernel timer
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};
static bool g_prof_on = false;
static std::vector<ProfRec> g_prof;
static std::vector<hipEvent_t> g_pool;
static std::mutex g_prof_mu;

static hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void prof_begin(hipStream_t s, const char* name) {
  if (!g_prof_on) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  ProfRec r{name, take_event(), take_event()};
  if (r.a) hipEventRecord(r.a, s);
  g_prof.push_back(r);
}

bool prof_enabled() { return g_prof_on; }

void prof_end(hipStream_t s) {
  if (!g_prof_on) return;
  std::lock_guard<std::mutex> lk(g_prof_mu);
  if (!g_prof.empty() && g_prof.back().b) hipEventRecord(g_prof.back().b, s);
}

// ---------------------------------------------------------------- workspace carving
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~(size_t)255;
    T* p = base ? (T*)(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

static int64_t rup8(int64_t x) { return (x + 7) / 8 * 8; }
static const int64_t DIM_MAX = (int64_t)1 << 30;

static bool dim_ok(int64_t v) { return v >= 0 && v < DIM_MAX; }

static int hessian_ksplit(int64_t n, int64_t d, int npass) {
  const int t = (int)((d + 255) / 256);
  const int ntiles = t * (t + 1) / 2;
  const int64_t ktiles = (n + 63) / 64;
  int ks = (int)((2048 + ntiles / 2) / (ntiles > 0 ? ntiles : 1));
  if (ks < 1) ks = 1;
  if (ks > ktiles) ks = (int)(ktiles > 0 ? ktiles : 1);
  (void)npass;
  return ks;
}

struct HessLayout {
  u16* xhi; u16* xlo; float* part; int ksplit; int64_t ldp;
};

static size_t hessian_layout(int xt, int64_t n, int64_t d, void* ws, HessLayout* L) {
  Carver c(ws);
  HessLayout l{};
  l.ldp = rup8(d);
  if (xt == FQ_F32) {
    l.xhi = c.take<u16>((size_t)n * l.ldp);
    l.xlo = c.take<u16>((size_t)n * l.ldp);
  }
  l.ksplit = hessian_ksplit(n, d, xt == FQ_F32 ? 3 : 1);
  l.part = c.take<float>(gemm_partial_bytes((int)d, l.ksplit) / sizeof(float));
  if (L) *L = l;
  return c.off + 256;
}

static int64_t rup32(int64_t x) { return (x + 31) / 32 * 32; }

// Analysis planes.  Every product reads both operands with the reduction index as the
// row (row-contiguous in the other index), so each operand is the caller's array as laid
// out, split into bf16 planes with rows and columns zero-padded:
//   po  = P_out [pad(d_out) x pad8(K_out)]     wn = W [pad(d_out) x pad(d_in)]
//   pi  = P_in  [pad(d_in) x pad8(K_in)]       h  = H [pad(d_in) x pad(d_in)]
//   tt  = T^T = W^T P_out [pad(d_in) x pad8(K_out)]   g = H P_in [pad(d_in) x pad8(K_in)]
// D = T P_in and H~ = P_in^T G then need no transposed copy.  bf16 weights whose shape
// needs no padding are read in place.
struct AnaLayout {
  u16 *po_hi, *po_lo, *pi_hi, *pi_lo, *wn_hi, *wn_lo, *tt_hi, *tt_lo, *h_hi, *h_lo, *g_hi, *g_lo;
  int64_t lo_, li_;   // pad(d_out), pad(d_in): multiples of 32
  int64_t ko8, ki8;   // pad8(K_out), pad8(K_in)
  float* tailp;       // K-split scratch for a short last round of tiles (or null)
};

// Products with this many output tiles or fewer fill at most one round of the compute
// units and never take the K-split tail; smaller layouts carry no scratch for it.
static constexpr int64_t kTailMinTiles = 64;

static size_t analysis_layout(int wt, int64_t d_out, int64_t d_in, int64_t K_out, int64_t K_in,
                              void* ws, AnaLayout* L) {
  Carver c(ws);
  AnaLayout l{};
  l.lo_ = rup32(d_out);
  l.li_ = rup32(d_in);
  l.ko8 = (K_out + 7) / 8 * 8;
  l.ki8 = (K_in + 7) / 8 * 8;
  l.po_hi = c.take<u16>((size_t)l.lo_ * l.ko8);
  l.po_lo = c.take<u16>((size_t)l.lo_ * l.ko8);
  l.pi_hi = c.take<u16>((size_t)l.li_ * l.ki8);
  l.pi_lo = c.take<u16>((size_t)l.li_ * l.ki8);
  l.wn_hi = c.take<u16>((size_t)l.lo_ * l.li_);
  if (wt != FQ_BF16) l.wn_lo = c.take<u16>((size_t)l.lo_ * l.li_);
  l.tt_hi = c.take<u16>((size_t)l.li_ * l.ko8);
  l.tt_lo = c.take<u16>((size_t)l.li_ * l.ko8);
  l.h_hi = c.take<u16>((size_t)l.li_ * l.li_);
  l.h_lo = c.take<u16>((size_t)l.li_ * l.li_);
  l.g_hi = c.take<u16>((size_t)l.li_ * l.ki8);
  l.g_lo = c.take<u16>((size_t)l.li_ * l.ki8);
  const int64_t tiles = std::max({gemm_tiles(l.li_, K_out),
                                  gemm_tiles(K_out, K_in),
                                  gemm_tiles(l.li_, K_in)});
  l.tailp = tiles > kTailMinTiles ? c.take<float>(gemm_tail_bytes() / sizeof(float)) : nullptr;
  if (L) *L = l;
  return c.off + 256;
}

// Columns are rounded in chunks of min(block, 128) by the sequential kernel; the
// residuals of consecutive chunks are applied to the columns right of them in spans of
// at least 512 columns (a whole number of blocks): inside a span each chunk receives
// those of the span's earlier chunks in the rounding kernel, right before it is rounded;
// the columns beyond the span receive the whole span's once, as one fp64 GEMM.  This
// regroups OPTQ's lazy block updates; every column still receives exactly the sum of the
// residual terms of all earlier columns.
static int64_t chunk_width(int block) { return block < 128 ? block : 128; }
static int64_t span_width(int block) {
  const int64_t b = block;
  return b * ((512 + b - 1) / b);
}
static int64_t res_width(int64_t K_in, int block) {
  int64_t w = span_width(block) < K_in ? span_width(block) : K_in;
  return w > 0 ? w : 1;
}

static size_t quant_layout(int64_t K_out, int64_t K_in, int block, void* ws, QuantScratch* Q) {
  Carver c(ws);
  QuantScratch q{};
  q.Y = c.take<double>((size_t)K_out * K_in);
  q.A = c.take<double>((size_t)K_in * K_in);
  q.R = c.take<double>((size_t)K_in * K_in);
  q.res = c.take<double>((size_t)K_out * res_width(K_in, block));
  q.codes8 = c.take<uint8_t>((size_t)K_out * K_in);
  q.red = c.take<double>(1024);
  q.scal = c.take<double>(8);
  q.scale64 = c.take<double>((size_t)K_out);
  q.zero64 = c.take<double>((size_t)K_out);
  q.inv_rdiag = c.take<double>((size_t)K_in);
  q.lslots = c.take<double>(2 * 64 * 64);
  q.dead = c.take<uint8_t>((size_t)K_in);
  q.flags = c.take<int>(4);
  if (Q) *Q = q;
  return c.off + 256;
}

// Synthesis planes (zero-padded):
//   q  = codes - zero           [pad(K_out) x pad(K_in)]   (natural layout, exact in bf16)
//   pl = P_out diag(scale)      [d_out x pad(K_out)]       pi = P_in [d_in x pad(K_in)]
//   nt = (pl q)^T = q^T pl^T    [pad(K_in) x pad8(d_out)]  (rows beyond K_in come out 0)
// W^ = pl q P_in^T is then nt^T P_in^T: the first product reads q with the reduction
// index as the row and pl with it as the column, the second nt and P_in likewise.
struct SynLayout {
  u16 *q, *pl_hi, *pl_lo, *pi_hi, *pi_lo, *nt_hi, *nt_lo;
  int64_t ko, ki;   // pad(K_out), pad(K_in): multiples of 32
  int64_t do8;      // pad8(d_out)
  float* tailp;     // K-split scratch for a short last round of tiles (or null)
};

static size_t synthesis_layout(int64_t K_out, int64_t K_in, int64_t d_out, int64_t d_in,
                               void* ws, SynLayout* L) {
  Carver c(ws);
  SynLayout l{};
  l.ko = rup32(K_out);
  l.ki = rup32(K_in);
  l.do8 = (d_out + 7) / 8 * 8;
  l.q = c.take<u16>((size_t)l.ko * l.ki);
  l.pl_hi = c.take<u16>((size_t)d_out * l.ko);
  l.pl_lo = c.take<u16>((size_t)d_out * l.ko);
  l.pi_hi = c.take<u16>((size_t)d_in * l.ki);
  l.pi_lo = c.take<u16>((size_t)d_in * l.ki);
  l.nt_hi = c.take<u16>((size_t)l.ki * l.do8);
  l.nt_lo = c.take<u16>((size_t)l.ki * l.do8);
  const int64_t tiles = std::max(gemm_tiles(l.ki, d_out),
                                 gemm_tiles(d_out, d_in));
  l.tailp = tiles > kTailMinTiles ? c.take<float>(gemm_tail_bytes() / sizeof(float)) : nullptr;
  if (L) *L = l;
  return c.off + 256;
}

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

__global__ void k_zero_i32(int* p, int n) {
  if ((int)threadIdx.x < n) p[threadIdx.x] = 0;
}

}  // namespace fq

using namespace fq;

// ---------------------------------------------------------------- allocation-free scratch
// The scratch area of fq_frame_apply_tff_noalloc: a device array in the library's code
// object, held by every GPU the library runs on until the process ends.  Host code never
// passes the array's name to a kernel (on the host it only stands in for the symbol); its
// device address is looked up once per device with hipGetSymbolAddress, with that device
// current, and kept here.
static __device__ __align__(256) char scratch[FQ_NOALLOC_SCRATCH_BYTES];
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[64];

static fq_status scratch_of_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= 64) return fail(FQ_ERR_UNSUPPORTED, "device index beyond 63");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(FQ_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FQ_OK;
}

// Streams made by fq_side_stream_create (their kernels share part of the device with the
// caller's other work), so that launchers can size their grids for dynamic balancing there.
static std::mutex g_side_mu;
static std::vector<hipStream_t> g_side_streams;

bool fq::is_side_stream(hipStream_t s) {
  if (!s) return false;
  std::lock_guard<std::mutex> lock(g_side_mu);
  return std::find(g_side_streams.begin(), g_side_streams.end(), s) != g_side_streams.end();
}

extern "C" {

const char* fq_status_string(int st) {
  switch (st) {
    case FQ_OK: return "FQ_OK";
    case FQ_ERR_INVALID_ARG: return "FQ_ERR_INVALID_ARG";
    case FQ_ERR_UNSUPPORTED: return "FQ_ERR_UNSUPPORTED";
    case FQ_ERR_NOT_POSITIVE_DEFINITE: return "FQ_ERR_NOT_POSITIVE_DEFINITE";
    case FQ_ERR_NONFINITE: return "FQ_ERR_NONFINITE";
    case FQ_ERR_WORKSPACE_TOO_SMALL: return "FQ_ERR_WORKSPACE_TOO_SMALL";
    case FQ_ERR_HIP: return "FQ_ERR_HIP";
  }
  return "FQ_UNKNOWN_STATUS";
}

const char* fq_last_error(void) { return g_last_error.c_str(); }

void fq_profile_enable(int on) { g_prof_on = on != 0; }

void fq_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  for (auto& r : g_prof) {
    if (r.a) { hipEventSynchronize(r.a); g_pool.push_back(r.a); }
    if (r.b) { hipEventSynchronize(r.b); g_pool.push_back(r.b); }
  }
  g_prof.clear();
}

int fq_profile_query(const char* prefix, int* count, double* total_ms) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  const size_t pl = prefix ? strlen(prefix) : 0;
  int n = 0;
  double t = 0.0;
  for (auto& r : g_prof) {
    if (pl && strncmp(r.name, prefix, pl) != 0) continue;
    if (!r.a || !r.b) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) return -1;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return -1;
    ++n;
    t += ms;
  }
  if (count) *count = n;
  if (total_ms) *total_ms = t;
  return 0;
}

// ================================================================ S1: Hessian
size_t fq_hessian_workspace_bytes(int xt, int64_t n_tokens, int64_t d_in) {
  if (!dim_ok(n_tokens) || !dim_ok(d_in) || xt < 0 || xt > 2) return 0;
  return hessian_layout(xt, n_tokens, d_in, nullptr, nullptr);
}

fq_status fq_hessian_accumulate(void* stream, const void* X, int xt, int64_t n_tokens,
                                int64_t d_in, int64_t ldx, float* H, int accumulate, void* ws,
                                size_t ws_bytes) {
  if (xt < FQ_F32 || xt > FQ_BF16) return fail(FQ_ERR_INVALID_ARG, "xt must be FQ_F32, FQ_F16 or FQ_BF16");
  if (!dim_ok(n_tokens) || !dim_ok(d_in)) return fail(FQ_ERR_INVALID_ARG, "n_tokens and d_in must be in [0, 2^30)");
  if (ldx < d_in) return fail(FQ_ERR_INVALID_ARG, "ldx must be >= d_in");
  if (d_in == 0) return FQ_OK;
  if (!H) return fail(FQ_ERR_INVALID_ARG, "H is NULL");
  if (n_tokens > 0 && !X) return fail(FQ_ERR_INVALID_ARG, "X is NULL");
  const size_t need = hessian_layout(xt, n_tokens, d_in, nullptr, nullptr);
  if (ws_bytes < need) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_hessian_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  // align the carve base to 256 bytes inside the provided workspace
  char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
  HessLayout L;
  hessian_layout(xt, n_tokens, d_in, base, &L);
  hipError_t e;
  GemmDesc g;
  g.M = (int)d_in; g.N = (int)d_in; g.K = (int)n_tokens;
  g.a_kmajor = false; g.b_kmajor = false;
  g.epi = EPI_PARTIAL;
  g.ksplit = L.ksplit;
  g.name = "gemm_hessian";
  if (xt == FQ_F32) {
    e = split_bf16(X, 0, ldx, (int)n_tokens, (int)d_in, nullptr, L.xhi, L.xlo, L.ldp, s);
    if (e != hipSuccess) return hip_fail(e, "split X");
    g.a[0] = L.xhi; g.a[1] = L.xlo; g.b[0] = L.xhi; g.b[1] = L.xlo;
    g.lda = g.ldb = L.ldp;
    g.npass = 3;
    g.pa[0] = 0; g.pb[0] = 0; g.pa[1] = 0; g.pb[1] = 1; g.pa[2] = 1; g.pb[2] = 0;
  } else {
    g.a[0] = (const u16*)X; g.b[0] = (const u16*)X;
    g.lda = g.ldb = ldx;
    g.npass = 1;
    g.f16 = (xt == FQ_F16);
  }
  e = gemm_run(g, L.part, s);
  if (e != hipSuccess) return hip_fail(e, "hessian gemm");
  e = syrk_reduce(L.part, (int)d_in, L.ksplit, H, d_in, accumulate, s);
  if (e != hipSuccess) return hip_fail(e, "hessian reduce");
  return FQ_OK;
}

// ================================================================ S2: analysis
size_t fq_frame_analysis_workspace_bytes(int wt, int64_t d_out, int64_t d_in, int64_t K_out,
                                         int64_t K_in) {
  if (wt < 0 || wt > 2 || !dim_ok(d_out) || !dim_ok(d_in) || !dim_ok(K_out) || !dim_ok(K_in)) return 0;
  return analysis_layout(wt, d_out, d_in, K_out, K_in, nullptr, nullptr);
}

fq_status fq_frame_analysis(void* stream, const void* W, int wt, int64_t d_out, int64_t d_in,
                            const float* P_out, int64_t K_out, const float* P_in, int64_t K_in,
                            const float* H, float* D, float* Ht, void* ws, size_t ws_bytes) {
  if (wt < FQ_F32 || wt > FQ_BF16) return fail(FQ_ERR_INVALID_ARG, "wt must be FQ_F32, FQ_F16 or FQ_BF16");
  if (!dim_ok(d_out) || !dim_ok(d_in) || !dim_ok(K_out) || !dim_ok(K_in))
    return fail(FQ_ERR_INVALID_ARG, "dimensions must be in [0, 2^30)");
  if (K_out < d_out || K_in < d_in)
    return fail(FQ_ERR_INVALID_ARG, "a frame needs K >= d (K_out >= d_out, K_in >= d_in)");
  if (D && (!W || !P_out || !P_in) && d_out > 0 && d_in > 0)
    return fail(FQ_ERR_INVALID_ARG, "W, P_out and P_in are required for D");
  if (Ht && (!H || !P_in) && d_in > 0) return fail(FQ_ERR_INVALID_ARG, "H and P_in are required for Ht");
  const size_t need = analysis_layout(wt, d_out, d_in, K_out, K_in, nullptr, nullptr);
  if (ws_bytes < need) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_frame_analysis_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
  AnaLayout L;
  analysis_layout(wt, d_out, d_in, K_out, K_in, base, &L);
  hipError_t e;
  auto three = [](GemmDesc& g) {
    g.npass = 3;
    g.pa[0] = 0; g.pb[0] = 0; g.pa[1] = 0; g.pb[1] = 1; g.pa[2] = 1; g.pb[2] = 0;
  };
  // C (+ or SPLIT / SYM) = A B with A(m, k) at a[k * lda + m] and B(k, n) at b[k * ldb + n]
  auto mn_gemm = [](int M, int N, int K, const u16* a0, const u16* a1, int64_t lda,
                    const u16* b0, const u16* b1, int64_t ldb) {
    GemmDesc g;
    g.M = M; g.N = N; g.K = K;
    g.a[0] = a0; g.a[1] = a1; g.lda = lda; g.a_kmajor = false;
    g.b[0] = b0; g.b[1] = b1; g.ldb = ldb; g.b_kmajor = false;
    return g;
  };
  if (d_in > 0 && K_in > 0) {
    e = split_bf16_pad(P_in, 0, K_in, (int)d_in, (int)K_in, nullptr, L.pi_hi, L.pi_lo, L.ki8,
                       (int)L.li_, s);
    if (e != hipSuccess) return hip_fail(e, "split P_in");
  }
  if (D && K_out > 0 && K_in > 0) {
    if (d_out == 0 || d_in == 0) {
      e = fill_zero_f32(D, (int)K_out, (int)K_in, K_in, s);
      if (e != hipSuccess) return hip_fail(e, "zero D");
    } else {
      e = split_bf16_pad(P_out, 0, K_out, (int)d_out, (int)K_out, nullptr, L.po_hi, L.po_lo, L.ko8,
                         (int)L.lo_, s);
      if (e != hipSuccess) return hip_fail(e, "split P_out");
      // W: bf16 weights are exact in one plane and are read in place when no padding is
      // needed; otherwise a zero-padded copy (f16 / f32 weights take a bf16 pair)
      const int in_t = wt == FQ_BF16 ? 2 : (wt == FQ_F16 ? 1 : 0);
      const u16* wb0 = L.wn_hi;
      const u16* wb1 = L.wn_lo;
      int64_t ldw = L.li_;
      if (wt == FQ_BF16 && d_out == L.lo_ && d_in == L.li_ && aligned16(W)) {
        wb0 = (const u16*)W;
        ldw = d_in;
      } else {
        e = split_bf16_pad(W, in_t, d_in, (int)d_out, (int)d_in, nullptr, L.wn_hi,
                           wt == FQ_BF16 ? nullptr : L.wn_lo, L.li_, (int)L.lo_, s);
        if (e != hipSuccess) return hip_fail(e, "split W");
      }
      // T^T = W^T P_out  (pad(d_in) x K_out; rows beyond d_in come out zero), bf16 pair
      GemmDesc g = mn_gemm((int)L.li_, (int)K_out, (int)L.lo_, wb0, wb1, ldw, L.po_hi, L.po_lo,
                           L.ko8);
      if (wt != FQ_BF16) {
        three(g);
      } else {
        g.npass = 2;
        g.pa[0] = 0; g.pb[0] = 0; g.pa[1] = 0; g.pb[1] = 1;
      }
      g.epi = EPI_SPLIT; g.c_hi = L.tt_hi; g.c_lo = L.tt_lo; g.ldc = L.ko8; g.ldc_pad = L.ko8;
      g.name = "gemm_analysis_w1";
      e = gemm_run(g, L.tailp, s);
      if (e != hipSuccess) return hip_fail(e, "analysis gemm 1");
      // D = T P_in  (K_out x K_in)
      GemmDesc g2 = mn_gemm((int)K_out, (int)K_in, (int)L.li_, L.tt_hi, L.tt_lo, L.ko8, L.pi_hi,
                            L.pi_lo, L.ki8);
      three(g2);
      g2.epi = EPI_F32; g2.c = D; g2.ldc = K_in;
      g2.name = "gemm_analysis_w2";
      e = gemm_run(g2, L.tailp, s);
      if (e != hipSuccess) return hip_fail(e, "analysis gemm 2");
    }
  }
  if (Ht && K_in > 0) {
    if (d_in == 0) {
      e = fill_zero_f32(Ht, (int)K_in, (int)K_in, K_in, s);
      if (e != hipSuccess) return hip_fail(e, "zero Ht");
    } else {
      e = split_bf16_pad(H, 0, d_in, (int)d_in, (int)d_in, nullptr, L.h_hi, L.h_lo, L.li_,
                         (int)L.li_, s);
      if (e != hipSuccess) return hip_fail(e, "split H");
      // G = H P_in  (pad(d_in) x K_in; H is symmetric, rows beyond d_in come out zero)
      GemmDesc g = mn_gemm((int)L.li_, (int)K_in, (int)L.li_, L.h_hi, L.h_lo, L.li_, L.pi_hi,
                           L.pi_lo, L.ki8);
      three(g);
      g.epi = EPI_SPLIT; g.c_hi = L.g_hi; g.c_lo = L.g_lo; g.ldc = L.ki8; g.ldc_pad = L.ki8;
      g.name = "gemm_analysis_h1";
      e = gemm_run(g, L.tailp, s);
      if (e != hipSuccess) return hip_fail(e, "analysis gemm 3");
      // Ht = P_in^T G  (K_in x K_in, upper tiles mirrored)
      GemmDesc g2 = mn_gemm((int)K_in, (int)K_in, (int)L.li_, L.pi_hi, L.pi_lo, L.ki8, L.g_hi,
                            L.g_lo, L.ki8);
      three(g2);
      g2.epi = EPI_SYM; g2.c = Ht; g2.ldc = K_in;
      g2.name = "gemm_analysis_h2";
      e = gemm_run(g2, nullptr, s);
      if (e != hipSuccess) return hip_fail(e, "analysis gemm 4");
    }
  }
  return FQ_OK;
}

// ================================================================ S3: quantize
size_t fq_quantize_frames_workspace_bytes(int64_t K_out, int64_t K_in, int block) {
  if (!dim_ok(K_out) || !dim_ok(K_in) || block < 1) return 0;
  return quant_layout(K_out, K_in, block, nullptr, nullptr);
}

// the H~ phase: dead columns, damping, the reversed Cholesky factor R (no sync).  It
// touches only its own parts of the workspace (A, R, its diagonal, the dead mask,
// lambda, flags[0..1]), so the D phase's first part may run beside it on another stream.
static fq_status quantize_prepare(hipStream_t s, const float* Ht, int64_t K_in, double damp,
                                  QuantScratch& Q) {
  hipError_t e;
  prof_begin(s, "q_init");
  hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(64), 0, s, Q.flags, 2);
  prof_end(s);
  if ((e = q_hdiag_build(Ht, K_in, damp, Q, s)) != hipSuccess) return hip_fail(e, "hessian prep");
  if ((e = q_cholesky(Q.A, K_in, Q.lslots, Q.flags, s)) != hipSuccess) return hip_fail(e, "cholesky");
  if ((e = q_reverse_upper(Q.A, K_in, Q.R, Q.inv_rdiag, s)) != hipSuccess) return hip_fail(e, "reverse");
  return FQ_OK;
}

// the D phase, first part: moments, clip, per-row grid, and the working matrix Y = the
// clipped D (no sync).  Its own parts of the workspace: Y, the moment partials,
// scal[0..3], scale64, zero64, flags[2]; it reads nothing the H~ phase writes.
static fq_status quantize_grid(hipStream_t s, const float* D, int64_t K_out, int64_t K_in,
                               int bits, double clip_sigmas, float* scale, float* zero,
                               QuantScratch& Q) {
  hipError_t e;
  // this call's own D check (the H~ checks of the prepare phase stay in flags[0..1])
  prof_begin(s, "q_init");
  hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(64), 0, s, Q.flags + 2, 1);
  prof_end(s);
  if ((e = q_stats(D, K_out, K_in, clip_sigmas, Q, s)) != hipSuccess) return hip_fail(e, "stats");
  if ((e = q_clip_grid(D, K_out, K_in, bits, Q, scale, zero, s)) != hipSuccess) return hip_fail(e, "clip/grid");
  return FQ_OK;
}

// the D phase, second part (after both the H~ phase and the first part): rounding with
// error feedback and packing (no sync)
static fq_status quantize_round_launch(hipStream_t s, const float* D, int64_t K_out,
                                       int64_t K_in, int bits, int block, uint32_t* codes,
                                       QuantScratch& Q) {
  hipError_t e;
  const int64_t ldr = res_width(K_in, block);
  const int64_t cw = chunk_width(block), sw = span_width(block);
  for (int64_t s1 = 0; s1 < K_in; s1 += sw) {
    const int64_t s2 = (s1 + sw < K_in) ? s1 + sw : K_in;
    for (int64_t i1 = s1; i1 < s2; i1 += cw) {
      const int64_t i2 = (i1 + cw < s2) ? i1 + cw : s2;
      // the rounding kernel first adds the residuals of the span's earlier chunks to
      // this chunk's columns (the in-span update), then rounds them
      if ((e = q_gptq_block(D, K_out, K_in, (int)i1, (int)i2, (int)s1, (int)cw, ldr, bits, Q,
                            s)) != hipSuccess)
        return hip_fail(e, "rounding block");
    }
    if (s2 < K_in) {
      e = dgemm(K_out, K_in - s2, s2 - s1, 1.0, 1.0, Q.res, ldr, Q.R + s1 * K_in + s2, K_in, false,
                Q.Y + s2, K_in, false, s, "gptq_update_lazy", g_dgemm_tile);
      if (e != hipSuccess) return hip_fail(e, "lazy update");
    }
  }
  if ((e = bits == 2 ? q_pack2(Q.codes8, K_out, K_in, codes, s)
                    : q_pack_nbit(Q.codes8, K_out, K_in, bits, codes, s)) != hipSuccess)
    return hip_fail(e, "pack");
  return FQ_OK;
}

// the checks of all three phases, recorded in the workspace: sync, then report
static fq_status quantize_check(hipStream_t s, QuantScratch& Q) {
  hipError_t e;
  int flags[4] = {0, 0, 0, 0};
  if ((e = hipMemcpyAsync(flags, Q.flags, sizeof(flags), hipMemcpyDeviceToHost, s)) != hipSuccess)
    return hip_fail(e, "flag copy");
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return hip_fail(e, "stream sync");
  if (flags[2]) return fail(FQ_ERR_NONFINITE, "D holds NaN or Inf");
  if (flags[1]) return fail(FQ_ERR_NONFINITE, "Ht holds NaN or Inf");
  if (flags[0]) return fail(FQ_ERR_NOT_POSITIVE_DEFINITE, "damped Ht is not positive definite");
  return FQ_OK;
}

static fq_status quantize_round(hipStream_t s, const float* D, int64_t K_out, int64_t K_in,
                                int bits, int block, uint32_t* codes, QuantScratch& Q) {
  const fq_status st = quantize_round_launch(s, D, K_out, K_in, bits, block, codes, Q);
  return st != FQ_OK ? st : quantize_check(s, Q);
}

static fq_status quantize_ws_check(int64_t K_out, int64_t K_in, int block, void* ws,
                                   size_t ws_bytes) {
  const size_t need = quant_layout(K_out, K_in, block, nullptr, nullptr);
  if (ws_bytes < need) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_quantize_frames_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  return FQ_OK;
}

static QuantScratch quantize_scratch(int64_t K_out, int64_t K_in, int block, void* ws) {
  char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
  QuantScratch Q;
  quant_layout(K_out, K_in, block, base, &Q);
  return Q;
}

fq_status fq_quantize_frames(void* stream, const float* D, const float* Ht, int64_t K_out,
                             int64_t K_in, int bits, int block, double damp, double clip_sigmas,
                             uint32_t* codes, float* scale, float* zero, void* ws,
                             size_t ws_bytes) {
  if (!dim_ok(K_out) || !dim_ok(K_in)) return fail(FQ_ERR_INVALID_ARG, "K_out and K_in must be in [0, 2^30)");
  if (bits < 2 || bits > 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2, 3 or 4");
  if (block < 1) return fail(FQ_ERR_INVALID_ARG, "block must be >= 1");
  if (!(damp >= 0.0) || !isfinite(damp)) return fail(FQ_ERR_INVALID_ARG, "damp must be finite and >= 0");
  if (!(clip_sigmas > 0.0)) return fail(FQ_ERR_INVALID_ARG, "clip_sigmas must be > 0 (+inf disables the clip)");
  if (K_out == 0 || K_in == 0) return FQ_OK;
  if (!D || !Ht || !codes || !scale || !zero) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  fq_status st = quantize_ws_check(K_out, K_in, block, ws, ws_bytes);
  if (st != FQ_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  QuantScratch Q = quantize_scratch(K_out, K_in, block, ws);
  if ((st = quantize_prepare(s, Ht, K_in, damp, Q)) != FQ_OK) return st;
  if ((st = quantize_grid(s, D, K_out, K_in, bits, clip_sigmas, scale, zero, Q)) != FQ_OK)
    return st;
  return quantize_round(s, D, K_out, K_in, bits, block, codes, Q);
}

fq_status fq_quantize_prepare(void* stream, const float* Ht, int64_t K_out, int64_t K_in,
                              int block, double damp, void* ws, size_t ws_bytes) {
  if (!dim_ok(K_out) || !dim_ok(K_in)) return fail(FQ_ERR_INVALID_ARG, "K_out and K_in must be in [0, 2^30)");
  if (block < 1) return fail(FQ_ERR_INVALID_ARG, "block must be >= 1");
  if (!(damp >= 0.0) || !isfinite(damp)) return fail(FQ_ERR_INVALID_ARG, "damp must be finite and >= 0");
  if (K_out == 0 || K_in == 0) return FQ_OK;
  if (!Ht) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  fq_status st = quantize_ws_check(K_out, K_in, block, ws, ws_bytes);
  if (st != FQ_OK) return st;
  QuantScratch Q = quantize_scratch(K_out, K_in, block, ws);
  return quantize_prepare((hipStream_t)stream, Ht, K_in, damp, Q);
}

fq_status fq_quantize_apply(void* stream, const float* D, int64_t K_out, int64_t K_in, int bits,
                            int block, double clip_sigmas, uint32_t* codes, float* scale,
                            float* zero, void* ws, size_t ws_bytes) {
  if (!dim_ok(K_out) || !dim_ok(K_in)) return fail(FQ_ERR_INVALID_ARG, "K_out and K_in must be in [0, 2^30)");
  if (bits < 2 || bits > 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2, 3 or 4");
  if (block < 1) return fail(FQ_ERR_INVALID_ARG, "block must be >= 1");
  if (!(clip_sigmas > 0.0)) return fail(FQ_ERR_INVALID_ARG, "clip_sigmas must be > 0 (+inf disables the clip)");
  if (K_out == 0 || K_in == 0) return FQ_OK;
  if (!D || !codes || !scale || !zero) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  fq_status st = quantize_ws_check(K_out, K_in, block, ws, ws_bytes);
  if (st != FQ_OK) return st;
  QuantScratch Q = quantize_scratch(K_out, K_in, block, ws);
  if ((st = quantize_grid((hipStream_t)stream, D, K_out, K_in, bits, clip_sigmas, scale, zero,
                          Q)) != FQ_OK)
    return st;
  return quantize_round((hipStream_t)stream, D, K_out, K_in, bits, block, codes, Q);
}

fq_status fq_quantize_grid(void* stream, const float* D, int64_t K_out, int64_t K_in, int bits,
                           int block, double clip_sigmas, float* scale, float* zero, void* ws,
                           size_t ws_bytes) {
  if (!dim_ok(K_out) || !dim_ok(K_in)) return fail(FQ_ERR_INVALID_ARG, "K_out and K_in must be in [0, 2^30)");
  if (bits < 2 || bits > 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2, 3 or 4");
  if (block < 1) return fail(FQ_ERR_INVALID_ARG, "block must be >= 1");
  if (!(clip_sigmas > 0.0)) return fail(FQ_ERR_INVALID_ARG, "clip_sigmas must be > 0 (+inf disables the clip)");
  if (K_out == 0 || K_in == 0) return FQ_OK;
  if (!D || !scale || !zero) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  fq_status st = quantize_ws_check(K_out, K_in, block, ws, ws_bytes);
  if (st != FQ_OK) return st;
  QuantScratch Q = quantize_scratch(K_out, K_in, block, ws);
  return quantize_grid((hipStream_t)stream, D, K_out, K_in, bits, clip_sigmas, scale, zero, Q);
}

fq_status fq_quantize_round(void* stream, const float* D, int64_t K_out, int64_t K_in, int bits,
                            int block, uint32_t* codes, void* ws, size_t ws_bytes) {
  if (!dim_ok(K_out) || !dim_ok(K_in)) return fail(FQ_ERR_INVALID_ARG, "K_out and K_in must be in [0, 2^30)");
  if (bits < 2 || bits > 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2, 3 or 4");
  if (block < 1) return fail(FQ_ERR_INVALID_ARG, "block must be >= 1");
  if (K_out == 0 || K_in == 0) return FQ_OK;
  if (!D || !codes) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  fq_status st = quantize_ws_check(K_out, K_in, block, ws, ws_bytes);
  if (st != FQ_OK) return st;
  QuantScratch Q = quantize_scratch(K_out, K_in, block, ws);
  return quantize_round((hipStream_t)stream, D, K_out, K_in, bits, block, codes, Q);
}

fq_status fq_quantize_round_async(void* stream, const float* D, int64_t K_out, int64_t K_in,
                                  int bits, int block, uint32_t* codes, void* ws,
                                  size_t ws_bytes) {
  if (!dim_ok(K_out) || !dim_ok(K_in)) return fail(FQ_ERR_INVALID_ARG, "K_out and K_in must be in [0, 2^30)");
  if (bits < 2 || bits > 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2, 3 or 4");
  if (block < 1) return fail(FQ_ERR_INVALID_ARG, "block must be >= 1");
  if (K_out == 0 || K_in == 0) return FQ_OK;
  if (!D || !codes) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  fq_status st = quantize_ws_check(K_out, K_in, block, ws, ws_bytes);
  if (st != FQ_OK) return st;
  QuantScratch Q = quantize_scratch(K_out, K_in, block, ws);
  return quantize_round_launch((hipStream_t)stream, D, K_out, K_in, bits, block, codes, Q);
}

fq_status fq_quantize_status(void* stream, int64_t K_out, int64_t K_in, int block, void* ws,
                             size_t ws_bytes) {
  if (!dim_ok(K_out) || !dim_ok(K_in)) return fail(FQ_ERR_INVALID_ARG, "K_out and K_in must be in [0, 2^30)");
  if (block < 1) return fail(FQ_ERR_INVALID_ARG, "block must be >= 1");
  if (K_out == 0 || K_in == 0) return FQ_OK;
  fq_status st = quantize_ws_check(K_out, K_in, block, ws, ws_bytes);
  if (st != FQ_OK) return st;
  QuantScratch Q = quantize_scratch(K_out, K_in, block, ws);
  return quantize_check((hipStream_t)stream, Q);
}

// A stream kept off the first reserve_cus compute units (bit c of the mask = unit c).
fq_status fq_side_stream_create(int reserve_cus, void** stream) {
  if (!stream) return fail(FQ_ERR_INVALID_ARG, "stream is NULL");
  *stream = nullptr;
  int dev = 0, n_cu = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "compute-unit count");
  if (reserve_cus < 0 || reserve_cus > 3 * n_cu / 4)
    return fail(FQ_ERR_INVALID_ARG, "reserve_cus must be in [0, 3/4 of the compute units]");
  hipStream_t s = nullptr;
  if (reserve_cus == 0) {
    e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
  } else {
    std::vector<uint32_t> mask((size_t)(n_cu + 31) / 32, 0u);
    for (int c = reserve_cus; c < n_cu; ++c) mask[(size_t)c / 32] |= 1u << (c % 32);
    e = hipExtStreamCreateWithCUMask(&s, (uint32_t)mask.size(), mask.data());
  }
  if (e != hipSuccess) return hip_fail(e, "stream creation");
  {
    std::lock_guard<std::mutex> lock(g_side_mu);
    g_side_streams.push_back(s);
  }
  *stream = s;
  return FQ_OK;
}

fq_status fq_side_stream_destroy(void* stream) {
  if (!stream) return fail(FQ_ERR_INVALID_ARG, "stream is NULL");
  {
    std::lock_guard<std::mutex> lock(g_side_mu);
    auto it = std::find(g_side_streams.begin(), g_side_streams.end(), (hipStream_t)stream);
    if (it != g_side_streams.end()) g_side_streams.erase(it);
  }
  const hipError_t e = hipStreamDestroy((hipStream_t)stream);
  return e == hipSuccess ? FQ_OK : hip_fail(e, "stream destruction");
}

// ================================================================ S4: synthesis
size_t fq_frame_apply_workspace_bytes(int64_t d_in, int64_t K_out, int64_t K_in) {
  if (!dim_ok(d_in) || !dim_ok(K_out) || !dim_ok(K_in)) return 0;
  return apply_scratch_floats(d_in, K_out, K_in, nullptr, nullptr) * sizeof(float) + 256;
}

fq_status fq_frame_apply(void* stream, const void* X, int xt, int64_t n_tokens, int64_t ldx,
                         int64_t d_in, const uint32_t* codes, const float* scale,
                         const float* zero, int64_t K_out, int64_t K_in, const float* P_out,
                         int64_t d_out, const float* P_in, float* Y, void* ws,
                         size_t ws_bytes) {
  return fq_frame_apply_nbit(stream, X, xt, n_tokens, ldx, d_in, codes, 2, scale, zero, K_out,
                             K_in, P_out, d_out, P_in, Y, ws, ws_bytes);
}

fq_status fq_frame_apply_nbit(void* stream, const void* X, int xt, int64_t n_tokens, int64_t ldx,
                              int64_t d_in, const uint32_t* codes, int bits, const float* scale,
                              const float* zero, int64_t K_out, int64_t K_in, const float* P_out,
                              int64_t d_out, const float* P_in, float* Y, void* ws,
                              size_t ws_bytes) {
  if (bits != 2 && bits != 4) return fail(FQ_ERR_UNSUPPORTED, "the float inference kernels take 2- or 4-bit codes");
  if (xt < FQ_F32 || xt > FQ_BF16) return fail(FQ_ERR_INVALID_ARG, "xt must be FQ_F32, FQ_F16 or FQ_BF16");
  if (!dim_ok(n_tokens) || !dim_ok(d_in) || !dim_ok(K_out) || !dim_ok(K_in) || !dim_ok(d_out))
    return fail(FQ_ERR_INVALID_ARG, "dimensions must be in [0, 2^30)");
  if (K_out < d_out || K_in < d_in)
    return fail(FQ_ERR_INVALID_ARG, "a frame needs K >= d (K_out >= d_out, K_in >= d_in)");
  if (ldx < d_in) return fail(FQ_ERR_INVALID_ARG, "ldx must be >= d_in");
  if (n_tokens == 0 || d_out == 0) return FQ_OK;
  if (!Y) return fail(FQ_ERR_INVALID_ARG, "NULL Y");
  hipStream_t s = (hipStream_t)stream;
  hipError_t e;
  if (d_in == 0 || K_out == 0 || K_in == 0) {
    e = fill_zero_f32(Y, (int)n_tokens, (int)d_out, d_out, s);
    return e == hipSuccess ? FQ_OK : hip_fail(e, "zero Y");
  }
  if (!X || !codes || !scale || !zero || !P_out || !P_in) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  const size_t need = fq_frame_apply_workspace_bytes(d_in, K_out, K_in);
  if (ws_bytes < need) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_frame_apply_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  float* base = (float*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
  ApplyScratch w;
  apply_scratch_floats(d_in, K_out, K_in, &w, base);
  if ((e = frame_apply(X, xt, n_tokens, ldx, d_in, codes, bits, scale, zero, K_out, K_in, P_out,
                       d_out, P_in, Y, w, s)) != hipSuccess)
    return hip_fail(e, "frame apply");
  return FQ_OK;
}

size_t fq_frame_synthesis_workspace_bytes(int64_t K_out, int64_t K_in, int64_t d_out,
                                          int64_t d_in) {
  if (!dim_ok(K_out) || !dim_ok(K_in) || !dim_ok(d_out) || !dim_ok(d_in)) return 0;
  return synthesis_layout(K_out, K_in, d_out, d_in, nullptr, nullptr);
}

fq_status fq_frame_synthesis(void* stream, const uint32_t* codes, const float* scale,
                             const float* zero, int64_t K_out, int64_t K_in, const float* P_out,
                             int64_t d_out, const float* P_in, int64_t d_in, float* W_hat,
                             void* ws, size_t ws_bytes) {
  return fq_frame_synthesis_nbit(stream, codes, 2, scale, zero, K_out, K_in, P_out, d_out, P_in,
                                 d_in, W_hat, ws, ws_bytes);
}

fq_status fq_frame_synthesis_nbit(void* stream, const uint32_t* codes, int bits,
                                  const float* scale, const float* zero, int64_t K_out,
                                  int64_t K_in, const float* P_out, int64_t d_out,
                                  const float* P_in, int64_t d_in, float* W_hat, void* ws,
                                  size_t ws_bytes) {
  if (bits < 2 || bits > 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2, 3 or 4");
  if (!dim_ok(K_out) || !dim_ok(K_in) || !dim_ok(d_out) || !dim_ok(d_in))
    return fail(FQ_ERR_INVALID_ARG, "dimensions must be in [0, 2^30)");
  if (K_out < d_out || K_in < d_in)
    return fail(FQ_ERR_INVALID_ARG, "a frame needs K >= d (K_out >= d_out, K_in >= d_in)");
  if (d_out == 0 || d_in == 0) return FQ_OK;
  if (!W_hat || !P_out || !P_in) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  if (K_out > 0 && K_in > 0 && (!codes || !scale || !zero)) return fail(FQ_ERR_INVALID_ARG, "NULL codes/scale/zero");
  const size_t need = synthesis_layout(K_out, K_in, d_out, d_in, nullptr, nullptr);
  if (ws_bytes < need) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_frame_synthesis_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  hipError_t e;
  if (K_out == 0 || K_in == 0) {
    e = fill_zero_f32(W_hat, (int)d_out, (int)d_in, d_in, s);
    return e == hipSuccess ? FQ_OK : hip_fail(e, "zero W_hat");
  }
  char* base = (char*)(((uintptr_t)ws + 255) & ~(uintptr_t)255);
  SynLayout L;
  synthesis_layout(K_out, K_in, d_out, d_in, base, &L);
  if ((e = dequant_nbit_bf16(codes, bits, zero, K_out, K_in, L.q, L.ki, L.ko, s)) != hipSuccess)
    return hip_fail(e, "dequant");
  if ((e = split_bf16_pad(P_out, 0, K_out, (int)d_out, (int)K_out, scale, L.pl_hi, L.pl_lo, L.ko, (int)d_out, s)) != hipSuccess)
    return hip_fail(e, "split P_out");
  if ((e = split_bf16_pad(P_in, 0, K_in, (int)d_in, (int)K_in, nullptr, L.pi_hi, L.pi_lo, L.ki, (int)d_in, s)) != hipSuccess)
    return hip_fail(e, "split P_in");
  // N^T = q^T (P_out diag(scale))^T   (pad(K_in) x d_out), bf16 pair
  GemmDesc g;
  g.M = (int)L.ki; g.N = (int)d_out; g.K = (int)L.ko;
  g.a[0] = L.q; g.lda = L.ki; g.a_kmajor = false;
  g.b[0] = L.pl_hi; g.b[1] = L.pl_lo; g.ldb = L.ko; g.b_kmajor = true;
  g.npass = 2;
  g.pa[0] = 0; g.pb[0] = 0; g.pa[1] = 0; g.pb[1] = 1;
  g.epi = EPI_SPLIT; g.c_hi = L.nt_hi; g.c_lo = L.nt_lo; g.ldc = L.do8; g.ldc_pad = L.do8;
  g.name = "gemm_synthesis_1";
  if ((e = gemm_run(g, L.tailp, s)) != hipSuccess) return hip_fail(e, "synthesis gemm 1");
  // W_hat = N P_in^T  (d_out x d_in)
  GemmDesc g2;
  g2.M = (int)d_out; g2.N = (int)d_in; g2.K = (int)L.ki;
  g2.a[0] = L.nt_hi; g2.a[1] = L.nt_lo; g2.lda = L.do8; g2.a_kmajor = false;
  g2.b[0] = L.pi_hi; g2.b[1] = L.pi_lo; g2.ldb = L.ki; g2.b_kmajor = true;
  g2.npass = 3;
  g2.pa[0] = 0; g2.pb[0] = 0; g2.pa[1] = 0; g2.pb[1] = 1; g2.pa[2] = 1; g2.pb[2] = 0;
  g2.epi = EPI_F32; g2.c = W_hat; g2.ldc = d_in;
  g2.name = "gemm_synthesis_2";
  if ((e = gemm_run(g2, L.tailp, s)) != hipSuccess) return hip_fail(e, "synthesis gemm 2");
  return FQ_OK;
}

// ================================================================ diagonal Wiener filter
// Planes: q = codes - zero [pad(K_out) x pad(K_in)] (exact bf16, rows read as the
// reduction index's rows of A), h = H~ bf16 pair [pad(K_in) x pad8(K_in)], E = q H~ fp32
// [K_out x K_in].
struct WienerLayout {
  u16 *q, *h_hi, *h_lo;
  float* E;
  int64_t ko, ki, ki8;
  float* tailp;
};

static size_t wiener_layout(int64_t K_out, int64_t K_in, void* ws, WienerLayout* L) {
  Carver c(ws);
  WienerLayout l{};
  l.ko = rup32(K_out);
  l.ki = rup32(K_in);
  l.ki8 = (K_in + 7) / 8 * 8;
  l.q = c.take<u16>((size_t)l.ko * l.ki);
  l.h_hi = c.take<u16>((size_t)l.ki * l.ki8);
  l.h_lo = c.take<u16>((size_t)l.ki * l.ki8);
  l.E = c.take<float>((size_t)K_out * K_in);
  l.tailp = gemm_tiles(K_out, K_in) > kTailMinTiles ? c.take<float>(gemm_tail_bytes() / sizeof(float))
                                                    : nullptr;
  if (L) *L = l;
  return c.off + 256;
}

size_t fq_wiener_gains_workspace_bytes(int64_t K_out, int64_t K_in) {
  if (!dim_ok(K_out) || !dim_ok(K_in)) return 0;
  return wiener_layout(K_out, K_in, nullptr, nullptr);
}

fq_status fq_wiener_gains(void* stream, const float* D, const float* Ht, const uint32_t* codes,
                          int bits, const float* scale, const float* zero, int64_t K_out,
                          int64_t K_in, float* gain, float* scale_out, void* ws, size_t ws_bytes) {
  if (bits < 2 || bits > 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2, 3 or 4");
  if (!dim_ok(K_out) || !dim_ok(K_in)) return fail(FQ_ERR_INVALID_ARG, "K_out and K_in must be in [0, 2^30)");
  if (K_out == 0) return FQ_OK;
  if (!gain || !scale) return fail(FQ_ERR_INVALID_ARG, "NULL gain or scale");
  if (K_in > 0 && (!D || !Ht || !codes || !zero)) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  const size_t need = wiener_layout(K_out, K_in, nullptr, nullptr);
  if (ws_bytes < need) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_wiener_gains_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  WienerLayout L;
  wiener_layout(K_out, K_in, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &L);
  hipError_t e;
  if (K_in > 0) {
    if ((e = dequant_nbit_bf16(codes, bits, zero, K_out, K_in, L.q, L.ki, L.ko, s)) != hipSuccess)
      return hip_fail(e, "dequant");
    if ((e = split_bf16_pad(Ht, 0, K_in, (int)K_in, (int)K_in, nullptr, L.h_hi, L.h_lo, L.ki8,
                            (int)L.ki, s)) != hipSuccess)
      return hip_fail(e, "split Ht");
    // E = q H~  (K_out x K_in): A(m, k) = q[m ki + k], B(k, n) = h[k ki8 + n]; q is exact,
    // so the two passes q h_hi + q h_lo carry H~ to its bf16-pair precision
    GemmDesc g;
    g.M = (int)K_out; g.N = (int)K_in; g.K = (int)L.ki;
    g.a[0] = L.q; g.lda = L.ki; g.a_kmajor = true;
    g.b[0] = L.h_hi; g.b[1] = L.h_lo; g.ldb = L.ki8; g.b_kmajor = false;
    g.npass = 2;
    g.pa[0] = 0; g.pb[0] = 0; g.pa[1] = 0; g.pb[1] = 1;
    g.epi = EPI_F32; g.c = L.E; g.ldc = K_in;
    g.name = "gemm_wiener";
    if ((e = gemm_run(g, L.tailp, s)) != hipSuccess) return hip_fail(e, "wiener gemm");
  }
  if ((e = wiener_rows(D, L.E, L.q, L.ki, K_out, K_in, scale, gain, scale_out, s)) != hipSuccess)
    return hip_fail(e, "wiener rows");
  return FQ_OK;
}

// ================================================================ structured frames
static bool tff_dims_ok(const fq_tff* f) {
  return f && f->d > 0 && f->k > 0 && f->rho > 0 && dim_ok(f->d) && dim_ok(f->k) &&
         dim_ok(f->rho) && f->d % 2 == 0 && f->rho % 2 == 0 && f->d % f->rho == 0 &&
         f->d / f->rho <= f->k && f->k <= TFF_MAX_K && f->rho <= 131070 &&
         f->k * f->rho < DIM_MAX && f->d1 > 0 && f->d2 > 0 && f->d1 * f->d2 == f->d &&
         f->d2 <= TFF_MAX_D2;
}

static fq_status tff_check(const fq_tff* f, const char* which, TffDev* out) {
  char msg[160];
  auto bad = [&](fq_status st, const char* why) {
    snprintf(msg, sizeof msg, "%s: %s", which, why);
    return fail(st, msg);
  };
  if (!f) return bad(FQ_ERR_INVALID_ARG, "NULL frame");
  if (f->d <= 0 || f->k <= 0 || f->rho <= 0 || !dim_ok(f->d) || !dim_ok(f->k) || !dim_ok(f->rho))
    return bad(FQ_ERR_INVALID_ARG, "d, k and rho must be in [1, 2^30)");
  if (f->d % 2 || f->rho % 2) return bad(FQ_ERR_INVALID_ARG, "d and rho must be even (a realified complex frame)");
  if (f->d1 <= 0 || f->d2 <= 0 || f->d1 * f->d2 != f->d) return bad(FQ_ERR_INVALID_ARG, "d1 * d2 must equal d");
  if (!f->R1 || !f->R2) return bad(FQ_ERR_INVALID_ARG, "NULL rotation factor");
  if (f->d % f->rho) return bad(FQ_ERR_UNSUPPORTED, "d must be divisible by rho");
  if (f->d / f->rho > f->k) return bad(FQ_ERR_INVALID_ARG, "d / rho must not exceed k (the modulation is not tight otherwise)");
  if (f->k > TFF_MAX_K || f->rho > 131070) return bad(FQ_ERR_UNSUPPORTED, "k above 3968 or rho above 131070");
  if (f->d2 > TFF_MAX_D2) return bad(FQ_ERR_UNSUPPORTED, "d2 above 4096");
  if (f->k * f->rho >= DIM_MAX) return bad(FQ_ERR_INVALID_ARG, "k * rho must be below 2^30");
  out->d = f->d; out->k = f->k; out->rho = f->rho; out->m = f->d / f->rho;
  out->R1 = f->R1; out->d1 = (int)f->d1; out->R2 = f->R2; out->d2 = (int)f->d2;
  return FQ_OK;
}

struct TffLayout { float* a; float* r2t; };

static size_t tff_layout(int64_t n, const fq_tff* f, void* base, TffLayout* L) {
  const int64_t chunk = std::max<int64_t>(1, std::min<int64_t>(n, TFF_CHUNK));
  Carver c(base);
  TffLayout l{};
  l.a = c.take<float>((size_t)(chunk * f->d));
  l.r2t = c.take<float>((size_t)(f->d2 * f->d2));
  if (L) *L = l;
  return c.off + 256;
}

struct ApplyTffLayout { float* y; float* U; float* V; float* z; float* r2t; };

static size_t apply_tff_layout(const fq_tff* fo, const fq_tff* fi, void* base, ApplyTffLayout* L) {
  const int64_t K_in = fi->k * fi->rho, K_out = fo->k * fo->rho;
  Carver c(base);
  ApplyTffLayout l{};
  l.y = c.take<float>((size_t)(APPLY_NT * fi->d));
  l.U = c.take<float>((size_t)(APPLY_NT * ((K_in + 15) / 16 * 16)));
  l.V = c.take<float>((size_t)(APPLY_NT * K_out));
  l.z = c.take<float>((size_t)(APPLY_NT * fo->d));
  l.r2t = c.take<float>((size_t)(fo->d2 * fo->d2));
  if (L) *L = l;
  return c.off + 256;
}

size_t fq_tff_analysis_workspace_bytes(int64_t n, const fq_tff* frame) {
  if (!dim_ok(n) || !tff_dims_ok(frame)) return 0;
  return tff_layout(n, frame, nullptr, nullptr);
}

size_t fq_tff_synthesis_workspace_bytes(int64_t n, const fq_tff* frame) {
  return fq_tff_analysis_workspace_bytes(n, frame);
}

size_t fq_frame_apply_tff_workspace_bytes(const fq_tff* frame_out, const fq_tff* frame_in) {
  if (!tff_dims_ok(frame_out) || !tff_dims_ok(frame_in)) return 0;
  return apply_tff_layout(frame_out, frame_in, nullptr, nullptr);
}

fq_status fq_tff_analysis(void* stream, const void* X, int xt, int64_t n, int64_t ldx,
                          const fq_tff* frame, float* U, void* ws, size_t ws_bytes) {
  if (xt < FQ_F32 || xt > FQ_BF16) return fail(FQ_ERR_INVALID_ARG, "xt must be FQ_F32, FQ_F16 or FQ_BF16");
  if (!dim_ok(n)) return fail(FQ_ERR_INVALID_ARG, "n must be in [0, 2^30)");
  TffDev F;
  fq_status st = tff_check(frame, "frame", &F);
  if (st != FQ_OK) return st;
  if (ldx < F.d) return fail(FQ_ERR_INVALID_ARG, "ldx must be >= d");
  if (n == 0) return FQ_OK;
  if (!X || !U) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  if (ws_bytes < tff_layout(n, frame, nullptr, nullptr)) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_tff_analysis_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  TffLayout L;
  tff_layout(n, frame, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &L);
  hipError_t e;
  const int esz = xt == FQ_F32 ? 4 : 2;
  const int64_t K = F.k * F.rho;
  for (int64_t t0 = 0; t0 < n; t0 += TFF_CHUNK) {
    const int64_t nc = std::min<int64_t>(TFF_CHUNK, n - t0);
    if ((e = tff_analysis((const char*)X + t0 * ldx * esz, xt, ldx, nc, F, L.a, U + t0 * K, K,
                          s)) != hipSuccess)
      return hip_fail(e, "tff analysis");
  }
  return FQ_OK;
}

fq_status fq_tff_synthesis(void* stream, const float* V, int64_t n, const fq_tff* frame,
                           float* Y, void* ws, size_t ws_bytes) {
  if (!dim_ok(n)) return fail(FQ_ERR_INVALID_ARG, "n must be in [0, 2^30)");
  TffDev F;
  fq_status st = tff_check(frame, "frame", &F);
  if (st != FQ_OK) return st;
  if (n == 0) return FQ_OK;
  if (!V || !Y) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  if (ws_bytes < tff_layout(n, frame, nullptr, nullptr)) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_tff_synthesis_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  if (((uintptr_t)V & 7) != 0) return fail(FQ_ERR_INVALID_ARG, "V must be 8-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  TffLayout L;
  tff_layout(n, frame, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &L);
  hipError_t e;
  if ((e = tff_transpose_r2(F, L.r2t, s)) != hipSuccess) return hip_fail(e, "transpose R2");
  const int64_t K = F.k * F.rho;
  for (int64_t t0 = 0; t0 < n; t0 += TFF_CHUNK) {
    const int64_t nc = std::min<int64_t>(TFF_CHUNK, n - t0);
    if ((e = tff_synthesis(V + t0 * K, K, nc, F, L.r2t, L.a, Y + t0 * F.d, F.d, s)) != hipSuccess)
      return hip_fail(e, "tff synthesis");
  }
  return FQ_OK;
}

fq_status fq_frame_apply_tff(void* stream, const void* X, int xt, int64_t n_tokens,
                             int64_t ldx, const uint32_t* codes, const float* scale,
                             const float* zero, const fq_tff* frame_out,
                             const fq_tff* frame_in, float* Y, void* ws, size_t ws_bytes) {
  return fq_frame_apply_tff_nbit(stream, X, xt, n_tokens, ldx, codes, 2, scale, zero, frame_out,
                                 frame_in, Y, ws, ws_bytes);
}

// checks shared by fq_frame_apply_tff_nbit and its allocation-free variant (no launch)
static fq_status apply_tff_check(const void* X, int xt, int64_t n_tokens, int64_t ldx,
                                 const uint32_t* codes, int bits, const float* scale,
                                 const float* zero, const fq_tff* frame_out,
                                 const fq_tff* frame_in, float* Y, TffDev* Fo, TffDev* Fi) {
  if (bits != 2 && bits != 4) return fail(FQ_ERR_UNSUPPORTED, "the float inference kernels take 2- or 4-bit codes");
  if (xt < FQ_F32 || xt > FQ_BF16) return fail(FQ_ERR_INVALID_ARG, "xt must be FQ_F32, FQ_F16 or FQ_BF16");
  if (!dim_ok(n_tokens)) return fail(FQ_ERR_INVALID_ARG, "n_tokens must be in [0, 2^30)");
  fq_status st = tff_check(frame_out, "frame_out", Fo);
  if (st != FQ_OK) return st;
  if ((st = tff_check(frame_in, "frame_in", Fi)) != FQ_OK) return st;
  if (ldx < Fi->d) return fail(FQ_ERR_INVALID_ARG, "ldx must be >= d_in");
  if (n_tokens == 0) return FQ_OK;
  if (!X || !codes || !scale || !zero || !Y) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  return FQ_OK;
}

// the launches of fq_frame_apply_tff_nbit on a carved scratch area (256-byte aligned)
static fq_status apply_tff_launch(hipStream_t s, const void* X, int xt, int64_t n_tokens,
                                  int64_t ldx, const uint32_t* codes, int bits,
                                  const float* scale, const float* zero, const TffDev& Fo,
                                  const TffDev& Fi, float* Y, const ApplyTffLayout& L) {
  const int64_t K_in = Fi.k * Fi.rho, K_out = Fo.k * Fo.rho;
  const int64_t ldu = (K_in + 15) / 16 * 16;
  hipError_t e;
  if ((e = tff_transpose_r2(Fo, L.r2t, s)) != hipSuccess) return hip_fail(e, "transpose R2");
  const int esz = xt == FQ_F32 ? 4 : 2;
  for (int64_t t0 = 0; t0 < n_tokens; t0 += APPLY_NT) {
    const int nt = (int)std::min<int64_t>(APPLY_NT, n_tokens - t0);
    if ((e = tff_analysis((const char*)X + t0 * ldx * esz, xt, ldx, nt, Fi, L.y, L.U, ldu, s)) !=
        hipSuccess)
      return hip_fail(e, "tff analysis");
    const int64_t nwords = bits == 2 ? (K_in + 15) / 16 : (K_in + 7) / 8;
    if ((e = apply_codes(L.U, ldu, nt, codes, K_out, nwords, scale, zero, L.V, s, bits)) != hipSuccess)
      return hip_fail(e, "apply codes");
    if ((e = tff_synthesis(L.V, K_out, nt, Fo, L.r2t, L.z, Y + t0 * Fo.d, Fo.d, s)) != hipSuccess)
      return hip_fail(e, "tff synthesis");
  }
  return FQ_OK;
}

fq_status fq_frame_apply_tff_nbit(void* stream, const void* X, int xt, int64_t n_tokens,
                                  int64_t ldx, const uint32_t* codes, int bits, const float* scale,
                                  const float* zero, const fq_tff* frame_out,
                                  const fq_tff* frame_in, float* Y, void* ws, size_t ws_bytes) {
  TffDev Fo, Fi;
  fq_status st = apply_tff_check(X, xt, n_tokens, ldx, codes, bits, scale, zero, frame_out,
                                 frame_in, Y, &Fo, &Fi);
  if (st != FQ_OK || n_tokens == 0) return st;
  if (ws_bytes < apply_tff_layout(frame_out, frame_in, nullptr, nullptr))
    return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_frame_apply_tff_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  ApplyTffLayout L;
  apply_tff_layout(frame_out, frame_in, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &L);
  return apply_tff_launch((hipStream_t)stream, X, xt, n_tokens, ldx, codes, bits, scale, zero,
                          Fo, Fi, Y, L);
}

fq_status fq_frame_apply_tff_noalloc(void* stream, const void* X, int xt, int64_t n_tokens,
                                     int64_t ldx, const uint32_t* codes, int bits,
                                     const float* scale, const float* zero,
                                     const fq_tff* frame_out, const fq_tff* frame_in, float* Y) {
  TffDev Fo, Fi;
  fq_status st = apply_tff_check(X, xt, n_tokens, ldx, codes, bits, scale, zero, frame_out,
                                 frame_in, Y, &Fo, &Fi);
  if (st != FQ_OK || n_tokens == 0) return st;
  // the carve-up starts at the array's (256-byte aligned) base and must end inside it
  if (apply_tff_layout(frame_out, frame_in, nullptr, nullptr) - 256 > FQ_NOALLOC_SCRATCH_BYTES)
    return fail(FQ_ERR_UNSUPPORTED, "the frames need more scratch than FQ_NOALLOC_SCRATCH_BYTES "
                                    "(use fq_frame_apply_tff_nbit with a caller workspace)");
  void* base = nullptr;
  if ((st = scratch_of_current_device(&base)) != FQ_OK) return st;
  ApplyTffLayout L;
  apply_tff_layout(frame_out, frame_in, base, &L);
  return apply_tff_launch((hipStream_t)stream, X, xt, n_tokens, ldx, codes, bits, scale, zero,
                          Fo, Fi, Y, L);
}

// ================================================================ rounded activations
fq_status fq_act_quantize(void* stream, const float* U, int64_t n, int64_t K, int act_bits,
                          int8_t* Cq, float* delta) {
  if (act_bits < 2 || act_bits > 8) return fail(FQ_ERR_INVALID_ARG, "act_bits must be in [2, 8]");
  if (!dim_ok(n) || !dim_ok(K)) return fail(FQ_ERR_INVALID_ARG, "dimensions must be in [0, 2^30)");
  if (n == 0) return FQ_OK;
  if (!U || !Cq || !delta) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  hipError_t e = act_quantize(U, K, n, K, act_bits, Cq, K, 0, delta, nullptr, (hipStream_t)stream);
  return e == hipSuccess ? FQ_OK : hip_fail(e, "activation rounding");
}

struct ApplyActqLayout { ApplyTffLayout base; int8_t* Cq; float* delta; int* csum; };

static size_t apply_actq_layout(const fq_tff* fo, const fq_tff* fi, void* base, ApplyActqLayout* L) {
  ApplyActqLayout l{};
  const size_t head = apply_tff_layout(fo, fi, base, &l.base);      // includes 256 of slack
  const int64_t nwords = (fi->k * fi->rho + 15) / 16;
  Carver c(base ? (char*)base + head : nullptr);
  l.Cq = c.take<int8_t>((size_t)(APPLY_NT * 16 * nwords));
  l.delta = c.take<float>(APPLY_NT);
  l.csum = c.take<int>(APPLY_NT);
  if (L) *L = l;
  return head + c.off + 256;
}

size_t fq_frame_apply_tff_actq_workspace_bytes(const fq_tff* frame_out, const fq_tff* frame_in) {
  if (!tff_dims_ok(frame_out) || !tff_dims_ok(frame_in)) return 0;
  return apply_actq_layout(frame_out, frame_in, nullptr, nullptr);
}

fq_status fq_frame_apply_tff_actq(void* stream, const void* X, int xt, int64_t n_tokens,
                                  int64_t ldx, const uint32_t* codes, int bits,
                                  const float* scale, const float* zero,
                                  const fq_tff* frame_out, const fq_tff* frame_in, int act_bits,
                                  float* Y, void* ws, size_t ws_bytes) {
  if (xt < FQ_F32 || xt > FQ_BF16) return fail(FQ_ERR_INVALID_ARG, "xt must be FQ_F32, FQ_F16 or FQ_BF16");
  if (bits != 2 && bits != 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2 or 4 (3-bit codes do not spread into bytes)");
  if (act_bits < 2 || act_bits > 8) return fail(FQ_ERR_INVALID_ARG, "act_bits must be in [2, 8]");
  if (!dim_ok(n_tokens)) return fail(FQ_ERR_INVALID_ARG, "n_tokens must be in [0, 2^30)");
  TffDev Fo, Fi;
  fq_status st = tff_check(frame_out, "frame_out", &Fo);
  if (st != FQ_OK) return st;
  if ((st = tff_check(frame_in, "frame_in", &Fi)) != FQ_OK) return st;
  if (ldx < Fi.d) return fail(FQ_ERR_INVALID_ARG, "ldx must be >= d_in");
  if (n_tokens == 0) return FQ_OK;
  if (!X || !codes || !scale || !zero || !Y) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  if (ws_bytes < apply_actq_layout(frame_out, frame_in, nullptr, nullptr))
    return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_frame_apply_tff_actq_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  ApplyActqLayout L;
  apply_actq_layout(frame_out, frame_in, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &L);
  const int64_t K_in = Fi.k * Fi.rho, K_out = Fo.k * Fo.rho;
  const int cpw = 32 / bits;
  const int64_t ldu = (K_in + 15) / 16 * 16, nwords = (K_in + cpw - 1) / cpw;
  hipError_t e;
  if ((e = tff_transpose_r2(Fo, L.base.r2t, s)) != hipSuccess) return hip_fail(e, "transpose R2");
  const int esz = xt == FQ_F32 ? 4 : 2;
  for (int64_t t0 = 0; t0 < n_tokens; t0 += APPLY_NT) {
    const int nt = (int)std::min<int64_t>(APPLY_NT, n_tokens - t0);
    if ((e = tff_analysis((const char*)X + t0 * ldx * esz, xt, ldx, nt, Fi, L.base.y, L.base.U, ldu, s)) !=
        hipSuccess)
      return hip_fail(e, "tff analysis");
    if ((e = act_quantize(L.base.U, ldu, nt, K_in, act_bits, L.Cq, cpw * nwords, cpw, L.delta, L.csum, s)) !=
        hipSuccess)
      return hip_fail(e, "activation rounding");
    if ((e = apply_codes_i8(L.Cq, cpw * nwords, L.delta, L.csum, nt, bits, codes, K_out, nwords, scale,
                            zero, L.base.V, s)) != hipSuccess)
      return hip_fail(e, "apply codes");
    if ((e = tff_synthesis(L.base.V, K_out, nt, Fo, L.base.r2t, L.base.z, Y + t0 * Fo.d, Fo.d, s)) != hipSuccess)
      return hip_fail(e, "tff synthesis");
  }
  return FQ_OK;
}

// ================================================================ dense frame on the device
static constexpr int64_t TFF_MAT_COLS = 512;   // frame columns per pass of the materialisation

static size_t tff_mat_layout(const fq_tff* f, void* base, float** Z, float** Pt, float** R2t) {
  Carver c(base);
  const int64_t nc = std::min<int64_t>(TFF_MAT_COLS, f->k * f->rho);
  float* z = c.take<float>((size_t)(nc * f->d));
  float* pt = c.take<float>((size_t)(nc * f->d));
  float* r = c.take<float>((size_t)(f->d2 * f->d2));
  if (Z) *Z = z;
  if (Pt) *Pt = pt;
  if (R2t) *R2t = r;
  return c.off + 256;
}

size_t fq_tff_materialize_workspace_bytes(const fq_tff* frame) {
  if (!tff_dims_ok(frame)) return 0;
  return tff_mat_layout(frame, nullptr, nullptr, nullptr, nullptr);
}

fq_status fq_tff_materialize(void* stream, const fq_tff* frame, float* P, int64_t ldp, void* ws,
                             size_t ws_bytes) {
  TffDev F;
  fq_status st = tff_check(frame, "frame", &F);
  if (st != FQ_OK) return st;
  const int64_t K = F.k * F.rho;
  if (ldp < K) return fail(FQ_ERR_INVALID_ARG, "ldp must be >= k * rho");
  if (!P) return fail(FQ_ERR_INVALID_ARG, "NULL P");
  if (ws_bytes < tff_mat_layout(frame, nullptr, nullptr, nullptr, nullptr))
    return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_tff_materialize_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  float *Z, *Pt, *R2t;
  tff_mat_layout(frame, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &Z, &Pt, &R2t);
  hipError_t e;
  if ((e = tff_transpose_r2(F, R2t, s)) != hipSuccess) return hip_fail(e, "transpose R2");
  if ((e = tff_materialize(F, R2t, Z, Pt, std::min<int64_t>(TFF_MAT_COLS, K), P, ldp, s)) != hipSuccess)
    return hip_fail(e, "materialize");
  return FQ_OK;
}

// ================================================================ structured S2 / S4
static constexpr int64_t TFFP_MAX = (int64_t)1 << 21;   // d limit of the structured pass
static constexpr int64_t TFFP_MAX_K = (int64_t)65535 * 32; // K limit (32-tiles per grid axis)

static fq_status tffp_check(const fq_tff* f, const char* which, TffDev* F) {
  fq_status st = tff_check(f, which, F);
  if (st != FQ_OK) return st;
  if (F->d > TFFP_MAX || F->k * F->rho > TFFP_MAX_K) {
    char msg[128];
    snprintf(msg, sizeof msg, "%s: d must not exceed 2^21 and k * rho 65535 * 32 here", which);
    return fail(FQ_ERR_UNSUPPORTED, msg);
  }
  return FQ_OK;
}

static TffDev tff_dev_of(const fq_tff* f) {
  TffDev F;
  F.d = f->d; F.k = f->k; F.rho = f->rho; F.m = f->d / f->rho;
  F.R1 = f->R1; F.d1 = (int)f->d1; F.R2 = f->R2; F.d2 = (int)f->d2;
  return F;
}

static bool tffp_dims_ok(const fq_tff* f) {
  return tff_dims_ok(f) && f->d <= TFFP_MAX && f->k * f->rho <= TFFP_MAX_K;
}

// F_c planes of both frames, then the stage buffers (the largest stage of each).
struct TffAnaLayout {
  u16 *fi_hi, *fi_lo, *fo_hi, *fo_lo;   // F_c planes of frame_in / frame_out
  float* tmp;                           // rotation scratch, aliased with the DFT output
  u16 *y_hi, *y_lo;                     // rotated rows, block order
  float* mid;                           // (W P_in)^T or (H P_in)^T
};

static size_t tff_ana_layout(const fq_tff* fo, const fq_tff* fi, void* base, TffAnaLayout* L) {
  const TffDev Fo = tff_dev_of(fo), Fi = tff_dev_of(fi);
  const TffPassGeom go = tff_pass_geom(Fo), gi = tff_pass_geom(Fi);
  const int64_t d_out = fo->d, d_in = fi->d, K_out = fo->k * fo->rho, K_in = fi->k * fi->rho;
  const int64_t tmp = std::max({d_out * std::max(d_in, K_in), K_in * std::max(d_out, K_out),
                                d_in * std::max(d_in, K_in), K_in * std::max(d_in, K_in)});
  const int64_t yp = std::max({d_out * gi.nb * gi.pm, K_in * go.nb * go.pm,
                               std::max(d_in, K_in) * gi.nb * gi.pm});
  const int64_t mid = K_in * std::max(d_out, d_in);
  Carver c(base);
  TffAnaLayout l{};
  l.fi_hi = c.take<u16>((size_t)(gi.nb * gi.pm * gi.pk));
  l.fi_lo = c.take<u16>((size_t)(gi.nb * gi.pm * gi.pk));
  l.fo_hi = c.take<u16>((size_t)(go.nb * go.pm * go.pk));
  l.fo_lo = c.take<u16>((size_t)(go.nb * go.pm * go.pk));
  l.tmp = c.take<float>((size_t)tmp);
  l.y_hi = c.take<u16>((size_t)yp);
  l.y_lo = c.take<u16>((size_t)yp);
  l.mid = c.take<float>((size_t)mid);
  if (L) *L = l;
  return c.off + 256;
}

size_t fq_frame_analysis_tff_workspace_bytes(int wt, const fq_tff* frame_out,
                                             const fq_tff* frame_in) {
  if (wt < 0 || wt > 2 || !tffp_dims_ok(frame_out) || !tffp_dims_ok(frame_in)) return 0;
  return tff_ana_layout(frame_out, frame_in, nullptr, nullptr);
}

fq_status fq_frame_analysis_tff(void* stream, const void* W, int wt, const fq_tff* frame_out,
                                const fq_tff* frame_in, const float* H, float* D, float* Ht,
                                void* ws, size_t ws_bytes) {
  if (wt < FQ_F32 || wt > FQ_BF16) return fail(FQ_ERR_INVALID_ARG, "wt must be FQ_F32, FQ_F16 or FQ_BF16");
  TffDev Fo, Fi;
  fq_status st = tffp_check(frame_out, "frame_out", &Fo);
  if (st != FQ_OK) return st;
  if ((st = tffp_check(frame_in, "frame_in", &Fi)) != FQ_OK) return st;
  if (D && !W) return fail(FQ_ERR_INVALID_ARG, "W is required for D");
  if (Ht && !H) return fail(FQ_ERR_INVALID_ARG, "H is required for Ht");
  const size_t need = tff_ana_layout(frame_out, frame_in, nullptr, nullptr);
  if (ws_bytes < need) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_frame_analysis_tff_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  if (!D && !Ht) return FQ_OK;
  hipStream_t s = (hipStream_t)stream;
  TffAnaLayout L;
  tff_ana_layout(frame_out, frame_in, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &L);
  const int64_t K_in = Fi.k * Fi.rho;
  hipError_t e;
  if ((e = tff_dft_blocks(Fi, L.fi_hi, L.fi_lo, s)) != hipSuccess) return hip_fail(e, "frame_in blocks");
  if (D) {
    if ((e = tff_dft_blocks(Fo, L.fo_hi, L.fo_lo, s)) != hipSuccess) return hip_fail(e, "frame_out blocks");
    // (W P_in)^T: K_in x d_out
    if ((e = tff_rows_analysis_t(W, wt, Fi.d, Fo.d, Fi, L.fi_hi, L.fi_lo, L.tmp, L.y_hi, L.y_lo,
                                 L.tmp, L.mid, Fo.d, s)) != hipSuccess)
      return hip_fail(e, "analysis of the rows of W");
    // D = ((W P_in)^T P_out)^T: K_out x K_in
    if ((e = tff_rows_analysis_t(L.mid, FQ_F32, Fo.d, K_in, Fo, L.fo_hi, L.fo_lo, L.tmp, L.y_hi,
                                 L.y_lo, L.tmp, D, K_in, s)) != hipSuccess)
      return hip_fail(e, "analysis of the columns of W P_in");
  }
  if (Ht) {
    // (H P_in)^T: K_in x d_in, then Ht = ((H P_in)^T P_in)^T, symmetrized
    if ((e = tff_rows_analysis_t(H, FQ_F32, Fi.d, Fi.d, Fi, L.fi_hi, L.fi_lo, L.tmp, L.y_hi,
                                 L.y_lo, L.tmp, L.mid, Fi.d, s)) != hipSuccess)
      return hip_fail(e, "analysis of the rows of H");
    if ((e = tff_rows_analysis_t(L.mid, FQ_F32, Fi.d, K_in, Fi, L.fi_hi, L.fi_lo, L.tmp, L.y_hi,
                                 L.y_lo, L.tmp, Ht, K_in, s)) != hipSuccess)
      return hip_fail(e, "analysis of the columns of H P_in");
    if ((e = sym_average(Ht, K_in, K_in, s)) != hipSuccess) return hip_fail(e, "symmetrize Ht");
  }
  return FQ_OK;
}

struct TffSynLayout {
  u16 *fi_hi, *fi_lo, *fo_hi, *fo_lo;
  u16* v1;              // (codes - zero)^T, block order of frame_out (K_in rows)
  u16 *v2_hi, *v2_lo;   // P_out diag(scale) (Q - zero), block order of frame_in (d_out rows)
  float *z, *tmp, *mid;
};

static size_t tff_syn_layout(const fq_tff* fo, const fq_tff* fi, void* base, TffSynLayout* L) {
  const TffDev Fo = tff_dev_of(fo), Fi = tff_dev_of(fi);
  const TffPassGeom go = tff_pass_geom(Fo), gi = tff_pass_geom(Fi);
  const int64_t d_out = fo->d, d_in = fi->d, K_in = fi->k * fi->rho;
  const int64_t big = std::max(K_in * d_out, d_out * d_in);
  Carver c(base);
  TffSynLayout l{};
  l.fi_hi = c.take<u16>((size_t)(gi.nb * gi.pm * gi.pk));
  l.fi_lo = c.take<u16>((size_t)(gi.nb * gi.pm * gi.pk));
  l.fo_hi = c.take<u16>((size_t)(go.nb * go.pm * go.pk));
  l.fo_lo = c.take<u16>((size_t)(go.nb * go.pm * go.pk));
  l.v1 = c.take<u16>((size_t)(K_in * go.nb * go.pk));
  l.v2_hi = c.take<u16>((size_t)(d_out * gi.nb * gi.pk));
  l.v2_lo = c.take<u16>((size_t)(d_out * gi.nb * gi.pk));
  l.z = c.take<float>((size_t)big);
  l.tmp = c.take<float>((size_t)big);
  l.mid = c.take<float>((size_t)big);
  if (L) *L = l;
  return c.off + 256;
}

size_t fq_frame_synthesis_tff_workspace_bytes(const fq_tff* frame_out, const fq_tff* frame_in) {
  if (!tffp_dims_ok(frame_out) || !tffp_dims_ok(frame_in)) return 0;
  return tff_syn_layout(frame_out, frame_in, nullptr, nullptr);
}

fq_status fq_frame_synthesis_tff(void* stream, const uint32_t* codes, int bits,
                                 const float* scale, const float* zero, const fq_tff* frame_out,
                                 const fq_tff* frame_in, float* W_hat, void* ws, size_t ws_bytes) {
  if (bits < 2 || bits > 4) return fail(FQ_ERR_UNSUPPORTED, "bits must be 2, 3 or 4");
  TffDev Fo, Fi;
  fq_status st = tffp_check(frame_out, "frame_out", &Fo);
  if (st != FQ_OK) return st;
  if ((st = tffp_check(frame_in, "frame_in", &Fi)) != FQ_OK) return st;
  if (!codes || !scale || !zero || !W_hat) return fail(FQ_ERR_INVALID_ARG, "NULL array argument");
  const size_t need = tff_syn_layout(frame_out, frame_in, nullptr, nullptr);
  if (ws_bytes < need) return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_frame_synthesis_tff_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  TffSynLayout L;
  tff_syn_layout(frame_out, frame_in, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &L);
  const int64_t K_in = Fi.k * Fi.rho;
  hipError_t e;
  // W^ = P_out diag(scale) (Q - zero) P_in^T, formed from the left: the output frame's
  // blocks carry the scale (P_out diag(scale)), so the code matrix enters as exact
  // integers, and the last synthesis writes rows of W^ directly
  if ((e = tff_dft_blocks(Fi, L.fi_hi, L.fi_lo, s)) != hipSuccess) return hip_fail(e, "frame_in blocks");
  if ((e = tff_dft_blocks(Fo, L.fo_hi, L.fo_lo, s, scale)) != hipSuccess)
    return hip_fail(e, "frame_out blocks");
  // N = (P_out diag(scale) (Q - zero))^T: K_in x d_out, from the columns of the codes
  if ((e = tff_dequant_gather_t(codes, bits, zero, K_in, Fo, L.v1, s)) != hipSuccess)
    return hip_fail(e, "dequant");
  if ((e = tff_rows_synthesis(L.v1, nullptr, K_in, Fo, L.fo_hi, L.fo_lo, L.z, L.tmp, L.mid,
                              Fo.d, s)) != hipSuccess)
    return hip_fail(e, "synthesis of the code columns");
  // W^ = (N^T) P_in^T: d_out rows
  if ((e = tff_gather_rows(L.mid, Fo.d, Fo.d, nullptr, Fi, L.v2_hi, L.v2_lo, s)) != hipSuccess)
    return hip_fail(e, "gather");
  if ((e = tff_rows_synthesis(L.v2_hi, L.v2_lo, Fo.d, Fi, L.fi_hi, L.fi_lo, L.z, L.tmp, W_hat,
                              Fi.d, s)) != hipSuccess)
    return hip_fail(e, "synthesis of the rows");
  return FQ_OK;
}

// ================================================================ seeded rotation factors
static size_t seed_layout(int64_t n, void* base, double** G, double** V, double** ab) {
  Carver c(base);
  double* g = c.take<double>((size_t)(n * n));
  double* v = c.take<double>((size_t)(n * n));
  double* a = c.take<double>((size_t)(2 * n));
  if (G) *G = g;
  if (V) *V = v;
  if (ab) *ab = a;
  return c.off + 256;
}

// ================================================================ frame choice
// Longest row support of the unit-norm tight frame that spectral tetris builds for d_c
// vectors in C^rho_c (the appendix on constructing TFFs), in exact integer arithmetic with
// squared norms in units of 1 / rho_c: every row must reach d_c units; a 1 adds rho_c; a
// remainder 0 < x < rho_c closes the row with the 2 x 2 block T(x / rho_c), which also puts
// 2 rho_c - x units into the next row over the same two columns.  A row's support is the
// run of columns from its first entry (the previous row's block, if any) to its last.
// Returns false when the construction fails (a block overfills a row, the last row has a
// remainder, or the columns do not come out at d_c).
static bool st_max_support(int64_t rho_c, int64_t d_c, int64_t* maxsup) {
  if (rho_c < 1 || d_c < rho_c) return false;
  int64_t col = 0, carry = 0, block_col = 0, best = 0;
  for (int64_t r = 0; r < rho_c; ++r) {
    int64_t need = d_c - carry;
    if (need < 0) return false;
    const int64_t start = carry > 0 ? block_col : col;
    carry = 0;
    const int64_t ones = need / rho_c;
    col += ones;
    need -= ones * rho_c;
    if (need > 0) {
      if (r + 1 >= rho_c) return false;
      block_col = col;
      col += 2;
      carry = 2 * rho_c - need;
    }
    best = std::max(best, col - start);
  }
  if (col != d_c) return false;
  *maxsup = best;
  return true;
}

int fq_tff_frame_valid(int64_t d, int64_t k, int64_t rho) {
  if (d < 2 || rho < 2 || k < 1 || d % 2 || rho % 2 || !dim_ok(d) || !dim_ok(k) || !dim_ok(rho))
    return 0;
  int64_t sup = 0;
  if (!st_max_support(rho / 2, d / 2, &sup)) return 0;
  // the modulation by the k-th roots of unity is tight exactly when no row has two support
  // columns congruent mod k; a support is a run of consecutive columns
  return sup <= k ? 1 : 0;
}

fq_status fq_tff_choose(int64_t d, double r, int64_t rho, int64_t* k, int64_t* d1, int64_t* d2) {
  if (!k) return fail(FQ_ERR_INVALID_ARG, "NULL k");
  if (d < 2 || rho < 2 || d % 2 || rho % 2 || !dim_ok(d) || !dim_ok(rho))
    return fail(FQ_ERR_INVALID_ARG, "d and rho must be even and in [2, 2^30)");
  if (!(r > 0.0) || !isfinite(r)) return fail(FQ_ERR_INVALID_ARG, "r must be finite and > 0");
  const double k0 = nearbyint(r * (double)d / (double)rho);     // ties to even
  if (!(k0 >= 1.0) || k0 >= (double)DIM_MAX) return fail(FQ_ERR_UNSUPPORTED, "no k >= 1 at this redundancy");
  int64_t kk = (int64_t)k0;
  while (kk >= 1 && !fq_tff_frame_valid(d, kk, rho)) --kk;
  if (kk < 1) return fail(FQ_ERR_UNSUPPORTED, "no valid (k, rho) at or below this redundancy");
  *k = kk;
  // rotation factors: d1 the largest divisor of d not above sqrt(d), d2 = d / d1
  int64_t best = 1;
  for (int64_t a = 1; a * a <= d; ++a)
    if (d % a == 0) best = a;
  if (d1) *d1 = best;
  if (d2) *d2 = d / best;
  return FQ_OK;
}

size_t fq_tff_rotation_factors_workspace_bytes(int64_t d1, int64_t d2) {
  if (d1 < 1 || d2 < 1 || d1 > TFF_SEED_MAX_N || d2 > TFF_SEED_MAX_N) return 0;
  return seed_layout(std::max(d1, d2), nullptr, nullptr, nullptr, nullptr);
}

fq_status fq_tff_rotation_factors(void* stream, uint64_t seed, int64_t d1, int64_t d2, float* R1,
                                  float* R2, void* ws, size_t ws_bytes) {
  if (d1 < 1 || d2 < 1) return fail(FQ_ERR_INVALID_ARG, "d1 and d2 must be >= 1");
  if (d1 > TFF_SEED_MAX_N || d2 > TFF_SEED_MAX_N)
    return fail(FQ_ERR_UNSUPPORTED, "seeded factors are drawn for d1, d2 <= 1024");
  if (!R1 || !R2) return fail(FQ_ERR_INVALID_ARG, "NULL R1 or R2");
  const int64_t n = std::max(d1, d2);
  if (ws_bytes < seed_layout(n, nullptr, nullptr, nullptr, nullptr))
    return fail(FQ_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than fq_tff_rotation_factors_workspace_bytes()");
  if (!ws || !aligned16(ws)) return fail(FQ_ERR_INVALID_ARG, "workspace is NULL or not 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  double *G, *V, *ab;
  seed_layout(n, (void*)(((uintptr_t)ws + 255) & ~(uintptr_t)255), &G, &V, &ab);
  hipError_t e;
  if ((e = tff_seeded_factor(seed, 0, (int)d1, G, V, ab, R1, s)) != hipSuccess) return hip_fail(e, "R1");
  if ((e = tff_seeded_factor(seed, 1, (int)d2, G, V, ab, R2, s)) != hipSuccess) return hip_fail(e, "R2");
  return FQ_OK;
}

}  // extern "C"
