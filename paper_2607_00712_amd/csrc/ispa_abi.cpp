// Host side of libispa: argument validation, key-range arithmetic, the
// statistics handle over a caller-owned workspace, and kernel launches.
// Every argument error is reported before anything is enqueued.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <math.h>
#include <mutex>
#include <new>
#include <stdint.h>
#include <string.h>

#include "ispa.h"
#include "ispa_internal.h"

namespace {

constexpr int64_t kMaxDim = 16384;
constexpr size_t kWsAlign = 256;

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// byte ranges [p, p + np) and [q, q + nq) intersect
bool overlaps(const void* p, size_t np, const void* q, size_t nq) {
  return (const char*)p < (const char*)q + nq && (const char*)q < (const char*)p + np;
}

size_t round_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Workspace layout of a statistics handle (offsets in bytes, 256-aligned).
struct Layout {
  size_t G, C, L, W, Dinv, X, R, scalars, status, sqp, total;
};

bool layout_of(int32_t d_in, int32_t d_out, int64_t max_rows, Layout* out) {
  if (d_in < 1 || d_out < 1 || d_in > kMaxDim || d_out > kMaxDim) return false;
  if (d_in % 8 != 0 || d_out % 8 != 0) return false;
  if (max_rows < 1 || max_rows > (int64_t)1 << 24) return false;
  Layout l;
  size_t off = 0;
  l.G = off; off = round_up(off + (size_t)d_in * d_in * 4, kWsAlign);
  l.C = off; off = round_up(off + (size_t)d_in * d_out * 4, kWsAlign);
  l.L = off; off = round_up(off + (size_t)d_in * d_in * 4, kWsAlign);
  l.W = off; off = round_up(off + (size_t)d_in * d_out * 4, kWsAlign);
  l.Dinv = off; off = round_up(off + ispa::solve_dinv_bytes(d_in), kWsAlign);
  // L, W and Dinv are free between solves: with the room after them they hold
  // the Gram kernel's row pieces (the sums it adds in a second pass)
  {
    const size_t need = ispa::gram_fast_scratch_bytes(d_in, d_out);
    if (need > off - l.L) off = round_up(l.L + need, kWsAlign);
  }
  l.X = off; off = round_up(off + (size_t)max_rows * d_in * 2, kWsAlign);
  l.R = off; off = round_up(off + (size_t)max_rows * d_out * 2, kWsAlign);
  l.scalars = off; off = round_up(off + 4 * sizeof(double), kWsAlign);
  l.status = off; off = round_up(off + sizeof(int), kWsAlign);
  // per-workgroup partials of ||R||^2 (added to s in a fixed order)
  l.sqp = off; off = round_up(off + ispa::kDiscMaxGrid * sizeof(double), kWsAlign);
  l.total = off;
  *out = l;
  return true;
}

}  // namespace

struct ispa_stats {
  uint32_t magic;
  char* ws;
  size_t ws_bytes;
  int32_t d_in, d_out;
  int64_t max_rows;
  int64_t n_rows;
  hipStream_t stream;
  Layout lay;
};

static constexpr uint32_t kMagic = 0x49535041u;  // "ISPA"

static bool valid_handle(const ispa_stats* h) { return h != nullptr && h->magic == kMagic; }

extern "C" {

const char* ispa_status_string(int status) {
  switch (status) {
    case ISPA_OK: return "ISPA_OK";
    case ISPA_ERR_INVALID_ARG: return "ISPA_ERR_INVALID_ARG: invalid argument";
    case ISPA_ERR_UNSUPPORTED: return "ISPA_ERR_UNSUPPORTED: unsupported head_dim or dtype";
    case ISPA_ERR_NOT_SPD: return "ISPA_ERR_NOT_SPD: G + lambda I is not positive definite";
    case ISPA_ERR_HIP: return "ISPA_ERR_HIP: HIP runtime or launch failure";
    case ISPA_ERR_STATE: return "ISPA_ERR_STATE: bad handle or workspace";
    case ISPA_ERR_SCRATCH: return "ISPA_ERR_SCRATCH: needs more than the library's fixed device scratch";
    default: return "ISPA: unknown status";
  }
}

int ispa_abi_version(void) { return 104; }

}  // extern "C"

namespace {

// Validates the arguments shared by the attention calls and fills the
// launch-independent part of AttnArgs.
int attn_common(const void* q, const void* k_cache, const void* v_cache, int32_t n_q, int32_t n_heads,
                int32_t head_dim, float scale, float* out, float* lse, ispa::AttnArgs* a) {
  if (head_dim != 64 && head_dim != 128) return ISPA_ERR_UNSUPPORTED;
  if (!q || !k_cache || !v_cache || !out) return ISPA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(out)) return ISPA_ERR_INVALID_ARG;
  if ((uintptr_t)lse & 3u) return ISPA_ERR_INVALID_ARG;
  if (n_q < 1 || n_heads < 1 || n_heads > 65535) return ISPA_ERR_INVALID_ARG;
  if (!(scale == scale) || isinf(scale)) return ISPA_ERR_INVALID_ARG;
  if ((int64_t)n_heads * head_dim > ((int64_t)1 << 20)) return ISPA_ERR_INVALID_ARG;
  const float s = scale > 0.f ? scale : 1.0f / sqrtf((float)head_dim);
  memset(a, 0, sizeof(*a));
  a->q = (const uint16_t*)q;
  a->k = (const uint16_t*)k_cache;
  a->v = (const uint16_t*)v_cache;
  a->out = out;
  a->lse = lse;
  a->ld = (int64_t)n_heads * head_dim;
  a->n_q = n_q;
  a->n_heads = n_heads;
  a->scale = s;
  a->scale_log2 = s * 1.4426950408889634f;
  return ISPA_OK;
}

// Key sets of Sec. 3.4, Eq. 7-8: local = [0, s') U [lo, N), hist = [s', lo).
int chunk_ranges(int64_t cache_len, int64_t window, int64_t sink_len, int32_t n_q, bool dual, ispa::AttnRanges* r) {
  if (cache_len < n_q || cache_len > ((int64_t)1 << 31)) return ISPA_ERR_INVALID_ARG;
  if (window < 1 || sink_len < 0) return ISPA_ERR_INVALID_ARG;
  const int64_t N = cache_len;
  const int64_t s1 = sink_len < N ? sink_len : N;
  const int64_t lo = N - window > 0 ? N - window : 0;
  if (lo <= s1) {
    r->begin[0] = 0; r->end[0] = N;
    r->n_local = 1;
    r->n_total = 1;
  } else {
    int i = 0;
    if (s1 > 0) { r->begin[i] = 0; r->end[i] = s1; ++i; }
    r->begin[i] = lo; r->end[i] = N; ++i;
    r->n_local = i;
    r->n_total = i;
    if (dual) { r->begin[i] = s1; r->end[i] = lo; ++i; r->n_total = i; }
  }
  for (int i = r->n_total; i < 3; ++i) { r->begin[i] = 0; r->end[i] = 0; }
  return ISPA_OK;
}

}  // namespace

extern "C" {

int ispa_attn_chunk(const void* q, const void* k_cache, const void* v_cache, int64_t cache_len,
                    int64_t window, int64_t sink_len, int32_t n_q, int32_t n_heads, int32_t head_dim,
                    float scale, float* out, float* lse, float* out_local, float* lse_local,
                    hipStream_t stream) {
  return ispa_attn_chunk_ws(q, k_cache, v_cache, cache_len, window, sink_len, n_q, n_heads, head_dim, scale,
                            out, lse, out_local, lse_local, -1, nullptr, 0, stream);
}

size_t ispa_attn_workspace_bytes(int64_t cache_len, int64_t window, int64_t sink_len, int32_t n_q,
                                 int32_t n_heads, int32_t head_dim, int32_t dual, int32_t segments) {
  if (head_dim != 64 && head_dim != 128) return 0;
  if (n_q < 1 || n_heads < 1 || n_heads > 65535) return 0;
  ispa::AttnArgs a;
  memset(&a, 0, sizeof(a));
  a.n_q = n_q;
  a.n_heads = n_heads;
  if (chunk_ranges(cache_len, window, sink_len, n_q, dual != 0, &a.r) != ISPA_OK) return 0;
  ispa::AttnSplit sp;
  return ispa::attn_plan_split(a, head_dim, segments, &sp);
}

int ispa_attn_chunk_ws(const void* q, const void* k_cache, const void* v_cache, int64_t cache_len,
                       int64_t window, int64_t sink_len, int32_t n_q, int32_t n_heads, int32_t head_dim,
                       float scale, float* out, float* lse, float* out_local, float* lse_local,
                       int32_t segments, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  ispa::AttnArgs a;
  int st = attn_common(q, k_cache, v_cache, n_q, n_heads, head_dim, scale, out, lse, &a);
  if (st != ISPA_OK) return st;
  if (out_local && !aligned16(out_local)) return ISPA_ERR_INVALID_ARG;
  if ((uintptr_t)lse_local & 3u) return ISPA_ERR_INVALID_ARG;
  if (lse_local && !out_local) return ISPA_ERR_INVALID_ARG;
  st = chunk_ranges(cache_len, window, sink_len, n_q, out_local != nullptr, &a.r);
  if (st != ISPA_OK) return st;
  a.out_local = out_local;
  a.lse_local = lse_local;
  const size_t need = ispa::attn_plan_split(a, head_dim, segments, &a.split);
  if (a.split.n_seg > 0) {
    if (!workspace || ((uintptr_t)workspace & 255u) || workspace_bytes < need) return ISPA_ERR_INVALID_ARG;
    a.split.part_o = (float*)workspace;
    a.split.part_lse = (float*)((char*)workspace + a.split.lse_offset);
    a.split.ctr = (uint32_t*)((char*)workspace + a.split.ctr_offset);
  }
  return ispa::launch_attn_chunk(a, head_dim, stream) == hipSuccess ? ISPA_OK : ISPA_ERR_HIP;
}

}  // extern "C"

// Fixed device scratch of ispa_attn_chunk_noalloc (the split's partial
// results), one copy per GPU. In host code `scratch` only stands for the
// symbol: its device address, different on every GPU, comes from
// hipGetSymbolAddress with that GPU current, once per device, and only that
// address is passed to kernels.
static __device__ __align__(256) char scratch[ISPA_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of the current GPU's scratch (nullptr on failure).
void* device_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    g_scratch_ptr[dev] = p;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

int ispa_attn_chunk_noalloc(const void* q, const void* k_cache, const void* v_cache, int64_t cache_len,
                            int64_t window, int64_t sink_len, int32_t n_q, int32_t n_heads, int32_t head_dim,
                            float scale, float* out, float* lse, float* out_local, float* lse_local,
                            hipStream_t stream) {
  // The plan of the automatic split; 0 also for invalid arguments, which
  // ispa_attn_chunk_ws then rejects.
  const size_t need = ispa_attn_workspace_bytes(cache_len, window, sink_len, n_q, n_heads, head_dim,
                                                out_local != nullptr, 0);
  if (need > ISPA_STATIC_SCRATCH_BYTES) return ISPA_ERR_SCRATCH;
  void* ws = nullptr;
  if (need > 0 && (ws = device_scratch()) == nullptr) return ISPA_ERR_HIP;
  return ispa_attn_chunk_ws(q, k_cache, v_cache, cache_len, window, sink_len, n_q, n_heads, head_dim, scale, out,
                            lse, out_local, lse_local, 0, ws, ISPA_STATIC_SCRATCH_BYTES, stream);
}

int ispa_attn_ranges(const void* q, const void* k_cache, const void* v_cache, const int64_t* ranges,
                     int32_t n_ranges, int32_t n_q, int32_t n_heads, int32_t head_dim, float scale, float* out,
                     float* lse, hipStream_t stream) {
  ispa::AttnArgs a;
  int st = attn_common(q, k_cache, v_cache, n_q, n_heads, head_dim, scale, out, lse, &a);
  if (st != ISPA_OK) return st;
  if (n_ranges < 0 || n_ranges > 3 || (n_ranges > 0 && !ranges)) return ISPA_ERR_INVALID_ARG;
  for (int i = 0; i < n_ranges; ++i) {
    const int64_t b = ranges[2 * i], e = ranges[2 * i + 1];
    if (b < 0 || e <= b || e > ((int64_t)1 << 31)) return ISPA_ERR_INVALID_ARG;
    a.r.begin[i] = b;
    a.r.end[i] = e;
  }
  if (n_ranges == 0)
    return ispa::launch_attn_empty(out, lse, n_q, n_heads, head_dim, stream) == hipSuccess ? ISPA_OK
                                                                                           : ISPA_ERR_HIP;
  a.r.n_local = n_ranges;
  a.r.n_total = n_ranges;
  return ispa::launch_attn_chunk(a, head_dim, stream) == hipSuccess ? ISPA_OK : ISPA_ERR_HIP;
}

int ispa_attn_merge(const float* out_a, const float* lse_a, const float* out_b, const float* lse_b, int32_t n_q,
                    int32_t n_heads, int32_t head_dim, float* out, float* lse, hipStream_t stream) {
  if (!out_a || !lse_a || !out_b || !lse_b || !out) return ISPA_ERR_INVALID_ARG;
  if (!aligned16(out_a) || !aligned16(out_b) || !aligned16(out)) return ISPA_ERR_INVALID_ARG;
  if (((uintptr_t)lse_a & 3u) || ((uintptr_t)lse_b & 3u) || ((uintptr_t)lse & 3u)) return ISPA_ERR_INVALID_ARG;
  if (n_q < 1 || n_heads < 1 || head_dim < 4 || head_dim % 4 != 0) return ISPA_ERR_INVALID_ARG;
  if ((int64_t)n_heads * head_dim > ((int64_t)1 << 20)) return ISPA_ERR_INVALID_ARG;
  // the merged LSE is written while other rows still read the inputs' LSE
  const size_t lse_bytes = (size_t)n_q * n_heads * 4;
  auto overlap = [](const void* x, const void* y, size_t n) {
    return (const char*)x < (const char*)y + n && (const char*)y < (const char*)x + n;
  };
  if (lse && (overlap(lse, lse_a, lse_bytes) || overlap(lse, lse_b, lse_bytes))) return ISPA_ERR_INVALID_ARG;
  return ispa::launch_attn_merge2(out_a, lse_a, out_b, lse_b, n_q, n_heads, head_dim, out, lse, stream) ==
                 hipSuccess
             ? ISPA_OK
             : ISPA_ERR_HIP;
}

size_t ispa_stats_workspace_bytes(int32_t d_in, int32_t d_out, int64_t max_rows) {
  Layout l;
  return layout_of(d_in, d_out, max_rows, &l) ? l.total : 0;
}

int ispa_stats_create(ispa_stats** handle, void* workspace, size_t workspace_bytes, int32_t d_in,
                      int32_t d_out, int64_t max_rows, hipStream_t stream) {
  if (!handle) return ISPA_ERR_INVALID_ARG;
  *handle = nullptr;
  Layout l;
  if (!layout_of(d_in, d_out, max_rows, &l)) return ISPA_ERR_INVALID_ARG;
  if (!workspace || ((uintptr_t)workspace % kWsAlign) != 0) return ISPA_ERR_INVALID_ARG;
  if (workspace_bytes < l.total) return ISPA_ERR_STATE;
  ispa_stats* h = new (std::nothrow) ispa_stats;
  if (!h) return ISPA_ERR_STATE;
  h->magic = kMagic;
  h->ws = (char*)workspace;
  h->ws_bytes = workspace_bytes;
  h->d_in = d_in;
  h->d_out = d_out;
  h->max_rows = max_rows;
  h->n_rows = 0;
  h->stream = stream;
  h->lay = l;
  const int rc = ispa_stats_reset(h);
  if (rc != ISPA_OK) {
    h->magic = 0;
    delete h;
    return rc;
  }
  *handle = h;
  return ISPA_OK;
}

int ispa_stats_reset(ispa_stats* h) {
  if (!valid_handle(h)) return ISPA_ERR_STATE;
  h->n_rows = 0;
  // G, C (contiguous at the start of the workspace) and the scalars
  if (ispa::launch_zero(h->ws + h->lay.G, h->lay.L, h->stream) != hipSuccess) return ISPA_ERR_HIP;
  if (ispa::launch_zero(h->ws + h->lay.scalars, 4 * sizeof(double), h->stream) != hipSuccess) return ISPA_ERR_HIP;
  return ISPA_OK;
}

int ispa_stats_destroy(ispa_stats* h) {
  if (!valid_handle(h)) return ISPA_ERR_STATE;
  h->magic = 0;
  delete h;
  return ISPA_OK;
}

int ispa_stats_views(const ispa_stats* h, float** G, float** C, double** sq_norm_r, int64_t* n_rows) {
  if (!valid_handle(h)) return ISPA_ERR_STATE;
  if (G) *G = (float*)(h->ws + h->lay.G);
  if (C) *C = (float*)(h->ws + h->lay.C);
  if (sq_norm_r) *sq_norm_r = (double*)(h->ws + h->lay.scalars);
  if (n_rows) *n_rows = h->n_rows;
  return ISPA_OK;
}

int ispa_accum_stats(ispa_stats* h, const void* x, int32_t x_dtype, const void* y_full,
                     const void* y_local, int32_t y_dtype, int64_t n_rows) {
  if (!valid_handle(h)) return ISPA_ERR_STATE;
  if (x_dtype != ISPA_DTYPE_BF16 && x_dtype != ISPA_DTYPE_F32) return ISPA_ERR_UNSUPPORTED;
  if (y_dtype != ISPA_DTYPE_BF16 && y_dtype != ISPA_DTYPE_F32) return ISPA_ERR_UNSUPPORTED;
  if (n_rows < 0) return ISPA_ERR_INVALID_ARG;
  if (n_rows == 0) return ISPA_OK;
  if (!x || !y_full || !y_local) return ISPA_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(y_full) || !aligned16(y_local)) return ISPA_ERR_INVALID_ARG;

  const size_t xs = x_dtype == ISPA_DTYPE_F32 ? 4 : 2;
  const size_t ys = y_dtype == ISPA_DTYPE_F32 ? 4 : 2;
  uint16_t* xb = (uint16_t*)(h->ws + h->lay.X);
  uint16_t* rb = (uint16_t*)(h->ws + h->lay.R);
  float* G = (float*)(h->ws + h->lay.G);
  float* C = (float*)(h->ws + h->lay.C);
  double* sq = (double*)(h->ws + h->lay.scalars);
  double* sqp = (double*)(h->ws + h->lay.sqp);
  for (int64_t r0 = 0; r0 < n_rows; r0 += h->max_rows) {
    const int64_t rows = n_rows - r0 < h->max_rows ? n_rows - r0 : h->max_rows;
    const char* xp = (const char*)x + (size_t)r0 * h->d_in * xs;
    const char* yf = (const char*)y_full + (size_t)r0 * h->d_out * ys;
    const char* yl = (const char*)y_local + (size_t)r0 * h->d_out * ys;
    // keep the aliasing of x and y_local visible to the kernel for every block
    const void* xarg = (x == y_local) ? (const void*)yl : (const void*)xp;
    if (ispa::launch_discrepancy(xarg, x_dtype, yf, yl, y_dtype, rows, h->d_in, h->d_out, xb, rb, sqp,
                                 h->stream) != hipSuccess)
      return ISPA_ERR_HIP;
    const uint16_t* xg = x_dtype == ISPA_DTYPE_BF16 ? (const uint16_t*)xp : xb;
    // the solve's areas (L to X) are free between solves: scratch for the Gram
    if (ispa::launch_gram(xg, rb, rows, h->d_in, h->d_out, G, C, sqp,
                          ispa::discrepancy_grid(rows, h->d_in, h->d_out), sq, (float*)(h->ws + h->lay.L),
                          h->lay.X - h->lay.L, h->stream) != hipSuccess)
      return ISPA_ERR_HIP;
  }
  h->n_rows += n_rows;
  return ISPA_OK;
}

namespace {
// Enqueue the solve of handle h; eps and the status word land in the
// workspace scalars [4], [5] and, when given, in eps_dev / status_dev.
int enqueue_solve(ispa_stats* h, float lambda, float* delta_w, double* eps_dev, int32_t* status_dev) {
  if (!valid_handle(h)) return ISPA_ERR_STATE;
  if (!delta_w || !aligned16(delta_w)) return ISPA_ERR_INVALID_ARG;
  if (!(lambda >= 0.f) || isinf(lambda)) return ISPA_ERR_INVALID_ARG;
  if (((uintptr_t)eps_dev & 7u) || ((uintptr_t)status_dev & 3u)) return ISPA_ERR_INVALID_ARG;
  ispa::SolveWork w;
  w.L = (float*)(h->ws + h->lay.L);
  w.work = (float*)(h->ws + h->lay.W);
  w.dinv = (float*)(h->ws + h->lay.Dinv);
  w.status = (int*)(h->ws + h->lay.status);
  w.scalars = (double*)(h->ws + h->lay.scalars);
  w.eps_out = eps_dev;
  w.status_out = status_dev;
  const float* G = (const float*)(h->ws + h->lay.G);
  const float* C = (const float*)(h->ws + h->lay.C);
  return ispa::launch_solve(G, C, h->d_in, h->d_out, lambda, delta_w, w, h->stream) == hipSuccess ? ISPA_OK
                                                                                                   : ISPA_ERR_HIP;
}
}  // namespace

int ispa_solve_modulation(ispa_stats* h, float lambda, float* delta_w, double* eps_out) {
  const int st = enqueue_solve(h, lambda, delta_w, nullptr, nullptr);
  if (st != ISPA_OK) return st;
  // one copy of the scalars: [4] eps, [5] the status word
  double sc[6] = {0, 0, 0, 0, 0, 0};
  if (hipMemcpyAsync(sc, h->ws + h->lay.scalars, sizeof(sc), hipMemcpyDeviceToHost, h->stream) != hipSuccess)
    return ISPA_ERR_HIP;
  if (hipStreamSynchronize(h->stream) != hipSuccess) return ISPA_ERR_HIP;
  if (sc[5] != 0.0) return ISPA_ERR_NOT_SPD;
  if (eps_out) *eps_out = sc[4];
  return ISPA_OK;
}

int ispa_solve_modulation_async(ispa_stats* h, float lambda, float* delta_w, double* eps_dev, int32_t* status_dev) {
  return enqueue_solve(h, lambda, delta_w, eps_dev, status_dev);
}

int ispa_solve_lookahead_check(int32_t n_panels, int32_t n_cu) { return ispa::solve_lookahead_check(n_panels, n_cu); }

int ispa_solve_modulation_batch(ispa_stats* const* handles, int32_t n_layers, float lambda, float* delta_w,
                                double* eps_dev, int32_t* status_dev) {
  if (!handles || n_layers < 1 || n_layers > 4096) return ISPA_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n_layers; ++i)
    if (!valid_handle(handles[i])) return ISPA_ERR_STATE;
  const ispa_stats* h = handles[0];
  const int64_t stride = n_layers > 1 ? (int64_t)(handles[1]->ws - h->ws) : 0;
  if (n_layers > 1 && stride < (int64_t)h->lay.total) return ISPA_ERR_INVALID_ARG;
  for (int32_t i = 1; i < n_layers; ++i) {
    const ispa_stats* g = handles[i];
    if (g->d_in != h->d_in || g->d_out != h->d_out || g->max_rows != h->max_rows) return ISPA_ERR_INVALID_ARG;
    if (g->ws != h->ws + (size_t)i * (size_t)stride) return ISPA_ERR_INVALID_ARG;
  }
  if (!delta_w || !aligned16(delta_w)) return ISPA_ERR_INVALID_ARG;
  if (!(lambda >= 0.f) || isinf(lambda)) return ISPA_ERR_INVALID_ARG;
  if (((uintptr_t)eps_dev & 7u) || ((uintptr_t)status_dev & 3u)) return ISPA_ERR_INVALID_ARG;
  ispa::SolveWork w;
  w.L = (float*)(h->ws + h->lay.L);
  w.work = (float*)(h->ws + h->lay.W);
  w.dinv = (float*)(h->ws + h->lay.Dinv);
  w.status = (int*)(h->ws + h->lay.status);
  w.scalars = (double*)(h->ws + h->lay.scalars);
  w.eps_out = eps_dev;
  w.status_out = status_dev;
  w.n_layers = n_layers;
  w.ws_stride = stride;
  w.dw_stride = (int64_t)h->d_in * h->d_out * (int64_t)sizeof(float);
  const float* G = (const float*)(h->ws + h->lay.G);
  const float* C = (const float*)(h->ws + h->lay.C);
  return ispa::launch_solve(G, C, h->d_in, h->d_out, lambda, delta_w, w, h->stream) == hipSuccess ? ISPA_OK
                                                                                                   : ISPA_ERR_HIP;
}


int ispa_select_layers(const double* eps, int32_t n_layers, int32_t k, int32_t* selected) {
  if (!eps || n_layers < 0 || n_layers > (1 << 20) || k < 0 || k > n_layers || (k > 0 && !selected))
    return ISPA_ERR_INVALID_ARG;
  int32_t* idx = new (std::nothrow) int32_t[n_layers > 0 ? n_layers : 1];
  if (!idx) return ISPA_ERR_STATE;
  for (int32_t i = 0; i < n_layers; ++i) idx[i] = i;
  // ascending eps, NaN after every number, ties by layer index (stable sort)
  std::stable_sort(idx, idx + n_layers, [eps](int32_t a, int32_t b) {
    const double x = eps[a], y = eps[b];
    if (isnan(x)) return false;
    if (isnan(y)) return true;
    return x < y;
  });
  for (int32_t i = 0; i < k; ++i) selected[i] = idx[i];
  delete[] idx;
  return ISPA_OK;
}

int ispa_inject_modulation(void* weight, int32_t weight_dtype, int32_t transposed, const float* delta_w,
                           int32_t d_in, int32_t d_out, hipStream_t stream) {
  if (weight_dtype != ISPA_DTYPE_BF16 && weight_dtype != ISPA_DTYPE_F32) return ISPA_ERR_UNSUPPORTED;
  if (!weight || !delta_w) return ISPA_ERR_INVALID_ARG;
  if (d_in < 1 || d_out < 1 || d_in > 65536 || d_out > 65536) return ISPA_ERR_INVALID_ARG;
  const size_t esz = weight_dtype == ISPA_DTYPE_BF16 ? 2 : 4;
  if (((uintptr_t)weight % esz) || ((uintptr_t)delta_w & 3u)) return ISPA_ERR_INVALID_ARG;
  const size_t n = (size_t)d_in * d_out;
  const char* w0 = (const char*)weight;
  const char* d0 = (const char*)delta_w;
  if (w0 < d0 + n * 4 && d0 < w0 + n * esz) return ISPA_ERR_INVALID_ARG;
  return ispa::launch_inject(weight, weight_dtype == ISPA_DTYPE_BF16 ? 0 : 1, transposed != 0, delta_w, d_in, d_out,
                             stream) == hipSuccess
             ? ISPA_OK
             : ISPA_ERR_HIP;
}

int ispa_kv_evict(const void* k_cache, const void* v_cache, int64_t cache_len, int64_t window, int64_t sink_len,
                  int32_t hidden, void* k_ring, void* v_ring, int64_t* ring_rows, hipStream_t stream) {
  if (!k_cache || !v_cache || !k_ring || !v_ring) return ISPA_ERR_INVALID_ARG;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(k_ring) || !aligned16(v_ring))
    return ISPA_ERR_INVALID_ARG;
  if (hidden < 8 || hidden % 8 != 0 || hidden > (1 << 20)) return ISPA_ERR_INVALID_ARG;
  if (cache_len < 1 || cache_len > ((int64_t)1 << 31) || window < 1 || sink_len < 0) return ISPA_ERR_INVALID_ARG;
  if (k_ring == k_cache || v_ring == v_cache || k_ring == v_ring) return ISPA_ERR_INVALID_ARG;
  // local set of Eq. 7: sink rows [0, s'), window rows [max(N - w, s'), N)
  const int64_t N = cache_len;
  const int64_t s1 = sink_len < N ? sink_len : N;
  const int64_t lo = N - window > s1 ? N - window : s1;
  const int64_t src[2] = {0, lo}, dst[2] = {0, s1}, n[2] = {s1, N - lo};
  if (ring_rows) *ring_rows = s1 + (N - lo);
  return ispa::launch_kv_copy(k_cache, v_cache, k_ring, v_ring, (int64_t)hidden * 2, src, dst, n, 2, stream) ==
                 hipSuccess
             ? ISPA_OK
             : ISPA_ERR_HIP;
}

int ispa_kv_ring_append(void* k_ring, void* v_ring, int64_t sink_rows, int64_t window, int64_t head,
                        const void* k_new, const void* v_new, int64_t n_new, int32_t hidden, hipStream_t stream) {
  if (!k_ring || !v_ring || !k_new || !v_new) return ISPA_ERR_INVALID_ARG;
  if (!aligned16(k_ring) || !aligned16(v_ring) || !aligned16(k_new) || !aligned16(v_new)) return ISPA_ERR_INVALID_ARG;
  if (hidden < 8 || hidden % 8 != 0 || hidden > (1 << 20)) return ISPA_ERR_INVALID_ARG;
  if (sink_rows < 0 || window < 1 || head < 0 || n_new < 0 || window > ((int64_t)1 << 31)) return ISPA_ERR_INVALID_ARG;
  if (n_new == 0) return ISPA_OK;
  // new key r is window key number head + r, at ring row sink + (head + r) mod window;
  // only the last min(n_new, window) of them survive
  const int64_t m = n_new < window ? n_new : window;
  const int64_t p = (head + n_new - m) % window;
  const int64_t first = m < window - p ? m : window - p;
  const int64_t src[2] = {n_new - m, n_new - m + first}, dst[2] = {sink_rows + p, sink_rows};
  const int64_t n[2] = {first, m - first};
  return ispa::launch_kv_copy(k_new, v_new, k_ring, v_ring, (int64_t)hidden * 2, src, dst, n, 2, stream) ==
                 hipSuccess
             ? ISPA_OK
             : ISPA_ERR_HIP;
}


int ispa_project(const void* a, const void* weight, int64_t n_rows, int32_t d_in, int32_t d_out, void* y,
                 int32_t y_dtype, hipStream_t stream) {
  if (y_dtype != ISPA_DTYPE_BF16 && y_dtype != ISPA_DTYPE_F32) return ISPA_ERR_UNSUPPORTED;
  if (!a || !weight || !y) return ISPA_ERR_INVALID_ARG;
  if (!aligned16(a) || !aligned16(weight) || ((uintptr_t)y & 3u)) return ISPA_ERR_INVALID_ARG;
  if (n_rows < 1 || n_rows > ((int64_t)1 << 31) || d_in < 32 || d_in % 32 != 0 || d_in > 65536 || d_out < 1 ||
      d_out > 65536)
    return ISPA_ERR_INVALID_ARG;
  const size_t ybytes = (size_t)n_rows * d_out * (y_dtype == ISPA_DTYPE_BF16 ? 2 : 4);
  if (overlaps(y, ybytes, a, (size_t)n_rows * d_in * 2) || overlaps(y, ybytes, weight, (size_t)d_out * d_in * 2))
    return ISPA_ERR_INVALID_ARG;
  return ispa::launch_project(a, weight, n_rows, d_in, d_out, y, y_dtype == ISPA_DTYPE_BF16, ispa::attn_cu_count(),
                              stream) == hipSuccess
             ? ISPA_OK
             : ISPA_ERR_HIP;
}

int ispa_quantize_rows(const void* x, int32_t x_dtype, int64_t rows, int32_t cols, int8_t* q, float* scale,
                       hipStream_t stream) {
  if (x_dtype != ISPA_DTYPE_BF16 && x_dtype != ISPA_DTYPE_F32) return ISPA_ERR_UNSUPPORTED;
  if (!x || !q || !scale) return ISPA_ERR_INVALID_ARG;
  if (!aligned16(x) || ((uintptr_t)q & 7u) || ((uintptr_t)scale & 3u)) return ISPA_ERR_INVALID_ARG;
  if (rows < 1 || rows > ((int64_t)1 << 31) || cols < 8 || cols % 8 != 0) return ISPA_ERR_INVALID_ARG;
  const size_t xb = (size_t)rows * cols * (x_dtype == ISPA_DTYPE_F32 ? 4 : 2), qb = (size_t)rows * cols,
               sb = (size_t)rows * 4;
  if (overlaps(q, qb, x, xb) || overlaps(scale, sb, x, xb) || overlaps(q, qb, scale, sb)) return ISPA_ERR_INVALID_ARG;
  return ispa::launch_quantize_rows(x, x_dtype == ISPA_DTYPE_BF16, rows, cols, q, scale, stream) == hipSuccess
             ? ISPA_OK
             : ISPA_ERR_HIP;
}

int ispa_project_w8a8(const int8_t* q_a, const float* scale_a, const int8_t* q_w, const float* scale_w, int64_t n_rows,
                      int32_t d_in, int32_t d_out, void* y, int32_t y_dtype, hipStream_t stream) {
  if (y_dtype != ISPA_DTYPE_BF16 && y_dtype != ISPA_DTYPE_F32) return ISPA_ERR_UNSUPPORTED;
  if (!q_a || !scale_a || !q_w || !scale_w || !y) return ISPA_ERR_INVALID_ARG;
  if (!aligned16(q_a) || !aligned16(q_w) || ((uintptr_t)y & 3u) || ((uintptr_t)scale_a & 3u) ||
      ((uintptr_t)scale_w & 3u))
    return ISPA_ERR_INVALID_ARG;
  if (n_rows < 1 || n_rows > ((int64_t)1 << 31) || d_in < 64 || d_in % 64 != 0 || d_in > 65536 || d_out < 1 ||
      d_out > 65536)
    return ISPA_ERR_INVALID_ARG;
  const size_t ybytes = (size_t)n_rows * d_out * (y_dtype == ISPA_DTYPE_BF16 ? 2 : 4);
  if (overlaps(y, ybytes, q_a, (size_t)n_rows * d_in) || overlaps(y, ybytes, q_w, (size_t)d_out * d_in) ||
      overlaps(y, ybytes, scale_a, (size_t)n_rows * 4) || overlaps(y, ybytes, scale_w, (size_t)d_out * 4))
    return ISPA_ERR_INVALID_ARG;
  return ispa::launch_project_w8a8(q_a, scale_a, q_w, scale_w, n_rows, d_in, d_out, y, y_dtype == ISPA_DTYPE_BF16,
                                   ispa::attn_cu_count(), stream) == hipSuccess
             ? ISPA_OK
             : ISPA_ERR_HIP;
}

}  // extern "C"
