// C-ABI entry points: argument validation, host-side coordinate shift,
// workspace sizing, kernel tracing and error reporting.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <map>
#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "cs_common.h"

namespace cs {

static thread_local std::string t_error;

void set_error(const std::string& msg) { t_error = msg; }

cs_status fail(cs_status code, const std::string& msg) {
  t_error = msg;
  return code;
}

cs_status check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(CS_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return CS_OK;
}

cs_status check_grid(int64_t gx, int64_t gy, int64_t gz, int threads, const char* what) {
  if (gx >= (int64_t(1) << 31) || gx * threads >= (int64_t(1) << 32) || gy > 65535 || gz > 65535)
    return fail(CS_ERR_UNSUPPORTED, std::string(what) + ": the cache is too large for one launch (grid " +
                                        std::to_string(gx) + " x " + std::to_string(gy) + " x " + std::to_string(gz) + ")");
  return CS_OK;
}

// ------------------------------------------------------------------ tracing
namespace {
struct Pending {
  std::string name;
  hipEvent_t a, b;
};
struct Acc {
  int64_t launches = 0;
  double ms = 0.0;
};
// Tracing state is shared by every thread that calls the library; g_trace_mu
// guards all of it.
std::mutex g_trace_mu;
bool g_trace_on = false;
std::vector<Pending> g_pending;
std::vector<std::pair<std::string, Acc>> g_acc;
std::vector<hipEvent_t> g_pool;
std::vector<std::string> g_trace_names;  // kernels traced while tracing is on (empty: all)

// set while a call that must not allocate enqueues on this thread
thread_local bool t_trace_suppressed = false;
bool trace_suppressed() { return t_trace_suppressed; }

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

TraceScope::TraceScope(const char* n, hipStream_t s) : name(n), stream(s), a(nullptr), b(nullptr) {
  if (trace_suppressed()) return;
  std::lock_guard<std::mutex> lk(g_trace_mu);
  if (!g_trace_on) return;
  if (!g_trace_names.empty() &&
      std::find(g_trace_names.begin(), g_trace_names.end(), n) == g_trace_names.end())
    return;
  a = take_event();
  b = a ? take_event() : nullptr;
  if (!b) {
    if (a) g_pool.push_back(a);
    a = nullptr;
  }
}

TraceScope::~TraceScope() {
  if (!a) return;
  std::lock_guard<std::mutex> lk(g_trace_mu);
  g_pending.push_back({name, a, b});
}

// ------------------------------------------------------------------ geometry
cs_status check_geometry(const cs_geometry* g, Geo* o) {
  if (!g) return fail(CS_ERR_INVALID_ARGUMENT, "geometry is NULL");
  if (g->n_layers < 1) return fail(CS_ERR_INVALID_ARGUMENT, "n_layers must be >= 1");
  if (g->n_q_heads < 1 || g->n_kv_heads < 1)
    return fail(CS_ERR_INVALID_ARGUMENT, "head counts must be >= 1");
  if (g->n_q_heads % g->n_kv_heads)
    return fail(CS_ERR_INVALID_ARGUMENT, "n_q_heads must be a multiple of n_kv_heads");
  if (g->head_dim < 2 || g->head_dim > 512 || (g->head_dim & 1))
    return fail(CS_ERR_INVALID_ARGUMENT, "head_dim must be even and in [2, 512]");
  if (g->sections[0] < 0 || g->sections[1] < 0 || g->sections[2] < 0 ||
      (int64_t)g->sections[0] + g->sections[1] + g->sections[2] != g->head_dim / 2)
    return fail(CS_ERR_INVALID_ARGUMENT, "sections must be >= 0 and sum to head_dim/2");
  if (g->dtype != CS_F32 && g->dtype != CS_BF16)
    return fail(CS_ERR_INVALID_ARGUMENT, "dtype must be CS_F32 or CS_BF16");
  if (!g->inv_freq && !(g->rope_base > 0.0 && isfinite(g->rope_base)))
    return fail(CS_ERR_INVALID_ARGUMENT, "rope_base must be finite and > 0 when inv_freq is NULL");
  if (g->n_tokens < 1 || g->n_tokens >= (int64_t(1) << 31))
    return fail(CS_ERR_INVALID_ARGUMENT, "n_tokens must be in [1, 2^31)");
  if (g->n_chunks < 1) return fail(CS_ERR_INVALID_ARGUMENT, "n_chunks must be >= 1");
  if (!g->chunk_start) return fail(CS_ERR_INVALID_ARGUMENT, "chunk_start is NULL");
  if (g->chunk_start[0] != 0) return fail(CS_ERR_INVALID_ARGUMENT, "chunk_start[0] must be 0");
  for (int c = 0; c < g->n_chunks; ++c)
    if (g->chunk_start[c + 1] <= g->chunk_start[c])
      return fail(CS_ERR_INVALID_ARGUMENT, "chunk_start must be strictly increasing");
  if (g->chunk_start[g->n_chunks] != g->n_tokens)
    return fail(CS_ERR_INVALID_ARGUMENT, "chunk_start[n_chunks] must equal n_tokens");
  o->L = g->n_layers;
  o->Hq = g->n_q_heads;
  o->Hkv = g->n_kv_heads;
  o->G = g->n_q_heads / g->n_kv_heads;
  o->D = g->head_dim;
  o->P = g->head_dim / 2;
  for (int i = 0; i < 3; ++i) o->sec[i] = g->sections[i];
  o->dtype = g->dtype;
  o->esize = g->dtype == CS_BF16 ? 2 : 4;
  o->T = g->n_tokens;
  o->N = g->n_chunks;
  o->cs = g->chunk_start;
  o->cs1 = g->n_chunks >= 2 ? g->chunk_start[1] : g->n_tokens;
  o->n = o->T - o->cs1;
  return CS_OK;
}

int64_t n_select(double rho, int64_t n) {
  if (rho == 0.0 || n == 0) return 0;
  int64_t k = (int64_t)ceil(rho * (double)n - 1e-9);
  if (k < 0) k = 0;
  return k > n ? n : k;
}

static size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

static CacheView flat_view(void* k, void* v) {
  CacheView cv;
  cv.k = k;
  cv.v = v;
  return cv;
}

// A paged cache: n_chunks device pointers per tensor (v_chunks only when
// the call writes or reads values).
static cs_status paged_view(const Geo& g, void* const* k_chunks, void* const* v_chunks, bool need_v,
                            CacheView* cv) {
  const int cap = g.dtype == CS_BF16 && g.D == 128 ? kMaxPages : kMaxPagesGeneric;
  if (g.N > cap)
    return fail(CS_ERR_UNSUPPORTED, "a paged cache holds at most " + std::to_string(cap) + " chunks");
  if (!k_chunks || (need_v && !v_chunks)) return fail(CS_ERR_INVALID_ARGUMENT, "chunk pointer array is NULL");
  for (int c = 0; c < g.N; ++c)
    if (!k_chunks[c] || (need_v && !v_chunks[c]))
      return fail(CS_ERR_INVALID_ARGUMENT, "chunk " + std::to_string(c) + " has a NULL buffer");
  cv->paged = true;
  cv->k_chunks = k_chunks;
  cv->v_chunks = need_v ? v_chunks : nullptr;
  return CS_OK;
}

static cs_status theta_table(const cs_geometry* gp, const Geo& g, std::vector<double>* theta) {
  theta->resize(g.P);
  for (int i = 0; i < g.P; ++i)
    (*theta)[i] = gp->inv_freq ? gp->inv_freq[i] : pow(gp->rope_base, -2.0 * i / (double)g.D);
  for (int i = 0; i < g.P; ++i)
    if (!isfinite((*theta)[i])) return fail(CS_ERR_INVALID_ARGUMENT, "inv_freq holds a non-finite value");
  return CS_OK;
}

// ------------------------------------------------------------------ calls on either layout
static cs_status rebase_k(const cs_geometry* gp, const Geo& g, const CacheView& cv, const int32_t* chunk_offsets,
                          const int32_t* local_coords, int32_t* global_coords, void* stream) {
  if (!chunk_offsets) return fail(CS_ERR_INVALID_ARGUMENT, "chunk_offsets is NULL");
  if (global_coords && !local_coords)
    return fail(CS_ERR_INVALID_ARGUMENT, "global_coords needs local_coords");
  std::vector<double> theta;
  cs_status st = theta_table(gp, g, &theta);
  if (!st) st = launch_rebase(g, cv, chunk_offsets, theta.data(), (hipStream_t)stream, true);
  if (st) return st;
  // Coordinate shift (host): p' = p + Delta_c for every token of chunk c.
  if (global_coords) {
    for (int c = 0; c < g.N; ++c)
      for (int64_t t = g.cs[c]; t < g.cs[c + 1]; ++t)
        for (int a = 0; a < 3; ++a)
          global_coords[3 * t + a] = local_coords[3 * t + a] + chunk_offsets[3 * c + a];
  }
  return launch_rebase(g, cv, chunk_offsets, theta.data(), (hipStream_t)stream);
}

static cs_status rebase_k_tokens(const cs_geometry* gp, const Geo& g, const CacheView& cv,
                                 const int32_t* token_offsets, void* stream) {
  if (!token_offsets) return fail(CS_ERR_INVALID_ARGUMENT, "token_offsets is NULL");
  std::vector<double> theta;
  cs_status st = theta_table(gp, g, &theta);
  if (!st) st = launch_rebase_tokens(g, cv, token_offsets, theta.data(), (hipStream_t)stream, true);
  if (st) return st;
  return launch_rebase_tokens(g, cv, token_offsets, theta.data(), (hipStream_t)stream);
}

static cs_status score_topk(const Geo& g, const CacheView& cv, int32_t score_layer, const void* k_fresh, double rho,
                            float* scores, int32_t* sel_idx, int64_t* n_sel, void* workspace, size_t workspace_bytes,
                            void* stream) {
  if (!n_sel) return fail(CS_ERR_INVALID_ARGUMENT, "n_sel is NULL");
  if (!(rho >= 0.0 && rho <= 1.0)) return fail(CS_ERR_INVALID_ARGUMENT, "rho must lie in [0, 1]");
  if (score_layer < 0 || score_layer >= g.L)
    return fail(CS_ERR_INVALID_ARGUMENT, "score_layer out of range");
  int64_t k = n_select(rho, g.n);
  if (g.n > 0) {
    if ((!cv.paged && !cv.k) || !k_fresh) return fail(CS_ERR_INVALID_ARGUMENT, "k_cache or k_fresh is NULL");
    if (k > 0 && !sel_idx) return fail(CS_ERR_INVALID_ARGUMENT, "sel_idx is NULL");
    if (!scores) {
      size_t need = align_up((size_t)g.n * sizeof(float), 256);
      if (!workspace || workspace_bytes < need)
        return fail(CS_ERR_WORKSPACE_TOO_SMALL, "workspace must hold n float32 scores when scores is NULL");
      scores = (float*)workspace;
    }
  }
  if (g.n > 0) {
    cs_status st = launch_score_select(g, cv, score_layer, k_fresh, scores, sel_idx, k, (hipStream_t)stream, true);
    if (st) return st;
  }
  *n_sel = k;
  if (g.n == 0) return CS_OK;
  return launch_score_select(g, cv, score_layer, k_fresh, scores, sel_idx, k, (hipStream_t)stream);
}

// ------------------------------------------------------------------ debug validation
// With the environment variable CS_DEBUG_VALIDATE=1 the attention entry points
// check the selection's unchecked precondition on the device (strictly
// ascending, every index in [s_1, T)) before enqueuing anything else, at the
// cost of a synchronisation of the stream.  The violation flag is one word of
// device memory per GPU, so validated calls must not overlap.
static __device__ unsigned g_sel_bad;

__global__ __launch_bounds__(256) void validate_sel(const int32_t* __restrict__ sel, int64_t n_sel, int64_t lo,
                                                    int64_t hi) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_sel) return;
  const int64_t v = sel[i];
  unsigned bad = 0;
  if (v < lo || v >= hi) bad |= 1u;
  if (i > 0 && (int64_t)sel[i - 1] >= v) bad |= 2u;
  if (bad) atomicOr(&g_sel_bad, bad);
}

static bool debug_validate() {
  const char* e = getenv("CS_DEBUG_VALIDATE");
  return e && e[0] == '1' && e[1] == 0;
}

static cs_status check_selection(const Geo& g, const int32_t* sel, int64_t n_sel, hipStream_t s) {
  if (n_sel <= 0) return CS_OK;
  const int64_t blocks = (n_sel + 255) / 256;
  cs_status st = check_grid(blocks, 1, 1, 256, "selection check");
  if (st) return st;
  unsigned flag = 0;
  if (hipMemcpyToSymbolAsync(HIP_SYMBOL(g_sel_bad), &flag, sizeof flag, 0, hipMemcpyHostToDevice, s) != hipSuccess)
    return fail(CS_ERR_HIP, "selection check: clearing the flag failed");
  hipLaunchKernelGGL(validate_sel, dim3((unsigned)blocks), dim3(256), 0, s, sel, n_sel, g.cs1, g.T);
  st = check_launch("selection check launch");
  if (st) return st;
  if (hipMemcpyFromSymbolAsync(&flag, HIP_SYMBOL(g_sel_bad), sizeof flag, 0, hipMemcpyDeviceToHost, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess)
    return fail(CS_ERR_HIP, "selection check: reading the flag failed");
  if (flag & 1u) return fail(CS_ERR_INVALID_ARGUMENT, "sel_idx holds an index outside [chunk_start[1], n_tokens)");
  if (flag & 2u) return fail(CS_ERR_INVALID_ARGUMENT, "sel_idx is not strictly ascending");
  return CS_OK;
}

static size_t attn_ws_bytes(const AttnPlan& p, int layers) {
  return p.mfma ? p.ws_fixed_bytes + p.ws_bytes_per_layer * (size_t)layers : 0;
}

// Argument checks of the attention calls that need no HIP runtime call.
static cs_status attend_scatter_check(const Geo& g, const CacheView& cv, const int32_t* sel_idx,
                                      const void* q_fresh, const void* k_fresh, const void* v_fresh, void* out,
                                      const AttnPlan& p) {
  if (!sel_idx || !q_fresh || !k_fresh || !v_fresh || !out)
    return fail(CS_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  if (cv.paged && p.mfma && !chunks_tile_aligned(g))
    return fail(CS_ERR_UNSUPPORTED, "a paged cache needs chunk starts that are multiples of 64 on the MFMA path");
  return CS_OK;
}

// Scatter + attention with a plan whose workspace (attn_ws_bytes) is at
// `workspace`; every argument has been checked.
static cs_status attend_scatter_planned(const Geo& g, const CacheView& cv, int32_t layer_begin, int32_t layer_end,
                                        const int32_t* sel_idx, int64_t n_sel, const void* q_fresh,
                                        const void* k_fresh, const void* v_fresh, void* out, float* lse,
                                        const AttnPlan& p, void* workspace, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  // the scatter of the fresh rows runs inside the attention's first launch
  const ScatterJob job{k_fresh, v_fresh};
  for (int pass = 0; pass < 2; ++pass) {  // sizes of every launch first, then the launches
    if (pass == 1 && debug_validate()) {
      cs_status st = check_selection(g, sel_idx, n_sel, s);
      if (st) return st;
    }
    cs_status st = launch_attention(g, p, cv, layer_begin, layer_end, sel_idx, n_sel, q_fresh, false, out, lse,
                                    workspace, s, pass == 0, &job);
    if (st) return st;
  }
  return CS_OK;
}

static cs_status attend_scatter(const Geo& g, const CacheView& cv, int32_t layer_begin, int32_t layer_end,
                                const int32_t* sel_idx, int64_t n_sel, const void* q_fresh, const void* k_fresh,
                                const void* v_fresh, void* out, float* lse, void* workspace, size_t workspace_bytes,
                                void* stream) {
  const AttnPlan p = plan_attention(g, n_sel, layer_end - layer_begin);
  cs_status st = attend_scatter_check(g, cv, sel_idx, q_fresh, k_fresh, v_fresh, out, p);
  if (st) return st;
  const size_t need = attn_ws_bytes(p, layer_end - layer_begin);
  if (need && (!workspace || workspace_bytes < need))
    return fail(CS_ERR_WORKSPACE_TOO_SMALL,
                "workspace smaller than selective_attend_scatter_workspace() (" + std::to_string(need) +
                    " bytes)");
  return attend_scatter_planned(g, cv, layer_begin, layer_end, sel_idx, n_sel, q_fresh, k_fresh, v_fresh, out, lse,
                                p, workspace, stream);
}

// ------------------------------------------------------------------ no-allocation variant
// selective_attend_scatter_noalloc keeps the attention's plan and partials in
// this array instead of a caller workspace.  Each GPU the library runs on
// holds its own copy until the process ends; host code reaches it only through
// the device address hipGetSymbolAddress returns for the current device (the
// array's name in host code is not a device address).  The kernels write the
// plan, including its queue counters, before anything reads it, so no call
// needs the array cleared; calls that overlap on one GPU race on it.
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];
constexpr int kScratchDevices = 256;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kScratchDevices];

static cs_status scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return fail(CS_ERR_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kScratchDevices) return fail(CS_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(CS_ERR_HIP, std::string("hipGetSymbolAddress of the scratch array failed: ") + hipGetErrorString(e));
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return CS_OK;
}

// The library's plan, with its partial slots cut down until plan and
// partials fit in the scratch array (longer key pieces, or none).
static cs_status noalloc_plan(const Geo& g, int64_t n_sel, int layers, AttnPlan* out) {
  AttnPlan p = plan_attention(g, n_sel, layers);
  if (attn_ws_bytes(p, layers) > kNoAllocScratchBytes && p.part_cap > 0) {
    const size_t slot = p.ws_bytes_per_layer / (size_t)p.part_cap;
    const size_t room = p.ws_fixed_bytes < kNoAllocScratchBytes ? kNoAllocScratchBytes - p.ws_fixed_bytes : 0;
    p = plan_attention(g, n_sel, layers, (int64_t)(room / (slot * (size_t)layers)));
  }
  const size_t need = attn_ws_bytes(p, layers);
  if (need > kNoAllocScratchBytes)
    return fail(CS_ERR_UNSUPPORTED, "selective_attend_scatter_noalloc: the plan needs " + std::to_string(need) +
                                        " bytes, more than its " + std::to_string(kNoAllocScratchBytes) +
                                        "-byte scratch array");
  *out = p;
  return CS_OK;
}

// Kernel tracing creates events; calls that must not allocate turn it off on
// their thread while they enqueue.
struct TraceSuppress {
  bool prev;
  TraceSuppress() : prev(t_trace_suppressed) { t_trace_suppressed = true; }
  ~TraceSuppress() { t_trace_suppressed = prev; }
};

// Workspace of the fused-rotary variant: the attention's, then, on the MFMA
// path (bf16, head_dim 128), the cos/sin table of the selected tokens
// [n_sel][D/2] float2 (the attention rotates the queries as it loads them),
// elsewhere the rotated queries [layers in call][H_q][n_sel][D].
static size_t rope_ws(const Geo& g, const AttnPlan& p, int64_t n_sel, int layers, size_t* att_bytes) {
  const size_t att = p.mfma && n_sel > 0 && layers > 0 ? p.ws_fixed_bytes + p.ws_bytes_per_layer * (size_t)layers : 0;
  *att_bytes = align_up(att, 256);
  if (p.mfma) return *att_bytes + rope_table_bytes(n_sel);
  return *att_bytes + (size_t)layers * g.Hq * n_sel * g.D * g.esize;
}

static cs_status attend_scatter_rope(const cs_geometry* gp, const Geo& g, const CacheView& cv, int32_t layer_begin,
                                     int32_t layer_end, const int32_t* sel_idx, int64_t n_sel, const void* q_pre,
                                     const void* k_pre, const void* v_fresh, const int32_t* coords, void* out,
                                     float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  if (!sel_idx || !q_pre || !k_pre || !v_fresh || !coords || !out)
    return fail(CS_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  std::vector<double> theta;
  cs_status st = theta_table(gp, g, &theta);
  if (st) return st;
  const int layers = layer_end - layer_begin;
  AttnPlan p = plan_attention(g, n_sel, layers);
  size_t att = 0;
  const size_t need = rope_ws(g, p, n_sel, layers, &att);
  if (!workspace || workspace_bytes < need)
    return fail(CS_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than selective_attend_scatter_rope_workspace() (" +
                                                std::to_string(need) + " bytes)");
  if (cv.paged && p.mfma && !chunks_tile_aligned(g))
    return fail(CS_ERR_UNSUPPORTED, "a paged cache needs chunk starts that are multiples of 64 on the MFMA path");
  hipStream_t s = (hipStream_t)stream;
  void* extra = (char*)workspace + att;  // the cos/sin table (MFMA path) or the rotated queries
  const RopeJob rope{k_pre, v_fresh, coords, theta.data(), extra};
  for (int pass = 0; pass < 2; ++pass) {  // sizes of every launch first, then the launches
    const bool check = pass == 0;
    if (!check && debug_validate()) {
      st = check_selection(g, sel_idx, n_sel, s);
      if (st) return st;
    }
    if (p.mfma) {  // the rotations run inside the attention's two launches
      st = launch_attention(g, p, cv, layer_begin, layer_end, sel_idx, n_sel, q_pre, false, out, lse, workspace, s,
                            check, nullptr, &rope);
    } else {
      st = launch_rope_scatter(g, cv, layer_begin, layer_end, sel_idx, n_sel, q_pre, k_pre, v_fresh, coords,
                               theta.data(), extra, s, check);
      if (!st)
        st = launch_attention(g, p, cv, layer_begin, layer_end, sel_idx, n_sel, extra, true, out, lse, workspace, s,
                              check);
    }
    if (st) return st;
  }
  return CS_OK;
}

}  // namespace cs

using namespace cs;

// ====================================================================== exports
extern "C" {

const char* cs_last_error(void) { return t_error.c_str(); }

cs_status compose_rebase_k(const cs_geometry* gp, void* k_cache, const int32_t* chunk_offsets,
                           const int32_t* local_coords, int32_t* global_coords, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  if (!k_cache) return fail(CS_ERR_INVALID_ARGUMENT, "k_cache is NULL");
  return rebase_k(gp, g, flat_view(k_cache, nullptr), chunk_offsets, local_coords, global_coords, stream);
}

cs_status compose_rebase_k_paged(const cs_geometry* gp, void* const* k_chunks, const int32_t* chunk_offsets,
                                 const int32_t* local_coords, int32_t* global_coords, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  CacheView cv;
  st = paged_view(g, k_chunks, nullptr, false, &cv);
  if (st) return st;
  return rebase_k(gp, g, cv, chunk_offsets, local_coords, global_coords, stream);
}

// Three events, created on first use and kept: the call's start on the
// compute stream (the copies wait for the work enqueued before the call), the
// keys' arrival on the copy stream (the re-basing waits for it) and the last
// copy (the compute stream waits for it).  A wait takes the event's record at
// the time it is enqueued, so a later call may record the same events again.
static std::mutex g_load_mu;
static hipEvent_t g_load_events[3];

cs_status compose_load_rebase_k_paged(const cs_geometry* gp, void* const* k_chunks, void* const* v_chunks,
                                      const void* const* k_host, const void* const* v_host,
                                      const int32_t* chunk_offsets, void* copy_stream, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  CacheView cv;
  st = paged_view(g, k_chunks, v_chunks, true, &cv);
  if (st) return st;
  if (!k_host || !v_host) return fail(CS_ERR_INVALID_ARGUMENT, "host chunk pointer array is NULL");
  for (int c = 0; c < g.N; ++c)
    if (!k_host[c] || !v_host[c])
      return fail(CS_ERR_INVALID_ARGUMENT, "host chunk " + std::to_string(c) + " is NULL");
  if (!chunk_offsets) return fail(CS_ERR_INVALID_ARGUMENT, "chunk_offsets is NULL");
  std::vector<double> theta;
  st = theta_table(gp, g, &theta);
  if (!st) st = launch_rebase(g, cv, chunk_offsets, theta.data(), (hipStream_t)stream, true);
  if (st) return st;
  const hipStream_t s = (hipStream_t)stream;
  const hipStream_t cps = copy_stream ? (hipStream_t)copy_stream : s;
  const bool two = cps != s;
  std::lock_guard<std::mutex> lk(g_load_mu);  // (the events are shared by every caller)
  if (two) {
    for (hipEvent_t& e : g_load_events)
      if (!e && hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess)
        return fail(CS_ERR_HIP, "hipEventCreateWithFlags failed");
    if (hipEventRecord(g_load_events[0], s) != hipSuccess || hipStreamWaitEvent(cps, g_load_events[0], 0) != hipSuccess)
      return fail(CS_ERR_HIP, "ordering the copies after the stream's earlier work failed");
  }
  auto copy = [&](void* const* dst, const void* const* src, const char* what) -> cs_status {
    for (int c = 0; c < g.N; ++c) {
      const size_t bytes = (size_t)g.L * g.Hkv * (size_t)(g.cs[c + 1] - g.cs[c]) * g.D * g.esize;
      if (hipMemcpyAsync(dst[c], src[c], bytes, hipMemcpyHostToDevice, cps) != hipSuccess)
        return fail(CS_ERR_HIP, "hipMemcpyAsync of chunk " + std::to_string(c) + "'s " + what + " failed");
    }
    return CS_OK;
  };
  // every chunk's keys, then their re-basing on the compute stream while the
  // values follow on the copy stream
  st = copy(k_chunks, k_host, "keys");
  if (st) return st;
  if (two && (hipEventRecord(g_load_events[1], cps) != hipSuccess || hipStreamWaitEvent(s, g_load_events[1], 0) != hipSuccess))
    return fail(CS_ERR_HIP, "ordering the re-basing after the keys' copies failed");
  st = launch_rebase(g, cv, chunk_offsets, theta.data(), s);
  if (st) return st;
  st = copy(v_chunks, v_host, "values");
  if (st) return st;
  if (two && (hipEventRecord(g_load_events[2], cps) != hipSuccess || hipStreamWaitEvent(s, g_load_events[2], 0) != hipSuccess))
    return fail(CS_ERR_HIP, "ordering the stream after the last copy failed");
  return check_launch("load and re-base");
}

cs_status compose_rebase_k_tokens(const cs_geometry* gp, void* k_cache, const int32_t* token_offsets,
                                  void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  if (!k_cache) return fail(CS_ERR_INVALID_ARGUMENT, "k_cache is NULL");
  return rebase_k_tokens(gp, g, flat_view(k_cache, nullptr), token_offsets, stream);
}

cs_status compose_rebase_k_tokens_paged(const cs_geometry* gp, void* const* k_chunks, const int32_t* token_offsets,
                                        void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  CacheView cv;
  st = paged_view(g, k_chunks, nullptr, false, &cv);
  if (st) return st;
  return rebase_k_tokens(gp, g, cv, token_offsets, stream);
}

cs_status score_deviation_topk_workspace(const cs_geometry* gp, size_t* bytes) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  if (!bytes) return fail(CS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  *bytes = align_up((size_t)g.n * sizeof(float), 256);
  return CS_OK;
}

cs_status score_deviation_topk(const cs_geometry* gp, const void* k_cache, int32_t score_layer,
                               const void* k_fresh, double rho, float* scores, int32_t* sel_idx,
                               int64_t* n_sel, void* workspace, size_t workspace_bytes,
                               void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  return score_topk(g, flat_view((void*)k_cache, nullptr), score_layer, k_fresh, rho, scores, sel_idx, n_sel,
                    workspace, workspace_bytes, stream);
}

cs_status score_deviation_topk_paged(const cs_geometry* gp, void* const* k_chunks, int32_t score_layer,
                                     const void* k_fresh, double rho, float* scores, int32_t* sel_idx,
                                     int64_t* n_sel, void* workspace, size_t workspace_bytes, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  CacheView cv;
  st = paged_view(g, k_chunks, nullptr, false, &cv);
  if (st) return st;
  return score_topk(g, cv, score_layer, k_fresh, rho, scores, sel_idx, n_sel, workspace, workspace_bytes, stream);
}

cs_status selective_attend_scatter_workspace(const cs_geometry* gp, int64_t n_sel,
                                             int32_t n_layers_per_call, size_t* bytes) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  if (!bytes) return fail(CS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  if (n_sel < 0 || n_sel > g.n) return fail(CS_ERR_INVALID_ARGUMENT, "n_sel must be in [0, n]");
  if (n_layers_per_call < 0 || n_layers_per_call > g.L)
    return fail(CS_ERR_INVALID_ARGUMENT, "n_layers_per_call must be in [0, n_layers]");
  AttnPlan p = plan_attention(g, n_sel, n_layers_per_call);
  *bytes = n_layers_per_call > 0 && p.mfma && n_sel > 0
               ? p.ws_fixed_bytes + p.ws_bytes_per_layer * (size_t)n_layers_per_call
               : 0;
  return CS_OK;
}

static cs_status check_layers(const Geo& g, int32_t layer_begin, int32_t layer_end, int64_t n_sel) {
  if (layer_begin < 0 || layer_end < layer_begin || layer_end > g.L)
    return fail(CS_ERR_INVALID_ARGUMENT, "need 0 <= layer_begin <= layer_end <= n_layers");
  if (n_sel < 0 || n_sel > g.n) return fail(CS_ERR_INVALID_ARGUMENT, "n_sel must be in [0, n]");
  return CS_OK;
}

cs_status selective_attend_scatter(const cs_geometry* gp, void* k_cache, void* v_cache,
                                   int32_t layer_begin, int32_t layer_end, const int32_t* sel_idx,
                                   int64_t n_sel, const void* q_fresh, const void* k_fresh,
                                   const void* v_fresh, void* out, float* lse, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (!st) st = check_layers(g, layer_begin, layer_end, n_sel);
  if (st) return st;
  if (n_sel == 0 || layer_end == layer_begin) return CS_OK;
  if (!k_cache || !v_cache) return fail(CS_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  return attend_scatter(g, flat_view(k_cache, v_cache), layer_begin, layer_end, sel_idx, n_sel, q_fresh, k_fresh,
                        v_fresh, out, lse, workspace, workspace_bytes, stream);
}

cs_status selective_attend_scatter_noalloc(const cs_geometry* gp, void* k_cache, void* v_cache,
                                           int32_t layer_begin, int32_t layer_end, const int32_t* sel_idx,
                                           int64_t n_sel, const void* q_fresh, const void* k_fresh,
                                           const void* v_fresh, void* out, float* lse, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (!st) st = check_layers(g, layer_begin, layer_end, n_sel);
  if (st) return st;
  if (n_sel == 0 || layer_end == layer_begin) return CS_OK;
  if (!k_cache || !v_cache) return fail(CS_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  const CacheView cv = flat_view(k_cache, v_cache);
  AttnPlan p;
  st = noalloc_plan(g, n_sel, layer_end - layer_begin, &p);
  if (!st) st = attend_scatter_check(g, cv, sel_idx, q_fresh, k_fresh, v_fresh, out, p);
  if (st) return st;
  void* ws = nullptr;
  if (p.mfma) {
    st = scratch_address(&ws);
    if (st) return st;
  }
  TraceSuppress no_trace;
  return attend_scatter_planned(g, cv, layer_begin, layer_end, sel_idx, n_sel, q_fresh, k_fresh, v_fresh, out, lse,
                                p, ws, stream);
}

cs_status selective_attend_scatter_paged(const cs_geometry* gp, void* const* k_chunks, void* const* v_chunks,
                                         int32_t layer_begin, int32_t layer_end, const int32_t* sel_idx,
                                         int64_t n_sel, const void* q_fresh, const void* k_fresh,
                                         const void* v_fresh, void* out, float* lse, void* workspace,
                                         size_t workspace_bytes, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (!st) st = check_layers(g, layer_begin, layer_end, n_sel);
  if (st) return st;
  if (n_sel == 0 || layer_end == layer_begin) return CS_OK;
  CacheView cv;
  st = paged_view(g, k_chunks, v_chunks, true, &cv);
  if (st) return st;
  return attend_scatter(g, cv, layer_begin, layer_end, sel_idx, n_sel, q_fresh, k_fresh, v_fresh, out, lse,
                        workspace, workspace_bytes, stream);
}

cs_status selective_attend_scatter_rope_workspace(const cs_geometry* gp, int64_t n_sel, int32_t n_layers_per_call,
                                                  size_t* bytes) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (st) return st;
  if (!bytes) return fail(CS_ERR_INVALID_ARGUMENT, "bytes is NULL");
  if (n_sel < 0 || n_sel > g.n) return fail(CS_ERR_INVALID_ARGUMENT, "n_sel must be in [0, n]");
  if (n_layers_per_call < 0 || n_layers_per_call > g.L)
    return fail(CS_ERR_INVALID_ARGUMENT, "n_layers_per_call must be in [0, n_layers]");
  AttnPlan p = plan_attention(g, n_sel, n_layers_per_call);
  size_t att = 0;
  *bytes = n_sel > 0 && n_layers_per_call > 0 ? rope_ws(g, p, n_sel, n_layers_per_call, &att) : 0;
  return CS_OK;
}

cs_status selective_attend_scatter_rope(const cs_geometry* gp, void* k_cache, void* v_cache, int32_t layer_begin,
                                        int32_t layer_end, const int32_t* sel_idx, int64_t n_sel,
                                        const void* q_pre, const void* k_pre, const void* v_fresh,
                                        const int32_t* coords, void* out, float* lse, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (!st) st = check_layers(g, layer_begin, layer_end, n_sel);
  if (st) return st;
  if (n_sel == 0 || layer_end == layer_begin) return CS_OK;
  if (!k_cache || !v_cache) return fail(CS_ERR_INVALID_ARGUMENT, "a required device pointer is NULL");
  return attend_scatter_rope(gp, g, flat_view(k_cache, v_cache), layer_begin, layer_end, sel_idx, n_sel, q_pre,
                             k_pre, v_fresh, coords, out, lse, workspace, workspace_bytes, stream);
}

cs_status selective_attend_scatter_rope_paged(const cs_geometry* gp, void* const* k_chunks, void* const* v_chunks,
                                              int32_t layer_begin, int32_t layer_end, const int32_t* sel_idx,
                                              int64_t n_sel, const void* q_pre, const void* k_pre,
                                              const void* v_fresh, const int32_t* coords, void* out, float* lse,
                                              void* workspace, size_t workspace_bytes, void* stream) {
  Geo g;
  cs_status st = check_geometry(gp, &g);
  if (!st) st = check_layers(g, layer_begin, layer_end, n_sel);
  if (st) return st;
  if (n_sel == 0 || layer_end == layer_begin) return CS_OK;
  CacheView cv;
  st = paged_view(g, k_chunks, v_chunks, true, &cv);
  if (st) return st;
  return attend_scatter_rope(gp, g, cv, layer_begin, layer_end, sel_idx, n_sel, q_pre, k_pre, v_fresh, coords, out,
                             lse, workspace, workspace_bytes, stream);
}

// ------------------------------------------------------------------ tracing exports
cs_status cs_trace_enable(int32_t on) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  g_trace_on = on != 0;
  return CS_OK;
}

cs_status cs_trace_only(const char* names) {
  std::vector<std::string> list;
  if (names) {
    std::string cur;
    for (const char* c = names;; ++c) {
      if (*c == ',' || *c == 0) {
        if (!cur.empty()) list.push_back(cur);
        cur.clear();
        if (*c == 0) break;
      } else {
        cur += *c;
      }
    }
  }
  std::lock_guard<std::mutex> lk(g_trace_mu);
  g_trace_names.swap(list);
  return CS_OK;
}

cs_status cs_trace_collect(void) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  size_t done = 0;  // entries already added, dropped even when a later one fails
  struct Drop {
    size_t& n;
    ~Drop() { g_pending.erase(g_pending.begin(), g_pending.begin() + n); }
  } drop{done};
  for (auto& p : g_pending) {
    if (hipEventSynchronize(p.b) != hipSuccess) return fail(CS_ERR_HIP, "hipEventSynchronize failed");
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess)
      return fail(CS_ERR_HIP, "hipEventElapsedTime failed");
    bool found = false;
    for (auto& kv : g_acc)
      if (kv.first == p.name) {
        kv.second.launches += 1;
        kv.second.ms += ms;
        found = true;
        break;
      }
    if (!found) {
      Acc a;
      a.launches = 1;
      a.ms = ms;
      g_acc.push_back({p.name, a});
    }
    g_pool.push_back(p.a);
    g_pool.push_back(p.b);
    ++done;
  }
  return CS_OK;
}

int32_t cs_trace_count(void) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  return (int32_t)g_acc.size();
}

cs_status cs_trace_get(int32_t i, const char** name, int64_t* launches, double* total_ms) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  if (i < 0 || i >= (int32_t)g_acc.size()) return fail(CS_ERR_INVALID_ARGUMENT, "trace index out of range");
  if (name) *name = g_acc[i].first.c_str();
  if (launches) *launches = g_acc[i].second.launches;
  if (total_ms) *total_ms = g_acc[i].second.ms;
  return CS_OK;
}

void cs_trace_reset(void) {
  std::lock_guard<std::mutex> lk(g_trace_mu);
  g_acc.clear();
}

}  // extern "C"
