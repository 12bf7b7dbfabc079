// Fused rotary embedding of the recomputed rows (Eq. 2 at the global
// coordinates p' of Section 2), for callers that hand over pre-rotary fresh
// queries and keys: only the selected rows are rotated.
//
// For every selected token t (slot m) and layer of the call:
//   K row of each KV head:  f(k_pre, p'_t), rounded to the storage dtype,
//                           written into the cache at row t (the repair scatter);
//   V row of each KV head:  copied into the cache at row t;
//   Q row of each query head: f(q_pre, p'_t), rounded, written to the
//                           workspace at [layer][head][m] for the attention.
// A workgroup takes kRsTok selected tokens of one layer, builds their cos/sin
// table in LDS (angles in float64, reduced modulo 2*pi, rounded to float32,
// as the re-basing kernels do) and streams the tokens' rows.
#include <math.h>

#include <algorithm>

#include "cs_common.h"

namespace cs {

constexpr int kRsTok = 8;       // selected tokens per workgroup
constexpr int kRsTabW = 65;     // table row stride (float2): one pad entry spreads the LDS banks

struct RopeScatterArgs {
  uint16_t* q_ws;         // [layers in call][H_q][n_sel][128]
  const uint16_t* q_pre;  // [L][H_q][n][128]
  const uint16_t* k_pre;  // [L][H_kv][n][128]
  const uint16_t* v_new;  // [L][H_kv][n][128]
  const int32_t* sel;
  const int32_t* coords;  // [T][3] global coordinates
  int64_t T, n, n_sel, cs1;
  int Hq, Hkv, lb;
  int sec0, sec01;
  double theta[64];
};

// Cache rows (K, V) are reached through the row map `rows`.
template <typename Rows>
__global__ __launch_bounds__(256) void rope_scatter_bf16_d128(const RopeScatterArgs a, const Rows rows) {
  __shared__ float2 tab[kRsTok * kRsTabW];
  __shared__ int tok_of[kRsTok];
  const int64_t m0 = (int64_t)blockIdx.x * kRsTok;
  const int nm = (int)std::min<int64_t>(kRsTok, a.n_sel - m0);
  const int layer = a.lb + blockIdx.y;
  if (threadIdx.x < kRsTok) {
    int t = -1;
    if ((int)threadIdx.x < nm) {
      const int64_t g = a.sel[m0 + threadIdx.x];
      if (g >= a.cs1 && g < a.T) t = (int)g;  // out-of-contract index: the row is skipped
    }
    tok_of[threadIdx.x] = t;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < kRsTok * 64; e += 256) {
    const int r = e >> 6, i = e & 63;
    const int t = tok_of[r];
    float2 cs = make_float2(1.f, 0.f);
    if (t >= 0) cs = cos_sin_of((double)a.coords[(int64_t)t * 3 + axis_of(i, a.sec0, a.sec01)] * a.theta[i]);
    tab[r * kRsTabW + i] = cs;
  }
  __syncthreads();
  const int j = threadIdx.x & 7;
  const int r0 = threadIdx.x >> 3;  // 0..31
  const int rows_per_tok = 2 * a.Hkv + a.Hq;
  const int total = kRsTok * rows_per_tok;
  // rows in batches of four per lane group: all loads of a batch before its stores
#pragma unroll 1
  for (int base = 0; base < total; base += 128) {
    u32x4 wa[4], wb[4];
    uint16_t* dst[4];
    int rr[4];
    bool ok[4], rot[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int idx = base + 32 * u + r0;
      const int r = idx % kRsTok, kind = idx / kRsTok;  // kind: [0, Hkv) K, [Hkv, 2 Hkv) V, then Q heads
      const int t0 = idx < total ? tok_of[r] : -1;
      ok[u] = t0 >= 0;
      const int t = ok[u] ? t0 : (int)a.cs1;  // (addresses of skipped rows are formed but never used)
      rr[u] = r;
      rot[u] = kind < a.Hkv || kind >= 2 * a.Hkv;
      const uint16_t* src;
      if (kind < 2 * a.Hkv) {
        const bool is_k = kind < a.Hkv;
        const int h = is_k ? kind : kind - a.Hkv;
        src = (is_k ? a.k_pre : a.v_new) + (((int64_t)layer * a.Hkv + h) * a.n + (t - a.cs1)) * 128;
        dst[u] = (uint16_t*)rows.row(!is_k, (int64_t)layer * a.Hkv + h, t, 256);
      } else {
        const int h = kind - 2 * a.Hkv;
        src = a.q_pre + (((int64_t)layer * a.Hq + h) * a.n + (t - a.cs1)) * 128;
        dst[u] = a.q_ws + (((int64_t)blockIdx.y * a.Hq + h) * a.n_sel + m0 + r) * 128;
      }
      if (ok[u]) {
        wa[u] = *(const u32x4*)(src + 8 * j);
        wb[u] = *(const u32x4*)(src + 64 + 8 * j);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (!ok[u]) continue;
      if (rot[u]) {
        float cs_[8], sn_[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float2 c = tab[rr[u] * kRsTabW + 8 * j + e];
          cs_[e] = c.x;
          sn_[e] = c.y;
        }
        rotate8(wa[u], wb[u], cs_, sn_);
      }
      *(u32x4*)(dst[u] + 8 * j) = wa[u];
      *(u32x4*)(dst[u] + 64 + 8 * j) = wb[u];
    }
  }
}

// Any head_dim and either dtype: one workgroup per (selected slot, layer).
struct RopeScatterGenArgs {
  void* q_ws;
  const void* q_pre;
  const void* k_pre;
  const void* v_new;
  const int32_t* sel;
  const int32_t* coords;
  int64_t T, n, n_sel, cs1;
  int Hq, Hkv, lb, D, P;
  int sec0, sec01;
  double theta[256];
};

template <typename E>
__device__ __forceinline__ float ldx(const E* p);
template <>
__device__ __forceinline__ float ldx<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ldx<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <typename E>
__device__ __forceinline__ void stx(E* p, float x);
template <>
__device__ __forceinline__ void stx<float>(float* p, float x) { *p = x; }
template <>
__device__ __forceinline__ void stx<uint16_t>(uint16_t* p, float x) { *p = f32_to_bf16(x); }

template <typename E, typename Rows>
__global__ __launch_bounds__(64) void rope_scatter_generic(const RopeScatterGenArgs a, const Rows rows) {
  const int64_t m = blockIdx.x;
  const int layer = a.lb + blockIdx.y;
  const int64_t t = a.sel[m];
  if (t < a.cs1 || t >= a.T) return;  // whole workgroup: out-of-contract index
  const int64_t r = t - a.cs1;
  for (int i = threadIdx.x; i < a.P; i += blockDim.x) {
    const float2 cs = cos_sin_of((double)a.coords[t * 3 + axis_of(i, a.sec0, a.sec01)] * a.theta[i]);
    for (int h = 0; h < a.Hkv; ++h) {
      const E* kp = (const E*)a.k_pre + (((int64_t)layer * a.Hkv + h) * a.n + r) * a.D;
      char *kr, *vr;
      rows.kv_rows((int64_t)layer * a.Hkv + h, t, a.D * (int)sizeof(E), kr, vr);
      E* kd = (E*)kr;
      const float x = ldx(kp + i), y = ldx(kp + i + a.P);
      stx(kd + i, fmaf(x, cs.x, -y * cs.y));
      stx(kd + i + a.P, fmaf(x, cs.y, y * cs.x));
      const E* vp = (const E*)a.v_new + (((int64_t)layer * a.Hkv + h) * a.n + r) * a.D;
      E* vd = (E*)vr;
      vd[i] = vp[i];
      vd[i + a.P] = vp[i + a.P];
    }
    for (int h = 0; h < a.Hq; ++h) {
      const E* qp = (const E*)a.q_pre + (((int64_t)layer * a.Hq + h) * a.n + r) * a.D;
      E* qd = (E*)a.q_ws + (((int64_t)blockIdx.y * a.Hq + h) * a.n_sel + m) * a.D;
      const float x = ldx(qp + i), y = ldx(qp + i + a.P);
      stx(qd + i, fmaf(x, cs.x, -y * cs.y));
      stx(qd + i + a.P, fmaf(x, cs.y, y * cs.x));
    }
  }
}

template <typename Rows>
static void launch_rs_fast(const RopeScatterArgs& a, const Rows& rows, int64_t n_sel, int layers, hipStream_t s) {
  static_assert(sizeof(RopeScatterArgs) + sizeof(Rows) <= 4096, "kernel arguments within 4 KB");
  TraceScope tr("rope_scatter_bf16_d128", s);
  hipLaunchKernelGGL(rope_scatter_bf16_d128<Rows>, dim3((unsigned)((n_sel + kRsTok - 1) / kRsTok), layers),
                     dim3(256), 0, s, a, rows);
}

template <typename Rows>
static void launch_rs_generic(const Geo& g, const RopeScatterGenArgs& a, const Rows& rows, int64_t n_sel, int layers,
                              hipStream_t s) {
  static_assert(sizeof(RopeScatterGenArgs) + sizeof(Rows) <= 4096, "kernel arguments within 4 KB");
  TraceScope tr("rope_scatter_generic", s);
  if (g.dtype == CS_BF16)
    hipLaunchKernelGGL((rope_scatter_generic<uint16_t, Rows>), dim3((unsigned)n_sel, layers), dim3(64), 0, s, a, rows);
  else
    hipLaunchKernelGGL((rope_scatter_generic<float, Rows>), dim3((unsigned)n_sel, layers), dim3(64), 0, s, a, rows);
}

cs_status launch_rope_scatter(const Geo& g, const CacheView& cv, int lb, int le, const int32_t* sel, int64_t n_sel,
                              const void* q_pre, const void* k_pre, const void* v_new, const int32_t* coords,
                              const double* theta, void* q_ws, hipStream_t s, bool check_only) {
  const bool fast = g.dtype == CS_BF16 && g.D == 128;
  const cs_status stg = fast ? check_grid((n_sel + kRsTok - 1) / kRsTok, le - lb, 1, 256, "rope scatter")
                             : check_grid(n_sel, le - lb, 1, 64, "rope scatter");
  if (stg || check_only) return stg;
  if (fast) {
    RopeScatterArgs a;
    a.q_ws = (uint16_t*)q_ws;
    a.q_pre = (const uint16_t*)q_pre;
    a.k_pre = (const uint16_t*)k_pre;
    a.v_new = (const uint16_t*)v_new;
    a.sel = sel;
    a.coords = coords;
    a.T = g.T;
    a.n = g.n;
    a.n_sel = n_sel;
    a.cs1 = g.cs1;
    a.Hq = g.Hq;
    a.Hkv = g.Hkv;
    a.lb = lb;
    a.sec0 = g.sec[0];
    a.sec01 = g.sec[0] + g.sec[1];
    for (int i = 0; i < 64; ++i) a.theta[i] = theta[i];
    if (cv.paged) launch_rs_fast(a, cv.pages<kMaxPages>(g), n_sel, le - lb, s);
    else launch_rs_fast(a, cv.flat(g), n_sel, le - lb, s);
  } else {
    RopeScatterGenArgs a;
    a.q_ws = q_ws;
    a.q_pre = q_pre;
    a.k_pre = k_pre;
    a.v_new = v_new;
    a.sel = sel;
    a.coords = coords;
    a.T = g.T;
    a.n = g.n;
    a.n_sel = n_sel;
    a.cs1 = g.cs1;
    a.Hq = g.Hq;
    a.Hkv = g.Hkv;
    a.lb = lb;
    a.D = g.D;
    a.P = g.P;
    a.sec0 = g.sec[0];
    a.sec01 = g.sec[0] + g.sec[1];
    for (int i = 0; i < g.P; ++i) a.theta[i] = theta[i];
    if (cv.paged) launch_rs_generic(g, a, cv.pages<kMaxPagesGeneric>(g), n_sel, le - lb, s);
    else launch_rs_generic(g, a, cv.flat(g), n_sel, le - lb, s);
  }
  return check_launch("rope scatter launch");
}

}  // namespace cs
