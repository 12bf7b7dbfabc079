// Rotary embedding of the recomputed rows (Eq. 2 at the global coordinates
// p' of Section 2) for the generic attention path (any head_dim, either
// dtype), for callers that hand over pre-rotary fresh queries and keys: only
// the selected rows are rotated.  (On the bf16 / head_dim 128 path the
// rotation runs inside the attention's own launches.)
//
// For every selected token t (slot m) and layer of the call:
//   K row of each KV head:  f(k_pre, p'_t), rounded to the storage dtype,
//                           written into the cache at row t (the repair scatter);
//   V row of each KV head:  copied into the cache at row t;
//   Q row of each query head: f(q_pre, p'_t), rounded, written to the
//                           workspace at [layer][head][m] for the attention.
// One workgroup per (selected slot, layer); angles in float64, reduced modulo
// 2*pi, rounded to float32, as the re-basing kernels do.
#include <math.h>

#include <algorithm>

#include "cs_common.h"

namespace cs {

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
static void launch_rs_generic(const Geo& g, const RopeScatterGenArgs& a, const Rows& rows, int64_t n_sel, int layers,
                              hipStream_t s) {
  static_assert(sizeof(RopeScatterGenArgs) + sizeof(Rows) <= 4096, "kernel arguments within 4 KB");
  TraceScope tr("rope_scatter_generic", s);
  if (g.dtype == CS_BF16)
    CS_LAUNCH(tr, (rope_scatter_generic<uint16_t, Rows>), dim3((unsigned)n_sel, layers), dim3(64), 0, s, a, rows);
  else
    CS_LAUNCH(tr, (rope_scatter_generic<float, Rows>), dim3((unsigned)n_sel, layers), dim3(64), 0, s, a, rows);
}

cs_status launch_rope_scatter(const Geo& g, const CacheView& cv, int lb, int le, const int32_t* sel, int64_t n_sel,
                              const void* q_pre, const void* k_pre, const void* v_new, const int32_t* coords,
                              const double* theta, void* q_ws, hipStream_t s, bool check_only) {
  const cs_status stg = check_grid(n_sel, le - lb, 1, 64, "rope scatter");
  if (stg || check_only) return stg;
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
  return check_launch("rope scatter launch");
}

}  // namespace cs
