// Internal helpers shared by the HIP sources of the composition library.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "chronostitch.h"

namespace cs {

// ------------------------------------------------------------------ errors
void set_error(const std::string& msg);
cs_status fail(cs_status code, const std::string& msg);
cs_status check_launch(const char* what);
// A launch of gx x gy x gz workgroups of `threads` work-items within the
// hardware's grid limits (work-items along x below 2^32, gx below 2^31, gy and
// gz at most 65535); CS_ERR_UNSUPPORTED otherwise.
cs_status check_grid(int64_t gx, int64_t gy, int64_t gz, int threads, const char* what);

// ------------------------------------------------------------------ tracing
// While tracing is on, holds two events for the one launch of its scope
// (CS_LAUNCH): the dispatch itself stamps them at the kernel's start and end,
// so tracing adds no packets to the stream; the pair goes to the collector
// when the scope ends.
struct TraceScope {
  TraceScope(const char* name, hipStream_t s);
  ~TraceScope();
  const char* name;
  hipStream_t stream;
  hipEvent_t a, b;  // both null while tracing is off
};
#define CS_LAUNCH(tr, kernel, grid, block, shmem, stream, ...)                                           \
  do {                                                                                                   \
    if ((tr).a) hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, (tr).a, (tr).b, 0, __VA_ARGS__); \
    else hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);                             \
  } while (0)

// ------------------------------------------------------------------ geometry
struct Geo {
  int L, Hq, Hkv, G, D, P;
  int sec[3];
  int dtype;          // cs_dtype
  int esize;          // bytes per element
  int64_t T;
  int N;
  const int64_t* cs;  // chunk_start (host)
  int64_t cs1, n;     // first later-chunk token, candidate count
};

// Validates the geometry; on success fills `out`.
cs_status check_geometry(const cs_geometry* g, Geo* out);

int64_t n_select(double rho, int64_t n);

// ------------------------------------------------------------------ device-side types
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// bf16 <-> f32 on packed 32-bit words (element 0 in the low half).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
// Round two floats to bf16 (nearest even, native v_cvt_pk_bf16_f32) and pack.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 v = {lo, hi};
  bf16x2 b = __builtin_convertvector(v, bf16x2);
  return __builtin_bit_cast(uint32_t, b);
}
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float(((uint32_t)h) << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16(float x) { return (uint16_t)(pack_bf16x2(x, 0.f) & 0xffffu); }

// ------------------------------------------------------------------ rotation (Eq. 2, Eq. 3)
// cos/sin of a rotary angle formed in float64: reduced modulo 2*pi, evaluated
// in float64 and rounded once to float32.
// 2*pi = C1 + C2 + C3 with C1, C2 holding 26 significant bits each, so
// k*C1 and k*C2 are exact for |k| < 2^27.
#define CS_TWO_PI_C1 0x1.921fb50000000p+2
#define CS_TWO_PI_C2 0x1.110b460000000p-24
#define CS_TWO_PI_C3 0x1.1a62633145c07p-52
#define CS_INV_TWO_PI 0x1.45f306dc9c883p-3

__device__ __forceinline__ float2 cos_sin_of(double phi) {
  double k = rint(phi * CS_INV_TWO_PI);
  double r = phi;
  if (fabs(k) < 134217728.0) {  // 2^27
    r = fma(-k, CS_TWO_PI_C1, r);
    r = fma(-k, CS_TWO_PI_C2, r);
    r = fma(-k, CS_TWO_PI_C3, r);
  }
  double s, c;
  sincos(r, &s, &c);
  return make_float2((float)c, (float)s);
}

__device__ __forceinline__ int axis_of(int i, int sec0, int sec01) {
  return i < sec0 ? 0 : (i < sec01 ? 1 : 2);
}

// Rotates 8 rotary pairs held as bf16: wa = elements 8j..8j+7 of the first
// half-row, wb = the same of the second half (pair i = (i, i + 64)).
__device__ __forceinline__ void rotate8(u32x4& wa, u32x4& wb, const float* c, const float* s) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float a0 = bf16_lo(wa[w]), a1 = bf16_hi(wa[w]);
    float b0 = bf16_lo(wb[w]), b1 = bf16_hi(wb[w]);
    float c0 = c[2 * w], s0 = s[2 * w], c1 = c[2 * w + 1], s1 = s[2 * w + 1];
    float na0 = fmaf(a0, c0, -b0 * s0), nb0 = fmaf(a0, s0, b0 * c0);
    float na1 = fmaf(a1, c1, -b1 * s1), nb1 = fmaf(a1, s1, b1 * c1);
    wa[w] = pack_bf16x2(na0, na1);
    wb[w] = pack_bf16x2(nb0, nb1);
  }
}

// Row-contiguous lane layout: 16 lanes per 256-byte row, lane jj holding
// bytes 16 jj .. 16 jj + 15 (elements 8 jj .. 8 jj + 7); pair (i, i + 64) lies
// in lanes jj and jj ^ 8 of the same row, which swap their words through DPP
// (row_ror:8 within each 16-lane row).  The rotation is rotate8's arithmetic:
// first half a' = a c - b s, second half b' = a s + b c.  Every lane of a
// row must execute this (both halves of a pair are active or neither).
struct RowRot {
  float m1[8], m2[8];  // first half: (cos, sin); second half: (sin, cos)
  bool first;
};
__device__ __forceinline__ RowRot row_rot(const float2* tab, int jj) {
  RowRot r;
  r.first = jj < 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float2 t = tab[8 * (jj & 7) + e];
    r.m1[e] = r.first ? t.x : t.y;
    r.m2[e] = r.first ? t.y : t.x;
  }
  return r;
}
__device__ __forceinline__ u32x4 rotate_row16(u32x4 x, const RowRot& r) {
  u32x4 y;
#pragma unroll
  for (int w = 0; w < 4; ++w) y[w] = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x[w], 0x128, 0xf, 0xf, false);
  u32x4 o;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float x0 = bf16_lo(x[w]), x1 = bf16_hi(x[w]), y0 = bf16_lo(y[w]), y1 = bf16_hi(y[w]);
    // first half: fma(a, c, -(b s)) with a = own, b = partner; second: fma(a, s, b c) with a = partner, b = own
    const float u0 = r.first ? x0 : y0, v0 = r.first ? y0 : x0, u1 = r.first ? x1 : y1, v1 = r.first ? y1 : x1;
    const float n0 = r.first ? fmaf(u0, r.m1[2 * w], -(v0 * r.m2[2 * w])) : fmaf(u0, r.m1[2 * w], v0 * r.m2[2 * w]);
    const float n1 = r.first ? fmaf(u1, r.m1[2 * w + 1], -(v1 * r.m2[2 * w + 1])) : fmaf(u1, r.m1[2 * w + 1], v1 * r.m2[2 * w + 1]);
    o[w] = pack_bf16x2(n0, n1);
  }
  return o;
}

// ------------------------------------------------------------------ cache row addressing
// A contiguous cache is one buffer per tensor, [L][H_kv][T][D].  A paged
// cache keeps chunk c in buffers of its own, [L][H_kv][len_c][D] with
// len_c = start[c+1] - start[c]: the chunks stay where they were loaded and
// are never concatenated (Section 2 stores every chunk's cache on its own).
// Kernels reach a row through one of these two maps, a template argument, so
// the contiguous instantiation keeps its plain address arithmetic.
// plane = layer * H_kv + KV head; t = composed token index.
struct FlatRows {
  char* k;
  char* v;
  int64_t T;
  __device__ __forceinline__ char* row(bool val, int64_t plane, int64_t t, int row_bytes) const {
    return (val ? v : k) + (plane * T + t) * row_bytes;
  }
  __device__ __forceinline__ void kv_rows(int64_t plane, int64_t t, int row_bytes, char*& kr, char*& vr) const {
    const int64_t o = (plane * T + t) * row_bytes;
    kr = k + o;
    vr = v + o;
  }
  // Key row of token t in plane 0 and the byte distance between planes.
  __device__ __forceinline__ void token_rows(int64_t t, int row_bytes, char*& k0, int64_t& plane_bytes) const {
    k0 = k + t * row_bytes;
    plane_bytes = T * row_bytes;
  }
};

// Up to CAP chunks, carried in the kernel arguments.  The bf16 / D = 128
// kernels take 128; kernels whose arguments also hold a 256-entry float64
// table take 64, so that every argument block stays within 4 KB.
template <int CAP>
struct PagedRowsT {
  static constexpr int kCap = CAP;
  int n;               // chunks
  int start[CAP + 1];  // token start of each chunk, start[n] = T
  char* k[CAP];
  char* v[CAP];        // NULL entries when only keys are addressed
  // chunk of token t (0 <= t < T): the largest c with start[c] <= t
  __device__ __forceinline__ int chunk_of(int64_t t) const {
    int lo = 0, hi = n;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (start[mid] <= t) lo = mid;
      else hi = mid;
    }
    return lo;
  }
  __device__ __forceinline__ char* row(bool val, int64_t plane, int64_t t, int row_bytes) const {
    const int c = chunk_of(t);
    const int64_t len = start[c + 1] - start[c];
    return (val ? v[c] : k[c]) + (plane * len + (t - start[c])) * row_bytes;
  }
  __device__ __forceinline__ void kv_rows(int64_t plane, int64_t t, int row_bytes, char*& kr, char*& vr) const {
    const int c = chunk_of(t);
    const int64_t o = (plane * (int64_t)(start[c + 1] - start[c]) + (t - start[c])) * row_bytes;
    kr = k[c] + o;
    vr = v[c] + o;
  }
  __device__ __forceinline__ void token_rows(int64_t t, int row_bytes, char*& k0, int64_t& plane_bytes) const {
    const int c = chunk_of(t);
    k0 = k[c] + (t - start[c]) * row_bytes;
    plane_bytes = (int64_t)(start[c + 1] - start[c]) * row_bytes;
  }
};
constexpr int kMaxPages = 128;
constexpr int kMaxPagesGeneric = 64;
using PagedRows = PagedRowsT<kMaxPages>;
using PagedRowsG = PagedRowsT<kMaxPagesGeneric>;

// Host-side description of either layout, as the entry points receive it.
struct CacheView {
  bool paged = false;
  void* k = nullptr;  // contiguous buffers
  void* v = nullptr;
  void* const* k_chunks = nullptr;  // paged: HOST [N] device pointers
  void* const* v_chunks = nullptr;  // (NULL: keys only)
  FlatRows flat(const Geo& g) const {
    FlatRows r;
    r.k = (char*)k;
    r.v = (char*)v;
    r.T = g.T;
    return r;
  }
  template <int CAP>
  PagedRowsT<CAP> pages(const Geo& g) const {  // caller checked g.N <= CAP
    PagedRowsT<CAP> r;
    r.n = g.N;
    for (int c = 0; c <= g.N; ++c) r.start[c] = (int)g.cs[c];
    for (int c = 0; c < g.N; ++c) {
      r.k[c] = (char*)k_chunks[c];
      r.v[c] = v_chunks ? (char*)v_chunks[c] : nullptr;
    }
    return r;
  }
};

// ------------------------------------------------------------------ launches (per source file)
// Each launcher with check_only set validates its launch sizes and enqueues
// nothing, so that an entry point can reject a call before any device work.
cs_status launch_rebase(const Geo& g, const CacheView& cv, const int32_t* offsets, const double* theta,
                        hipStream_t s, bool check_only = false);
cs_status launch_rebase_tokens(const Geo& g, const CacheView& cv, const int32_t* token_offsets, const double* theta,
                               hipStream_t s, bool check_only = false);
cs_status launch_score_select(const Geo& g, const CacheView& cv, int score_layer, const void* k_fresh, float* scores,
                              int32_t* sel, int64_t k_sel, hipStream_t s, bool check_only = false);

struct AttnPlan {
  bool mfma;            // bf16, D = 128, 32 % G == 0
  int rows_per_tile;    // selected rows per workgroup tile
  int64_t n_tiles;      // per KV head
  int part_cap;         // partial slots per layer
  int desc_off;         // item descriptors in the plan (ints from its start)
  size_t ws_fixed_bytes;      // per call: tile plan
  size_t ws_bytes_per_layer;  // per layer in the call: partial segments
};
// max_part_slots caps the partial slots per layer below the library's own
// bound (the plan then makes longer key pieces, or none).
AttnPlan plan_attention(const Geo& g, int64_t n_sel, int layers_per_call, int64_t max_part_slots = INT64_MAX);
// Every chunk starts at a multiple of the 64-key tile (a paged cache on the MFMA path needs it).
bool chunks_tile_aligned(const Geo& g);
// The fresh K/V rows the attention launch also scatters into the cache
// before it reads it (the plain scatter of selective_attend_scatter).
struct ScatterJob {
  const void* kf;
  const void* vf;
};
// The rotary embedding of the recomputed rows, fused into the attention
// launches (bf16, head_dim 128): the scatter rotates the fresh keys at the
// global coordinates and the attention rotates the queries as it loads them,
// both from a cos/sin table of the selected tokens built once per call.
struct RopeJob {
  const void* k_pre;      // [L][H_kv][n][D] pre-rotary fresh keys
  const void* v_new;      // [L][H_kv][n][D] fresh values
  const int32_t* coords;  // DEVICE [T][3] global coordinates
  const double* theta;    // HOST [D/2]
  void* tab;              // DEVICE [n_sel][D/2] float2 (cos, sin), workspace
};
size_t rope_table_bytes(int64_t n_sel);
cs_status launch_attention(const Geo& g, const AttnPlan& plan, const CacheView& cv,
                           int lb, int le, const int32_t* sel, int64_t n_sel, const void* qf,
                           bool q_by_slot, void* out, float* lse, void* ws, hipStream_t s, bool check_only = false,
                           const ScatterJob* job = nullptr, const RopeJob* rope = nullptr);
cs_status launch_rope_scatter(const Geo& g, const CacheView& cv, int lb, int le, const int32_t* sel, int64_t n_sel,
                              const void* q_pre, const void* k_pre, const void* v_new, const int32_t* coords,
                              const double* theta, void* q_ws, hipStream_t s, bool check_only = false);

}  // namespace cs
