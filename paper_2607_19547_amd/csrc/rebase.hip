// Three-axis delta rotation of stored post-rotary keys, in place (Eq. 3).
//
// Chunk c turns rotary pair i of every key it owns by
//   phi_{c,i} = Delta_c[sigma(i)] * theta_i.
// Each workgroup first builds its chunk's cos/sin table: the angle is formed
// in float64, reduced modulo 2*pi (Cody-Waite, three-part constant), its
// cos/sin taken in float64 and rounded to float32.  The rows are then
// streamed: every element is read once and written once, so the kernel is
// bound by HBM bandwidth; the rotation itself is 4 flops per pair.
#include <math.h>

#include <algorithm>
#include <type_traits>
#include <vector>

#include "cs_common.h"

namespace cs {

// ---------------------------------------------------------------- bf16, D = 128
constexpr int kFastMaxChunks = 128;
constexpr int kFastTB = 64;  // tokens per workgroup
constexpr int kFastPG = 1;   // planes (layer x kv head) per workgroup
static_assert((kFastPG * kFastTB) % 16 == 0, "a workgroup covers whole row-group steps");

// Chunk q of a launch: its row of plane 0, token 0 at base[q]; planes are T
// rows apart in a contiguous cache and len[q] rows apart in a chunk buffer.
struct RebaseFastArgs {
  int64_t T;
  int planes;
  int sec0, sec01;
  int tblocks;  // token blocks of the longest chunk in this launch
  int nc;       // chunks in this launch
  int paged;
  double theta[64];
  uint16_t* base[kFastMaxChunks];
  int len[kFastMaxChunks];
  int off[kFastMaxChunks][3];
};
static_assert(sizeof(RebaseFastArgs) <= 4096, "kernel arguments within 4 KB");


// Lane layout: 16 lanes per 256-byte row, each with 16 contiguous bytes, so
// a wavefront's access is four whole rows (1 KB) and the pair halves meet
// through DPP (rotate_row16; measured 4% faster than 16 bytes from each half
// per lane, which splits every access into 32 half-rows).  A workgroup of 256
// threads covers kRows rows of one chunk, one row per 16-lane row group and
// step, all loads issued (non-temporal: every byte is touched once) before the
// chunk's table is built, then rotated and stored.  Small workgroups in
// address order keep many independent streams in flight over neighbouring
// memory (one plane x 64 tokens, 16 KB, measured 1-4% faster than 2 planes x
// 64 tokens on the 8k-262k caches).  Contiguous cache ([plane][T] rows): a
// workgroup takes kFastPG planes x kFastTB tokens, token block fastest, then
// chunk, then plane group.
// Paged cache: a chunk buffer is planes x len rows that all turn by the
// chunk's table, so workgroups take runs of kRows consecutive rows, one
// linear stream per chunk.
__global__ __launch_bounds__(256) void rebase_bf16_d128(const RebaseFastArgs a) {
  constexpr int kRows = kFastPG * kFastTB;
  constexpr int kSteps = kRows / 16;  // 16 rows per step: four per wavefront
  __shared__ float2 tab[64];
  const int tb = blockIdx.x % a.tblocks;
  const int rest = blockIdx.x / a.tblocks;
  const int c = a.paged ? rest : rest % a.nc;
  const int pg = rest / a.nc;  // (contiguous only)
  const int len = a.len[c];
  const int jj = threadIdx.x & 15;
  const int r0 = threadIdx.x >> 4;  // 0..15
  u32x4 w[kSteps];
  uint16_t* row[kSteps];
  bool ok[kSteps];
  if (a.paged) {
    const int64_t first = (int64_t)tb * kRows, rows = (int64_t)a.planes * len;
    if (first >= rows) return;  // whole workgroup
#pragma unroll
    for (int u = 0; u < kSteps; ++u) {
      const int64_t r = first + u * 16 + r0;
      ok[u] = r < rows;
      row[u] = a.base[c] + r * 128;
    }
  } else {
    const int t0 = tb * kFastTB;
    if (t0 >= len) return;  // whole workgroup
#pragma unroll
    for (int u = 0; u < kSteps; ++u) {
      const int idx = u * 16 + r0;
      const int plane = pg * kFastPG + idx / kFastTB;
      const int tok = idx % kFastTB;
      ok[u] = plane < a.planes && t0 + tok < len;
      row[u] = a.base[c] + ((int64_t)plane * a.T + t0 + tok) * 128;
    }
  }
#pragma unroll
  for (int u = 0; u < kSteps; ++u)
    w[u] = ok[u] ? __builtin_nontemporal_load((const u32x4*)(row[u] + 8 * jj)) : u32x4{0u, 0u, 0u, 0u};
  if (threadIdx.x < 64) {
    const int i = threadIdx.x;
    const double phi = (double)a.off[c][axis_of(i, a.sec0, a.sec01)] * a.theta[i];
    tab[i] = cos_sin_of(phi);
  }
  __syncthreads();
  const RowRot rr = row_rot(tab, jj);
#pragma unroll
  for (int u = 0; u < kSteps; ++u) {
    const u32x4 o = rotate_row16(w[u], rr);
    if (ok[u]) __builtin_nontemporal_store(o, (u32x4*)(row[u] + 8 * jj));
  }
}

// ---------------------------------------------------------------- generic
constexpr int kGenMaxChunks = 32;
constexpr int kGenTB = 32;

struct RebaseGenArgs {
  int64_t T;
  int planes, D, P;
  int sec0, sec01;
  int tblocks;
  int paged;
  double theta[256];
  char* base[kGenMaxChunks];  // as in RebaseFastArgs
  int len[kGenMaxChunks];
  int off[kGenMaxChunks][3];
};
static_assert(sizeof(RebaseGenArgs) <= 4096, "kernel arguments within 4 KB");

template <typename E>
__device__ __forceinline__ float ld(const E* p);
template <>
__device__ __forceinline__ float ld<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ld<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <typename E>
__device__ __forceinline__ void st(E* p, float x);
template <>
__device__ __forceinline__ void st<float>(float* p, float x) { *p = x; }
template <>
__device__ __forceinline__ void st<uint16_t>(uint16_t* p, float x) { *p = f32_to_bf16(x); }

template <typename E>
__global__ __launch_bounds__(256) void rebase_generic(const RebaseGenArgs a) {
  __shared__ float2 tab[256];
  const int c = blockIdx.y;
  const int tb = blockIdx.x % a.tblocks;
  const int plane = blockIdx.x / a.tblocks;
  const int len = a.len[c];
  const int t0 = tb * kGenTB;
  if (t0 >= len || plane >= a.planes) return;
  for (int i = threadIdx.x; i < a.P; i += blockDim.x) {
    const double phi = (double)a.off[c][axis_of(i, a.sec0, a.sec01)] * a.theta[i];
    tab[i] = cos_sin_of(phi);
  }
  __syncthreads();
  E* k = (E*)a.base[c];
  const int64_t pstride = a.paged ? len : a.T;
  const int ntok = min(kGenTB, len - t0);
  for (int w = threadIdx.x; w < ntok * a.P; w += blockDim.x) {
    const int tok = w / a.P, i = w % a.P;
    E* row = k + ((int64_t)plane * pstride + t0 + tok) * a.D;
    const float x = ld(row + i), y = ld(row + i + a.P);
    const float2 t = tab[i];
    st(row + i, fmaf(x, t.x, -y * t.y));
    st(row + i + a.P, fmaf(x, t.y, y * t.x));
  }
}

// ---------------------------------------------------------------- per-token offsets
// The same rotation with an offset per token (Section 3 compares position
// policies whose offset differs from token to token, e.g. scalar re-basing).
// A workgroup takes a block of kTokTB tokens and kTokPG planes: it first builds
// the block's cos/sin table in LDS (angles in float64, the same reduction as
// above), then streams the block's rows of its planes.  Rows whose token has
// offset (0, 0, 0) are not touched.
// Workgroup shape (tokens x planes) per cache layout, measured on the 65k
// cache under scalar re-basing: contiguous 32 x 4 (64 x 8: 440 us, 16 x 8:
// 595 us, 32 x 4: 416 us), chunk buffers 16 x 8 (64 x 8: 452 us, 32 x 4:
// 534 us, 16 x 8: 412 us).
template <typename Rows>
struct TokShape {
  static constexpr int TB = 32, PG = 4;
};
template <int N>
struct TokShape<PagedRowsT<N>> {
  static constexpr int TB = 16, PG = 8;
};
constexpr int kTokTabW = 65;  // table row stride (float2): one pad entry spreads the LDS banks

template <int P_MAX>
struct RebaseTokArgs {
  const int32_t* off;  // DEVICE [T][3]
  int64_t T;
  int planes, D, P;
  int sec0, sec01;
  double theta[P_MAX];
};

template <typename Rows>
__global__ __launch_bounds__(256) void rebase_tokens_bf16_d128(const RebaseTokArgs<64> a, const Rows rows) {
  constexpr bool kPaged = !std::is_same<Rows, FlatRows>::value;
  constexpr int kTokTB = TokShape<Rows>::TB, kTokPG = TokShape<Rows>::PG;
  constexpr int kU = (kTokPG * kTokTB) / 32;  // rows per lane group
  static_assert(kPaged || kU % 4 == 0, "the contiguous path turns whole batches of four rows per lane group");
  __shared__ float2 tab[kTokTB * kTokTabW];
  __shared__ int moved[kTokTB];
  __shared__ char* row0[kTokTB];         // the token's row in plane 0
  __shared__ int64_t plane_bytes[kTokTB];  // and the distance between planes (one chunk lookup per token)
  const int64_t t0 = (int64_t)blockIdx.x * kTokTB;
  const int ntok = (int)min((int64_t)kTokTB, a.T - t0);
  if (threadIdx.x < kTokTB) {
    const int tok = threadIdx.x;
    int mv = 0;
    if (tok < ntok) {
      const int32_t* o = a.off + (t0 + tok) * 3;
      mv = (o[0] | o[1] | o[2]) != 0;
      rows.token_rows(t0 + tok, 256, row0[tok], plane_bytes[tok]);
    }
    moved[tok] = mv;
  }
  __syncthreads();
  const int j = threadIdx.x & 7;
  const int r0 = threadIdx.x >> 3;  // 0..31
  auto build_table = [&]() {
    for (int e = threadIdx.x; e < kTokTB * 64; e += 256) {
      const int tok = e >> 6, i = e & 63;
      float2 cs = make_float2(1.f, 0.f);
      if (tok < ntok && moved[tok]) {
        const int32_t* o = a.off + (t0 + tok) * 3;
        cs = cos_sin_of((double)o[axis_of(i, a.sec0, a.sec01)] * a.theta[i]);
      }
      tab[tok * kTokTabW + i] = cs;
    }
  };
  auto locate = [&](int u, uint16_t*& row, int& tk) -> bool {  // row u of this lane group
    const int idx = u * 32 + r0;
    const int plane = blockIdx.y * kTokPG + idx / kTokTB;
    tk = idx % kTokTB;
    const bool ok = plane < a.planes && tk < ntok && moved[tk];
    row = ok ? (uint16_t*)(row0[tk] + plane * plane_bytes[tk]) : nullptr;
    return ok;
  };
  auto rotate_store = [&](int tk, uint16_t* row, u32x4& wa, u32x4& wb) {
    float cs_[8], sn_[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float2 t = tab[tk * kTokTabW + 8 * j + e];
      cs_[e] = t.x;
      sn_[e] = t.y;
    }
    rotate8(wa, wb, cs_, sn_);
    __builtin_nontemporal_store(wa, (u32x4*)(row + 8 * j));
    __builtin_nontemporal_store(wb, (u32x4*)(row + 64 + 8 * j));
  };
  if constexpr (kPaged) {
    // A chunk buffer keeps a token's planes len rows apart: every row of the
    // workgroup is loaded (non-temporal: touched once) before the table is
    // built, so the loads are in flight meanwhile (measured 67% of HBM peak
    // against 64% for the batched order below).
    u32x4 wa[kU], wb[kU];
    uint16_t* row[kU];
    int tk[kU];
    bool ok[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      ok[u] = locate(u, row[u], tk[u]);
      if (ok[u]) {
        wa[u] = __builtin_nontemporal_load((const u32x4*)(row[u] + 8 * j));
        wb[u] = __builtin_nontemporal_load((const u32x4*)(row[u] + 64 + 8 * j));
      }
    }
    build_table();
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kU; ++u)
      if (ok[u]) rotate_store(tk[u], row[u], wa[u], wb[u]);
  } else {
    // A contiguous cache keeps a token's planes T rows apart: batches of four
    // rows per lane group, two planes at a time (loading the whole workgroup
    // at once, eight planes 16 MB apart, measured 20% slower).
    build_table();
    __syncthreads();
#pragma unroll 1
    for (int it = 0; it < kU; it += 4) {
      u32x4 wa[4], wb[4];
      uint16_t* row[4];
      int tk[4];
      bool ok[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        ok[u] = locate(it + u, row[u], tk[u]);
        if (ok[u]) {
          wa[u] = __builtin_nontemporal_load((const u32x4*)(row[u] + 8 * j));
          wb[u] = __builtin_nontemporal_load((const u32x4*)(row[u] + 64 + 8 * j));
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (ok[u]) rotate_store(tk[u], row[u], wa[u], wb[u]);
    }
  }
}

// Any head_dim and either dtype: one workgroup per (token, plane), one pair per thread.
template <typename E, typename Rows>
__global__ __launch_bounds__(64) void rebase_tokens_generic(const RebaseTokArgs<256> a, const Rows rows) {
  const int64_t t = blockIdx.x;
  const int plane = blockIdx.y;
  const int32_t* o = a.off + t * 3;
  if ((o[0] | o[1] | o[2]) == 0) return;  // whole workgroup
  E* row = (E*)rows.row(false, plane, t, a.D * (int)sizeof(E));
  for (int i = threadIdx.x; i < a.P; i += blockDim.x) {
    const float2 cs = cos_sin_of((double)o[axis_of(i, a.sec0, a.sec01)] * a.theta[i]);
    const float x = ld(row + i), y = ld(row + i + a.P);
    st(row + i, fmaf(x, cs.x, -y * cs.y));
    st(row + i + a.P, fmaf(x, cs.y, y * cs.x));
  }
}

template <int P_MAX>
static void fill_tok_args(RebaseTokArgs<P_MAX>& a, const Geo& g, const int32_t* off, const double* theta) {
  a.off = off;
  a.T = g.T;
  a.planes = g.L * g.Hkv;
  a.D = g.D;
  a.P = g.P;
  a.sec0 = g.sec[0];
  a.sec01 = g.sec[0] + g.sec[1];
  for (int i = 0; i < g.P; ++i) a.theta[i] = theta[i];
}

template <typename Rows>
static void launch_tok_fast(const RebaseTokArgs<64>& a, const Rows& rows, hipStream_t s) {
  static_assert(sizeof(RebaseTokArgs<64>) + sizeof(Rows) <= 4096, "kernel arguments within 4 KB");
  TraceScope tr("rebase_tokens_bf16_d128", s);
  constexpr int TB = TokShape<Rows>::TB, PG = TokShape<Rows>::PG;
  CS_LAUNCH(tr, rebase_tokens_bf16_d128<Rows>, dim3((unsigned)((a.T + TB - 1) / TB), (unsigned)((a.planes + PG - 1) / PG)),
            dim3(256), 0, s, a, rows);
}

template <typename Rows>
static void launch_tok_generic(const Geo& g, const RebaseTokArgs<256>& a, const Rows& rows, hipStream_t s) {
  static_assert(sizeof(RebaseTokArgs<256>) + sizeof(Rows) <= 4096, "kernel arguments within 4 KB");
  TraceScope tr("rebase_tokens_generic", s);
  if (g.dtype == CS_BF16)
    CS_LAUNCH(tr, (rebase_tokens_generic<uint16_t, Rows>), dim3((unsigned)g.T, a.planes), dim3(64), 0, s, a, rows);
  else
    CS_LAUNCH(tr, (rebase_tokens_generic<float, Rows>), dim3((unsigned)g.T, a.planes), dim3(64), 0, s, a, rows);
}

cs_status launch_rebase_tokens(const Geo& g, const CacheView& cv, const int32_t* off, const double* theta,
                               hipStream_t s, bool check_only) {
  const int64_t planes = (int64_t)g.L * g.Hkv;
  const bool fast = g.dtype == CS_BF16 && g.D == 128;
  const int TB = cv.paged ? TokShape<PagedRowsT<kMaxPages>>::TB : TokShape<FlatRows>::TB;
  const int PG = cv.paged ? TokShape<PagedRowsT<kMaxPages>>::PG : TokShape<FlatRows>::PG;
  cs_status st = fast ? check_grid((g.T + TB - 1) / TB, (planes + PG - 1) / PG, 1, 256, "per-token rebase")
                      : check_grid(g.T, planes, 1, 64, "per-token rebase");
  if (st || check_only) return st;
  if (fast) {
    RebaseTokArgs<64> a;
    fill_tok_args(a, g, off, theta);
    if (cv.paged) launch_tok_fast(a, cv.pages<kMaxPages>(g), s);
    else launch_tok_fast(a, cv.flat(g), s);
  } else {
    RebaseTokArgs<256> a;
    fill_tok_args(a, g, off, theta);
    if (cv.paged) launch_tok_generic(g, a, cv.pages<kMaxPagesGeneric>(g), s);
    else launch_tok_generic(g, a, cv.flat(g), s);
  }
  return check_launch("per-token rebase kernel launch");
}

// ---------------------------------------------------------------- host launcher
cs_status launch_rebase(const Geo& g, const CacheView& cv, const int32_t* off, const double* theta,
                        hipStream_t s, bool check_only) {
  std::vector<int> todo;
  for (int c = 0; c < g.N; ++c)
    if (off[3 * c] || off[3 * c + 1] || off[3 * c + 2]) todo.push_back(c);
  const int planes = g.L * g.Hkv;
  const bool fast = g.dtype == CS_BF16 && g.D == 128;
  const int per = fast ? kFastMaxChunks : kGenMaxChunks;
  // first row of plane 0 of chunk c
  auto chunk_base = [&](int c) -> char* {
    return cv.paged ? (char*)cv.k_chunks[c] : (char*)cv.k + g.cs[c] * (int64_t)g.D * g.esize;
  };
  for (size_t b = 0; b < todo.size(); b += per) {
    const int nc = (int)std::min<size_t>(per, todo.size() - b);
    int maxlen = 0;
    for (int q = 0; q < nc; ++q) {
      const int c = todo[b + q];
      maxlen = std::max<int>(maxlen, (int)(g.cs[c + 1] - g.cs[c]));
    }
    // contiguous: token blocks of the longest chunk; paged: row runs of the largest chunk buffer
    const int64_t tb_fast = cv.paged ? ((int64_t)planes * maxlen + kFastPG * kFastTB - 1) / (kFastPG * kFastTB)
                                     : (maxlen + kFastTB - 1) / kFastTB;
    const int64_t pg_fast = cv.paged ? 1 : (planes + kFastPG - 1) / kFastPG;
    const int64_t tb_gen = (maxlen + kGenTB - 1) / kGenTB;
    cs_status st = fast ? check_grid(tb_fast * pg_fast * nc, 1, 1, 256, "rebase")
                        : check_grid(tb_gen * planes, nc, 1, 256, "rebase");
    if (st) return st;
    if (check_only) continue;
    if (fast) {
      RebaseFastArgs a;
      a.T = g.T;
      a.planes = planes;
      a.sec0 = g.sec[0];
      a.sec01 = g.sec[0] + g.sec[1];
      a.tblocks = (int)tb_fast;
      a.nc = nc;
      a.paged = cv.paged ? 1 : 0;
      for (int i = 0; i < 64; ++i) a.theta[i] = theta[i];
      for (int q = 0; q < nc; ++q) {
        const int c = todo[b + q];
        a.base[q] = (uint16_t*)chunk_base(c);
        a.len[q] = (int)(g.cs[c + 1] - g.cs[c]);
        for (int x = 0; x < 3; ++x) a.off[q][x] = off[3 * c + x];
      }
      TraceScope tr("rebase_bf16_d128", s);
      CS_LAUNCH(tr, rebase_bf16_d128, dim3((unsigned)(tb_fast * pg_fast * nc)), dim3(256), 0, s, a);
    } else {
      RebaseGenArgs a;
      a.T = g.T;
      a.planes = planes;
      a.D = g.D;
      a.P = g.P;
      a.sec0 = g.sec[0];
      a.sec01 = g.sec[0] + g.sec[1];
      a.tblocks = (int)tb_gen;
      a.paged = cv.paged ? 1 : 0;
      for (int i = 0; i < g.P; ++i) a.theta[i] = theta[i];
      for (int q = 0; q < nc; ++q) {
        const int c = todo[b + q];
        a.base[q] = chunk_base(c);
        a.len[q] = (int)(g.cs[c + 1] - g.cs[c]);
        for (int x = 0; x < 3; ++x) a.off[q][x] = off[3 * c + x];
      }
      TraceScope tr("rebase_generic", s);
      if (g.dtype == CS_BF16)
        CS_LAUNCH(tr, rebase_generic<uint16_t>, dim3(a.tblocks * planes, nc), dim3(256), 0, s, a);
      else
        CS_LAUNCH(tr, rebase_generic<float>, dim3(a.tblocks * planes, nc), dim3(256), 0, s, a);
    }
    st = check_launch("rebase kernel launch");
    if (st) return st;
  }
  return CS_OK;
}

}  // namespace cs
