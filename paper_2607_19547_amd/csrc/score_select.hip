// Per-token key deviation (Eq. 5) and deterministic top-k selection.
//
// delta_t = || k_fresh[:, t - s1, :] - k[score_layer][:, t, :] ||_2 over all
// KV heads x head_dim, accumulated in float64 (bf16 differences and their
// squares are exact in float64) and rounded once to float32.
//
// Selection ranks the float32 scores.  Scores are >= 0, so their IEEE bit
// patterns order like unsigned integers; a single workgroup finds the k-th
// largest bit pattern by a 4-pass, 8-bit MSB-first radix select with LDS
// histograms, then compacts in index order: every score above the threshold
// and the first (lowest-index) ties at the threshold, so the output is
// ascending and exactly k long.  All counts are order independent, so the
// result is deterministic.
#include "cs_common.h"

namespace cs {

template <typename E>
__device__ __forceinline__ double ldd(const E* p);
template <>
__device__ __forceinline__ double ldd<float>(const float* p) { return (double)*p; }
template <>
__device__ __forceinline__ double ldd<uint16_t>(const uint16_t* p) { return (double)bf16_to_f32(*p); }

// One wavefront per candidate token.  Rows of the score layer are reached
// through the cache's row map (plane = score_layer * H_kv + head).
template <typename E, typename Rows>
__global__ __launch_bounds__(256) void deviation_score(const Rows rows, const E* __restrict__ kf,
                                                       float* __restrict__ scores, int score_layer,
                                                       int64_t n, int64_t cs1, int Hkv, int D) {
  const int64_t tok = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (tok >= n) return;  // whole wavefront
  const int lane = threadIdx.x & 63;
  double acc = 0.0;
  for (int h = 0; h < Hkv; ++h) {
    const E* a = (const E*)rows.row(false, (int64_t)score_layer * Hkv + h, cs1 + tok, D * (int)sizeof(E));
    const E* b = kf + ((int64_t)h * n + tok) * D;
    for (int d = lane; d < D; d += 64) {
      const double x = ldd(b + d) - ldd(a + d);
      acc = fma(x, x, acc);
    }
  }
#pragma unroll
  for (int o = 32; o; o >>= 1) acc += __shfl_xor(acc, o);
  if (lane == 0) scores[tok] = (float)sqrt(acc);
}

// bf16, D = 128: 16 lanes per token, 8 elements per lane per head.
template <typename Rows>
__global__ __launch_bounds__(256) void deviation_score_bf16_d128(const Rows rows, const uint16_t* __restrict__ kf,
                                                                 float* __restrict__ scores, int score_layer,
                                                                 int64_t n, int64_t cs1, int Hkv) {
  const int64_t tok = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
  const int j = threadIdx.x & 15;
  double acc = 0.0;
  if (tok < n) {
    for (int h = 0; h < Hkv; ++h) {
      const u32x4 a = *(const u32x4*)((const uint16_t*)rows.row(false, (int64_t)score_layer * Hkv + h, cs1 + tok, 256) + 8 * j);
      const u32x4 b = *(const u32x4*)(kf + ((int64_t)h * n + tok) * 128 + 8 * j);
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const double x0 = (double)bf16_lo(b[w]) - (double)bf16_lo(a[w]);
        const double x1 = (double)bf16_hi(b[w]) - (double)bf16_hi(a[w]);
        acc = fma(x0, x0, acc);
        acc = fma(x1, x1, acc);
      }
    }
  }
#pragma unroll
  for (int o = 8; o; o >>= 1) acc += __shfl_xor(acc, o, 16);
  if (tok < n && j == 0) scores[tok] = (float)sqrt(acc);
}

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;

// Block-wide exclusive scan of one flag per thread; returns this thread's
// rank among set flags and writes the block total to *total.
__device__ __forceinline__ unsigned block_flag_scan(bool f, unsigned* wsum, unsigned* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long b = __ballot(f);
  const unsigned lane_rank = __popcll(b & ((1ull << lane) - 1ull));
  if (lane == 0) wsum[wave] = __popcll(b);
  __syncthreads();
  unsigned off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    const unsigned v = wsum[w];
    off += w < wave ? v : 0u;
    tot += v;
  }
  __syncthreads();
  *total = tot;
  return off + lane_rank;
}

__global__ __launch_bounds__(kSelThreads) void radix_select_topk(const float* __restrict__ scores,
                                                                 int n, int k, int cs1,
                                                                 int32_t* __restrict__ sel) {
  __shared__ unsigned hist[kSelWaves][256];
  __shared__ unsigned tot[256];
  __shared__ unsigned s_prefix, s_kk;
  __shared__ unsigned wsum[kSelWaves];
  const unsigned* bits = (const unsigned*)scores;
  const int tid = threadIdx.x, wave = tid >> 6;
  unsigned prefix = 0u, mask = 0u, kk = (unsigned)k;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < kSelWaves * 256; b += kSelThreads) (&hist[0][0])[b] = 0u;
    __syncthreads();
    for (int i = tid; i < n; i += kSelThreads) {
      const unsigned u = bits[i];
      if ((u & mask) == prefix) atomicAdd(&hist[wave][(u >> shift) & 255u], 1u);
    }
    __syncthreads();
    for (int b = tid; b < 256; b += kSelThreads) {
      unsigned s = 0;
#pragma unroll
      for (int w = 0; w < kSelWaves; ++w) s += hist[w][b];
      tot[b] = s;
    }
    __syncthreads();
    if (tid == 0) {
      unsigned cum = 0;
      for (int d = 255; d >= 0; --d) {
        if (cum + tot[d] >= kk) {
          s_prefix = prefix | ((unsigned)d << shift);
          s_kk = kk - cum;
          break;
        }
        cum += tot[d];
      }
    }
    __syncthreads();
    prefix = s_prefix;
    kk = s_kk;
    mask |= 255u << shift;
  }
  // prefix is now the k-th largest bit pattern; kk ties at it are taken.
  const unsigned thr = prefix;
  unsigned out_base = 0, eq_base = 0;
  for (int base = 0; base < n; base += kSelThreads) {
    const int i = base + tid;
    const unsigned u = i < n ? bits[i] : 0u;
    const bool gt = i < n && u > thr;
    const bool eq = i < n && u == thr;
    unsigned eq_total, take_total;
    const unsigned eq_rank = eq_base + block_flag_scan(eq, wsum, &eq_total);
    const bool take = gt || (eq && eq_rank < kk);
    const unsigned pos = block_flag_scan(take, wsum, &take_total);
    if (take && out_base + pos < (unsigned)k) sel[out_base + pos] = cs1 + i;
    out_base += take_total;
    eq_base += eq_total;
  }
}

template <typename Rows>
static void launch_score(const Geo& g, const Rows& rows, int score_layer, const void* k_fresh, float* scores,
                         hipStream_t s) {
  static_assert(sizeof(Rows) + 64 <= 4096, "kernel arguments within 4 KB");
  TraceScope tr("deviation_score", s);
  if (g.dtype == CS_BF16 && g.D == 128) {
    const int64_t blocks = (g.n + 15) / 16;
    hipLaunchKernelGGL(deviation_score_bf16_d128<Rows>, dim3((unsigned)blocks), dim3(256), 0, s, rows,
                       (const uint16_t*)k_fresh, scores, score_layer, g.n, g.cs1, g.Hkv);
  } else {
    const int64_t blocks = (g.n + 3) / 4;
    if (g.dtype == CS_BF16)
      hipLaunchKernelGGL((deviation_score<uint16_t, Rows>), dim3((unsigned)blocks), dim3(256), 0, s, rows,
                         (const uint16_t*)k_fresh, scores, score_layer, g.n, g.cs1, g.Hkv, g.D);
    else
      hipLaunchKernelGGL((deviation_score<float, Rows>), dim3((unsigned)blocks), dim3(256), 0, s, rows,
                         (const float*)k_fresh, scores, score_layer, g.n, g.cs1, g.Hkv, g.D);
  }
}

cs_status launch_score_select(const Geo& g, const CacheView& cv, int score_layer, const void* k_fresh, float* scores,
                              int32_t* sel, int64_t k_sel, hipStream_t s, bool check_only) {
  const bool fast = g.dtype == CS_BF16 && g.D == 128;
  cs_status st0 = check_grid(fast ? (g.n + 15) / 16 : (g.n + 3) / 4, 1, 1, 256, "deviation score");
  if (st0 || check_only) return st0;
  if (cv.paged) launch_score(g, cv.pages<kMaxPages>(g), score_layer, k_fresh, scores, s);
  else launch_score(g, cv.flat(g), score_layer, k_fresh, scores, s);
  cs_status st = check_launch("deviation score launch");
  if (st || k_sel == 0) return st;
  {
    TraceScope tr("radix_select_topk", s);
    hipLaunchKernelGGL(radix_select_topk, dim3(1), dim3(kSelThreads), 0, s, scores, (int)g.n, (int)k_sel,
                       (int)g.cs1, sel);
  }
  return check_launch("top-k select launch");
}

}  // namespace cs
