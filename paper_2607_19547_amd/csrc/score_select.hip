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
// ascending and exactly k long.  Up to 65,536 candidates the scores are read
// once into registers (64 per thread, a contiguous range each) and the
// compaction takes two workgroup scans; beyond that every pass re-reads them
// and each wavefront compacts a contiguous range.  All counts are order
// independent, so the result is deterministic.
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

constexpr int kSelBatch = 8;   // elements per thread (or lane) in flight
constexpr int kSelHeld = 64;   // elements a thread keeps in registers (n <= kSelHeld x kSelThreads)

// kHeld: n <= kSelHeld x kSelThreads, and wavefront w keeps the scores
// [64 kSelHeld w, 64 kSelHeld (w + 1)) in registers for all passes (lane l
// holds index 64 kSelHeld w + 64 j + l as its j-th value, so every load is
// coalesced); otherwise every pass re-reads the scores.  Either way each
// wavefront then compacts a contiguous range of indices.
template <bool kHeld>
__global__ __launch_bounds__(kSelThreads) void radix_select_topk(const float* __restrict__ scores,
                                                                 int n, int k, int cs1,
                                                                 int32_t* __restrict__ sel) {
  __shared__ unsigned hist[kSelWaves][256];
  __shared__ unsigned tot[4];  // per-wavefront totals of the digit scan
  __shared__ unsigned s_prefix, s_kk;
  __shared__ unsigned wgt[kSelWaves], weq[kSelWaves];
  const unsigned* bits = (const unsigned*)scores;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  // held slots past n carry 0xffffffff, a pattern with the sign bit set that
  // no score (all are >= 0) has, so it matches no prefix and is never above
  // or at the threshold (compared as signed integers)
  const int hb = 64 * kSelHeld * wave;  // first index this wavefront holds
  unsigned held[kHeld ? kSelHeld : 1];
  if constexpr (kHeld) {
#pragma unroll
    for (int j = 0; j < kSelHeld; ++j) {
      const int i = hb + 64 * j + lane;
      held[j] = i < n ? bits[i] : 0xffffffffu;
    }
  }
  // adds one element to this wavefront's histogram; when every counted lane
  // of the wavefront has the same digit (the common case in the high digits)
  // one lane adds for all of them
  auto count = [&](bool in, unsigned d) {
    const unsigned d0 = __builtin_amdgcn_readfirstlane(d);
    const unsigned long long act = __ballot(in);
    if (__ballot(in && d == d0) == act) {
      if (lane == __builtin_amdgcn_readfirstlane(lane) && act) atomicAdd(&hist[wave][d0], (unsigned)__popcll(act));
    } else if (in) {
      atomicAdd(&hist[wave][d], 1u);
    }
  };
  unsigned prefix = 0u, mask = 0u, kk = (unsigned)k;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int b = tid; b < kSelWaves * 256; b += kSelThreads) (&hist[0][0])[b] = 0u;
    __syncthreads();
    if constexpr (kHeld) {
#pragma unroll
      for (int j = 0; j < kSelHeld; ++j)
        if ((held[j] & (mask | 0x80000000u)) == prefix) atomicAdd(&hist[wave][(held[j] >> shift) & 255u], 1u);
    } else {
      for (int base = tid; base < n; base += kSelBatch * kSelThreads) {
        unsigned u[kSelBatch];
#pragma unroll
        for (int j = 0; j < kSelBatch; ++j) {
          const int i = base + j * kSelThreads;
          u[j] = i < n ? bits[i] : 0u;
        }
#pragma unroll
        for (int j = 0; j < kSelBatch; ++j)
          count(base + j * kSelThreads < n && (u[j] & mask) == prefix, (u[j] >> shift) & 255u);
      }
    }
    __syncthreads();
    // Thread b < 256 takes digit d = 255 - b: an inclusive scan over b gives
    // the count at or above d, and the one digit where that count first
    // reaches kk is the next digit of the k-th largest pattern.
    unsigned x = 0, p = 0;
    if (tid < 256) {
      const int d = 255 - tid;
#pragma unroll
      for (int w = 0; w < kSelWaves; ++w) x += hist[w][d];
      p = x;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const unsigned y = __shfl_up(p, o);
        if (lane >= o) p += y;
      }
      if (lane == 63) tot[wave] = p;
    }
    __syncthreads();
    if (tid < 256) {
      for (int w = 0; w < wave; ++w) p += tot[w];
      const unsigned above = p - x;
      if (above < kk && kk <= p) {
        s_prefix = prefix | ((unsigned)(255 - tid) << shift);
        s_kk = kk - above;
      }
    }
    __syncthreads();
    prefix = s_prefix;
    kk = s_kk;
    mask |= 255u << shift;
  }
  // prefix is now the k-th largest bit pattern; the first kk ties at it (in
  // index order) are taken.
  const unsigned thr = prefix;
  const unsigned long long below = (1ull << lane) - 1ull;
  if constexpr (kHeld) {
    // the held values in index order: j, then lane
    unsigned cgt = 0, ceq = 0;
#pragma unroll
    for (int j = 0; j < kSelHeld; ++j) {
      cgt += (int)held[j] > (int)thr;
      ceq += held[j] == thr;
    }
#pragma unroll
    for (int o = 32; o; o >>= 1) {
      cgt += __shfl_xor(cgt, o);
      ceq += __shfl_xor(ceq, o);
    }
    if (lane == 0) {
      wgt[wave] = cgt;
      weq[wave] = ceq;
    }
    __syncthreads();
    unsigned eq_run = 0, out_run = 0;  // ties and outputs before this wavefront's range
    for (int v = 0; v < wave; ++v) {
      out_run += wgt[v] + min(weq[v], kk > eq_run ? kk - eq_run : 0u);
      eq_run += weq[v];
    }
#pragma unroll
    for (int j = 0; j < kSelHeld; ++j) {
      const bool eq = held[j] == thr;
      const unsigned long long em = __ballot(eq);
      const bool take = (int)held[j] > (int)thr || (eq && eq_run + (unsigned)__popcll(em & below) < kk);
      const unsigned long long tm = __ballot(take);
      const unsigned pos = out_run + (unsigned)__popcll(tm & below);
      if (take && pos < (unsigned)k) sel[pos] = cs1 + hb + 64 * j + lane;
      out_run += (unsigned)__popcll(tm);
      eq_run += (unsigned)__popcll(em);
    }
  } else {
    // Wavefront w compacts the contiguous index range [w0, w1): a counting
    // pass, one exchange of per-wavefront counts, then a writing pass in
    // which ballots order the lanes.
    const int per_w = (n + kSelWaves - 1) / kSelWaves;
    const int w0 = min(n, wave * per_w), w1 = min(n, w0 + per_w);
    unsigned cgt = 0, ceq = 0;
    for (int b = w0; b < w1; b += 64 * kSelBatch) {
      unsigned u[kSelBatch];
#pragma unroll
      for (int j = 0; j < kSelBatch; ++j) {
        const int i = b + 64 * j + lane;
        u[j] = i < w1 ? bits[i] : 0u;
      }
#pragma unroll
      for (int j = 0; j < kSelBatch; ++j) {
        const bool ok = b + 64 * j + lane < w1;
        cgt += (unsigned)__popcll(__ballot(ok && u[j] > thr));
        ceq += (unsigned)__popcll(__ballot(ok && u[j] == thr));
      }
    }
    if (lane == 0) {
      wgt[wave] = cgt;
      weq[wave] = ceq;
    }
    __syncthreads();
    unsigned eq_run = 0, out_run = 0;  // ties and outputs before this wavefront's range
    for (int v = 0; v < wave; ++v) {
      out_run += wgt[v] + min(weq[v], kk > eq_run ? kk - eq_run : 0u);
      eq_run += weq[v];
    }
    for (int b = w0; b < w1; b += 64 * kSelBatch) {
      unsigned u[kSelBatch];
#pragma unroll
      for (int j = 0; j < kSelBatch; ++j) {
        const int i = b + 64 * j + lane;
        u[j] = i < w1 ? bits[i] : 0u;
      }
#pragma unroll
      for (int j = 0; j < kSelBatch; ++j) {
        const int i = b + 64 * j + lane;
        const bool ok = i < w1;
        const bool eq = ok && u[j] == thr;
        const unsigned long long em = __ballot(eq);
        const bool take = (ok && u[j] > thr) || (eq && eq_run + (unsigned)__popcll(em & below) < kk);
        const unsigned long long tm = __ballot(take);
        const unsigned pos = out_run + (unsigned)__popcll(tm & below);
        if (take && pos < (unsigned)k) sel[pos] = cs1 + i;
        out_run += (unsigned)__popcll(tm);
        eq_run += (unsigned)__popcll(em);
      }
    }
  }
}

template <typename Rows>
static void launch_score(const Geo& g, const Rows& rows, int score_layer, const void* k_fresh, float* scores,
                         hipStream_t s) {
  static_assert(sizeof(Rows) + 64 <= 4096, "kernel arguments within 4 KB");
  TraceScope tr("deviation_score", s);
  if (g.dtype == CS_BF16 && g.D == 128) {
    const int64_t blocks = (g.n + 15) / 16;
    CS_LAUNCH(tr, deviation_score_bf16_d128<Rows>, dim3((unsigned)blocks), dim3(256), 0, s, rows,
                       (const uint16_t*)k_fresh, scores, score_layer, g.n, g.cs1, g.Hkv);
  } else {
    const int64_t blocks = (g.n + 3) / 4;
    if (g.dtype == CS_BF16)
      CS_LAUNCH(tr, (deviation_score<uint16_t, Rows>), dim3((unsigned)blocks), dim3(256), 0, s, rows,
                         (const uint16_t*)k_fresh, scores, score_layer, g.n, g.cs1, g.Hkv, g.D);
    else
      CS_LAUNCH(tr, (deviation_score<float, Rows>), dim3((unsigned)blocks), dim3(256), 0, s, rows,
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
    if (g.n <= (int64_t)kSelHeld * kSelThreads)
      CS_LAUNCH(tr, radix_select_topk<true>, dim3(1), dim3(kSelThreads), 0, s, scores, (int)g.n, (int)k_sel,
                         (int)g.cs1, sel);
    else
      CS_LAUNCH(tr, radix_select_topk<false>, dim3(1), dim3(kSelThreads), 0, s, scores, (int)g.n,
                         (int)k_sel, (int)g.cs1, sel);
  }
  return check_launch("top-k select launch");
}

}  // namespace cs
