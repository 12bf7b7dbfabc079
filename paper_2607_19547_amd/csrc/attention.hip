// Scatter of fresh K/V rows and causal GQA attention of the selected rows
// (Eq. 1 and the repair step of Section 2).
//
// MFMA path (bf16, head_dim 128, G = H_q/H_kv dividing 32)
// ---------------------------------------------------------
// A row tile is one KV head and a run of consecutive selection slots.  Its 8
// wavefronts each hold 32 query vectors: 32/G selected rows x the G query
// heads that share the KV head, so every K/V tile staged in LDS serves 256
// query vectors.  Per 64-key tile a wavefront computes
//   S^T = K Q^T         (v_mfma_f32_32x32x16_bf16, K from LDS, Q in VGPRs)
// so each lane ends up holding 32 scores of ONE query; the softmax runs on
// those registers (exp2 with the 1/sqrt(D) and log2(e) factors folded into one
// FMA, a lazy running max that rescales only when the max grows by > 2^8),
// and the probabilities are packed to bf16 directly as the B operand of
//   O^T += V^T P^T      (V^T read from LDS with transposing loads).
// K/V tiles reach LDS by buffer->LDS DMA into a 4-slot ring: while the
// probabilities of tile i and the scores of tile i+1 are computed, tile i+3
// is fetched.  Rows are causal in cache order: key j is visible to row t iff
// j <= t; tiles below every row's limit skip the mask.
//
// Work is scheduled on the device: a planning workgroup (in the same launch
// as the scatter of the fresh rows) lists the (row tile, KV head, key piece)
// items, longest row tiles first, with a descriptor per item.  The attention
// launch is one resident workgroup per CU; each takes items from its queue
// through an atomic counter until every queue is empty, fetching the next
// item's first key tiles while the current item's results are written.  Row
// tiles too long for an even schedule are cut into key pieces whose partial
// (O, max, sum) a combine kernel merges in a fixed order, so results do not
// depend on timing.
//
// Generic path: one wavefront per (row, query head), float32 arithmetic, any
// head_dim <= 512 and either storage dtype.
#include <math.h>

#include <algorithm>
#include <type_traits>

#include "cs_common.h"

namespace cs {

// ============================================================== scatter
// K[layer][h][t] <- K_fresh[layer][h][t - s1] and the same for V, for every
// selected token t and every layer of the call; cache rows are reached through
// the row map.  W is the bytes one thread moves (16 when a row is a whole
// number of 16-byte words).  Work items first, first + stride, ...
struct ScatterArgs {
  const char* kf;
  const char* vf;
  const int32_t* sel;
  int64_t n_sel, T, n, cs1;
  int Hkv, row_bytes, lb, layers;
};

template <int W, typename Rows>
__device__ __forceinline__ void scatter_body(const Rows& rows, const ScatterArgs& a, int64_t first, int64_t stride) {
  typedef typename std::conditional<W == 16, u32x4, uint32_t>::type word;
  const int words = a.row_bytes / W;
  const int64_t per_layer = (int64_t)a.Hkv * a.n_sel * words;
  const int64_t total = per_layer * a.layers;
  for (int64_t w = first; w < total; w += stride) {
    const int lr = (int)(w / per_layer);
    const int64_t x = w - lr * per_layer;
    const int c = (int)(x % words);
    const int64_t hm = x / words;
    const int64_t m = hm % a.n_sel;
    const int h = (int)(hm / a.n_sel);
    const int layer = a.lb + lr;
    const int64_t t = a.sel[m];
    if (t < a.cs1 || t >= a.T) continue;  // out-of-contract index: never write outside the cache
    char *kr, *vr;
    rows.kv_rows((int64_t)layer * a.Hkv + h, t, a.row_bytes, kr, vr);
    const int64_t src = (((int64_t)layer * a.Hkv + h) * a.n + (t - a.cs1)) * a.row_bytes + W * c;
    *(word*)(kr + W * c) = *(const word*)(a.kf + src);
    *(word*)(vr + W * c) = *(const word*)(a.vf + src);
  }
}

template <int W, typename Rows>
__global__ __launch_bounds__(256) void scatter_rows(const Rows rows, const ScatterArgs a) {
  scatter_body<W>(rows, a, (int64_t)blockIdx.x * 256 + threadIdx.x, (int64_t)gridDim.x * 256);
}

static ScatterArgs scatter_args(const Geo& g, int lb, int le, const int32_t* sel, int64_t n_sel, const void* kf,
                                const void* vf) {
  ScatterArgs a;
  a.kf = (const char*)kf;
  a.vf = (const char*)vf;
  a.sel = sel;
  a.n_sel = n_sel;
  a.T = g.T;
  a.n = g.n;
  a.cs1 = g.cs1;
  a.Hkv = g.Hkv;
  a.row_bytes = g.D * g.esize;
  a.lb = lb;
  a.layers = le - lb;
  return a;
}
static int scatter_word(const ScatterArgs& a) { return a.row_bytes % 16 == 0 ? 16 : 4; }
static int64_t scatter_items(const ScatterArgs& a) {
  return (int64_t)a.Hkv * a.n_sel * (a.row_bytes / scatter_word(a)) * a.layers;
}

template <typename Rows>
static void launch_scatter_rows(const ScatterArgs& a, const Rows& rows, hipStream_t s) {
  static_assert(sizeof(Rows) + sizeof(ScatterArgs) <= 4096, "kernel arguments within 4 KB");
  const unsigned blocks = (unsigned)std::min<int64_t>((scatter_items(a) + 255) / 256, 65535);
  TraceScope tr("scatter_rows", s);
  if (scatter_word(a) == 16)
    CS_LAUNCH(tr, (scatter_rows<16, Rows>), dim3(blocks), dim3(256), 0, s, rows, a);
  else
    CS_LAUNCH(tr, (scatter_rows<4, Rows>), dim3(blocks), dim3(256), 0, s, rows, a);
}


// ============================================================== MFMA attention
constexpr int kKT = 64;                  // keys per tile
constexpr int kWaves = 8;                // wavefronts per workgroup (2 per SIMD)
constexpr int kThreads = 64 * kWaves;
constexpr int kQPerWG = 32 * kWaves;     // query vectors per workgroup
constexpr int kRow = 256;                // bytes of one K/V row (bf16 x 128)
constexpr int kHiLds = 65536;            // LDS bytes below the K ring (the V ring)
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kRescaleLog2 = 8.0f;     // lazy rescale threshold (max growth 2^8)

struct AttnArgs {
  const uint16_t* q;
  const int32_t* sel;
  uint16_t* out;
  float* lse;
  int* plan;       // work plan written by plan_items (see PlanView)
  uint16_t* part;  // [layers in call][part_cap][kQPerWG][128] partial O / sum / 2^e, fp16
  float* part_ml;  // [layers in call][part_cap][kQPerWG][4] running max (log2 units), sum, e
  int64_t T, n, n_sel, n_tiles;
  int cs1, Hq, Hkv, lb, layers;
  int part_cap;      // partial slots per layer
  int q_by_slot;     // q is [layers in call][H_q][n_sel][128] (rows in selection order), else [L][H_q][n][128]
  int desc_off;      // item descriptors in the plan (set by the planning kernel's caller)
  const float2* rope_tab;  // [n_sel][64] cos/sin of the selected tokens: q holds pre-rotary queries, rotated on
                           // load; NULL: q is already rotated
  float scale_log2;  // log2(e) / sqrt(D)
};

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// Lanes l and l^32 hold the same query: combine their values.
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// LDS tiles are row-major (one 256-byte row per key) with the 16-byte chunks
// of each row permuted so that the operand reads are free of bank conflicts:
//   K: chunk c of row r sits at position c ^ (r & 15)   (16 rows, same chunk)
//   V: chunk c of row r sits at position c ^ 4(r & 3)   (4 rows x 4 chunks)
// A 64-key tile (2 x 16 KB) is staged by buffer->LDS DMA: one wavefront
// instruction writes 1 KB = 4 rows, lane i landing at byte 16 i, so lane i
// fetches the global chunk that belongs at its position.  The buffer's
// hardware range check returns zeros for rows past the cache (those keys are
// masked).  Each ring slot is its own LDS variable, which lets the compiler
// see that reads of one slot do not wait for DMA into another.
typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t plane_rsrc(const char* base, int64_t rows) {
  return __builtin_amdgcn_make_buffer_rsrc((void*)base, 0, (int)(rows * kRow), 0x00020000);
}

struct StageOffsets {
  int k[2], v[2];  // byte offset of this lane's chunk within a tile, per instruction
};

__device__ __forceinline__ StageOffsets stage_offsets(int wave, int lane) {
  StageOffsets so;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = 4 * (2 * wave + j) + (lane >> 4);
    const int p = lane & 15;
    so.k[j] = row * kRow + 16 * (p ^ (row & 15));
    so.v[j] = row * kRow + 16 * (p ^ ((row & 3) << 2));
  }
  return so;
}

__device__ __forceinline__ void stage_dma(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv,
                                          const StageOffsets& so, int kt, char* Kd, char* Vd,
                                          int wave) {
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r0 = 4 * (2 * wave + j);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(Kd + r0 * kRow), 16, kt * kRow + so.k[j], 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(Vd + r0 * kRow), 16, kt * kRow + so.v[j], 0, 0, 0);
  }
}

// Work decomposition.  Row tiles are ordered longest first (they end at the
// highest selected tokens); row tile i needs n_i = ceil((g_last + 1) / 64)
// key tiles.  A row tile longer than the piece size S is cut into
// ceil(n_i / S) pieces at key tiles 0, S, 2S, ..., so piece j of every cut
// row tile covers the same keys.  An item is one piece of one row tile for
// one KV head.  Items sit in nq queues, queue j holding the KV heads
// kv = j (mod nq), and the workgroups of XCDs x = j (mod nq) take from queue
// j, so an XCD's L2 serves few KV heads; a workgroup whose queue is empty
// takes from the others, so XCDs that run faster take more.  Within a queue,
// the pieces of cut row tiles come first, piece-major (piece 0 of every cut
// row tile, then piece 1, ...: workgroups running side by side read the same
// keys, which the L2 then serves once), then the uncut row tiles, longest
// first; the last quarter is then reordered longest first, so a launch ends
// on its shortest items.  The pieces of a cut row tile leave partial (O, max,
// sum) in fixed workspace slots that sel_attn_combine merges in piece order.
constexpr int kPlanHdr = 32;    // header ints, see PlanView
constexpr int kPlanMagic = 0x43530231;  // marks a header the planning kernel wrote
constexpr int kPlanCUs = 256;   // CU count S is derived from (a constant: results do not depend on the device)
constexpr int kItemsPerCU = 6;  // target items per CU when row tiles must be cut
// Smallest piece: 16 key tiles.  Short caches and small rho leave few items
// per CU, and a launch then lasts as long as its longest item (measured: the
// 8,192-token composition at rho = 0.1 takes 3.04 ms with 16, 4.77 ms with
// 64; the 65,536-token one, whose pieces are ~137 tiles, is unchanged).
constexpr int kMinPiece = 16;
constexpr int kPartCap = 2560;  // partial slots per layer, at most
constexpr int kPlanLdsTiles = 4096;  // row tiles whose plan arrays the planning workgroup keeps in LDS
constexpr int kMaxPieces = 2048;     // most pieces of a row tile (the piece size is raised to keep to it)
constexpr int kPlanLdsPieces = kMaxPieces + 1;
constexpr int kPlanSortCap = 2048;   // longest tail (a quarter of a queue) the plan reorders
constexpr int kXcds = 8;

struct PlanView {
  int* hdr;   // [0, 8) queue counters, [8] nq, [9] S, [10] cut row tiles, [11] most pieces,
              // [12] items per queue and layer,
              // [14] offset of the item descriptors (ints from the plan's start);
              // [16, 24): what the plan was made from and its checksum (kPlanMagic,
              // n_tiles, RT, H_kv, part_cap, desc_off, two checksum words), [24] 1 when
              // the last planning launch reused the plan, 0 when it made it
  int* nu;    // [n_tiles] key tiles of row tile i (longest first)
  int* nsp;   // [n_tiles] pieces of row tile i
  int* ppre;  // [n_tiles + 1] first partial slot of row tile i (prefix sums of H_kv x pieces over cut row tiles)
  int* pj;    // [max_pieces + 1] first queue position of piece j (prefix sums of cut row tiles with > j pieces)
};
__host__ __device__ inline PlanView plan_view(int* base, int64_t n_tiles) {
  PlanView v;
  v.hdr = base;
  v.nu = base + kPlanHdr;
  v.nsp = v.nu + n_tiles;
  v.ppre = v.nsp + n_tiles;
  v.pj = v.ppre + n_tiles + 1;
  return v;
}
inline size_t plan_ints(int64_t n_tiles, int64_t max_pieces) {
  return kPlanHdr + 3 * (size_t)n_tiles + 1 + (size_t)max_pieces + 1;
}
// Queues: one per KV head (shared by 8/H_kv XCDs), one per XCD, or one.
__host__ __device__ inline int n_queues(int Hkv) {
  return Hkv % kXcds == 0 ? kXcds : (kXcds % Hkv == 0 ? Hkv : 1);
}

// Sum or max over the 1024 threads of the planning workgroup (every thread
// gets the result).
__device__ __forceinline__ int block_reduce(int v, bool is_max, int* red) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const int y = __shfl_xor(v, o);
    v = is_max ? max(v, y) : v + y;
  }
  __syncthreads();  // red may still be read by the previous call
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  int r = red[0];
  for (int w = 1; w < 16; ++w) r = is_max ? max(r, red[w]) : r + red[w];
  return r;
}

// Inclusive prefix sums (kMax: running maxima) of x over the 1024 threads,
// continuing from *base (shared); returns this thread's inclusive value and
// advances *base.
template <bool kMax = false>
__device__ __forceinline__ int block_scan(int x, int* wsum, int* base) {
  auto op = [](int u, int v) { return kMax ? max(u, v) : u + v; };
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x = op(x, y);
  }
  if (lane == 63) wsum[wave] = x;
  __syncthreads();
  int off = *base;
  for (int w = 0; w < wave; ++w) off = op(off, wsum[w]);
  __syncthreads();
  if (threadIdx.x == 1023) *base = op(off, x);
  __syncthreads();
  return op(off, x);
}

// Builds the work plan of one call (one workgroup of 1024 threads).  The
// plan's arrays are written and read back by different threads, always with
// a barrier between.
struct PlanArgs {
  const int32_t* sel;
  int64_t n_sel, n_tiles, T;
  int RT, Hkv, part_cap;
  int pj_cap, desc_cap;  // ints of the piece sections and item descriptors the workspace holds
  int desc_off;  // where the item descriptors start
  int* plan;
};
// Two checksum words over the plan's ints that the attention and combine
// kernels read (header [8, 16), pieces and partial slots per row tile, piece
// sections, item descriptors), each int weighted by its position: unsigned
// sums, so the order of the terms does not matter.
__device__ __forceinline__ uint2 plan_checksum(const int* plan, int64_t n_tiles, int nj, int desc_off, int per_q,
                                               unsigned* red) {
  unsigned c1 = 0, c2 = 0;
  auto add = [&](int64_t b, int64_t e) {
    for (int64_t i = b + threadIdx.x; i < e; i += 1024) {
      const unsigned v = (unsigned)plan[i], x = (unsigned)i;
      c1 += v * (2u * x + 1u);
      c2 += (v ^ (x * 0x9E3779B9u)) * 0x85EBCA6Bu + x;
    }
  };
  const PlanView pv = plan_view(const_cast<int*>(plan), n_tiles);
  add(8, 16);
  add(pv.nsp - plan, pv.pj - plan);  // nsp and ppre
  add(pv.pj - plan, pv.pj - plan + nj + 1);
  add(desc_off, desc_off + 4 * (int64_t)per_q);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    c1 += (unsigned)__shfl_xor((int)c1, o);
    c2 += (unsigned)__shfl_xor((int)c2, o);
  }
  __syncthreads();  // red may still be read by an earlier reduction
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6] = c1;
    red[16 + (threadIdx.x >> 6)] = c2;
  }
  __syncthreads();
  uint2 r = make_uint2(0u, 0u);
  for (int w = 0; w < 16; ++w) {
    r.x += red[w];
    r.y += red[16 + w];
  }
  return r;
}

__device__ void plan_body(const PlanArgs& p) {
  const int32_t* __restrict__ sel = p.sel;
  const int64_t n_sel = p.n_sel, n_tiles = p.n_tiles, T = p.T;
  const int RT = p.RT, Hkv = p.Hkv, part_cap = p.part_cap, desc_off = p.desc_off;
  int* __restrict__ plan = p.plan;
  __shared__ int red[16];
  __shared__ unsigned red_u[32];
  __shared__ int wsum[16];
  __shared__ int s_base;
  // the arrays the plan reads back live in LDS when they fit (global memory
  // otherwise); nsp is also written to the plan for the attention kernels
  __shared__ int l_nu[kPlanLdsTiles], l_nsp[kPlanLdsTiles], l_pj[kPlanLdsPieces];
  __shared__ int4 l_desc[kPlanSortCap];  // the reordered tail's descriptors (earlier, the piece counts)
  const PlanView pv = plan_view(plan, n_tiles);
  const bool in_lds = n_tiles <= kPlanLdsTiles;
  int* const nu = in_lds ? l_nu : pv.nu;
  int* const nsp = in_lds ? l_nsp : pv.nsp;
  const int tid = threadIdx.x;
  // Key tiles of row tile t: up to its last row's token, taken as a running
  // maximum over t.  For an ascending selection the maximum changes nothing;
  // for any other list it keeps n_i non-increasing along the longest-first
  // order, which the placement of the items below relies on (the cut row
  // tiles lead, and every queue position is written exactly once).
  //
  // The plan is a function of these counts and of n_tiles, RT, H_kv, part_cap
  // and desc_off alone.  The workspace may still hold the plan of an earlier
  // call (the layer calls of one composition share their selection): when it
  // was made from the same counts and sizes and its checksum holds, it is
  // kept and only its claim counters are cleared.  The counts are kept in the
  // plan for that comparison.
  int sum = 0, diff = 0;
  if (tid == 0) s_base = 0;
  __syncthreads();
  for (int64_t b = 0; b < n_tiles; b += 1024) {
    const int64_t t = b + tid;
    int v = 1;
    if (t < n_tiles) {
      const int64_t ml = min((t + 1) * RT, n_sel) - 1;
      const int64_t g = min((int64_t)sel[ml], T - 1);
      v = g < 0 ? 1 : (int)((g + kKT) / kKT);
    }
    v = block_scan<true>(v, wsum, &s_base);
    if (t < n_tiles) {
      const int64_t i = n_tiles - 1 - t;
      diff |= pv.nu[i] != v;  // (the stored count, read before it is replaced)
      pv.nu[i] = v;
      if (in_lds) l_nu[i] = v;
      sum += v;
    }
  }
  const int nmax = s_base;  // (block_scan ends on a barrier)
  const int W1 = block_reduce(sum, false, red);
  {
    const int* hdr = pv.hdr;  // (every thread reads the same values: the decision is uniform)
    bool same = block_reduce(diff, true, red) == 0 && hdr[16] == kPlanMagic && hdr[17] == n_tiles &&
                hdr[18] == RT && hdr[19] == Hkv && hdr[20] == part_cap && hdr[21] == desc_off;
    if (same) {
      const int nj_s = hdr[11], per_q_s = hdr[12];
      same = nj_s >= 0 && nj_s < p.pj_cap && per_q_s >= 0 && 4 * (int64_t)per_q_s <= p.desc_cap;
      if (same) {
        const uint2 c = plan_checksum(plan, n_tiles, nj_s, desc_off, per_q_s, red_u);
        same = c.x == (unsigned)hdr[22] && c.y == (unsigned)hdr[23];
      }
    }
    if (same) {
      __syncthreads();  // every thread has read the header
      if (tid < kXcds) pv.hdr[tid] = 0;  // the queues' claim counters
      if (tid == 0) pv.hdr[24] = 1;
      return;
    }
  }
  // piece size: about kItemsPerCU items per CU, raised until the partial
  // slots fit in part_cap (no cut at all always fits)
  const int64_t per = (int64_t)kPlanCUs * kItemsPerCU;
  const int S0 = (int)max<int64_t>(max(kMinPiece, (nmax + kMaxPieces - 1) / kMaxPieces), ((int64_t)W1 * Hkv + per - 1) / per);
  int S = nmax;
  if (S0 < nmax) {
    // the cut row tiles fill at most ceil(W1 / S0) + n_tiles slots per KV
    // head; when that fits, so does the exact count below, which then
    // settles on S0 at once
    if (((W1 + (int64_t)S0 - 1) / S0 + n_tiles) * Hkv <= part_cap) {
      S = S0;
    } else {
      const int step = max(1, S0 / 8);
      for (int k = 0; k < 64; ++k) {
        const int Sk = S0 + k * step;
        if (Sk >= nmax) break;
        int loc = 0;
        for (int64_t i = tid; i < n_tiles; i += 1024) {
          const int v = nu[i];
          if (v > Sk) loc += (v + Sk - 1) / Sk;
        }
        if ((int64_t)block_reduce(loc, false, red) * Hkv <= part_cap) {
          S = Sk;
          break;
        }
      }
    }
  }
  // pieces per row tile (non-increasing along the longest-first order, as
  // n_i is), partial slots of the cut ones
  if (tid == 0) s_base = 0;
  __syncthreads();
  for (int64_t b = 0; b < n_tiles; b += 1024) {
    const int64_t i = b + tid;
    int np = 1;
    if (i < n_tiles) {
      const int v = nu[i];
      np = v > S ? (v + S - 1) / S : 1;
      nsp[i] = np;
      if (in_lds) pv.nsp[i] = np;
    }
    const int inc = block_scan(np > 1 ? np * Hkv : 0, wsum, &s_base);
    if (i < n_tiles) pv.ppre[i + 1] = inc;
  }
  // (block_scan ends on a barrier: every nsp is written)  Most pieces:
  // nsp[0].  cnt_j, the cut row tiles with more than max(j, 1) pieces, is
  // where nsp drops to max(j, 1) or below: the row tile before each drop
  // writes the counts of the j it passes (every j in [1, nj) exactly once).
  // The counts live in l_desc's LDS until the descriptors are placed.
  int* const l_cnt = (int*)l_desc;
  const int np_max = nsp[0];
  const int nj = np_max > 1 ? np_max : 0;
  for (int64_t i = tid; i < n_tiles; i += 1024) {
    const int a = nsp[i], a_next = i + 1 < n_tiles ? nsp[i + 1] : 1;
    for (int j = max(a_next, 1); j < a; ++j) l_cnt[j] = (int)(i + 1);
  }
  // queue positions of piece j: pj[j] = (cnt_0 + ... + cnt_{j-1}) x KV heads per queue
  const int nq = n_queues(Hkv), kvq = Hkv / nq;
  if (tid == 0) s_base = 0;
  __syncthreads();
  for (int b = 0; b < nj; b += 1024) {
    const int j = b + tid;
    const int inc = block_scan(j < nj ? l_cnt[max(j, 1)] * kvq : 0, wsum, &s_base);
    if (j < nj) pv.pj[j + 1] = l_pj[j + 1] = inc;
  }
  const int n_cut = nj > 1 ? l_cnt[1] : 0;  // (read before l_desc takes descriptors)
  if (tid == 0) {
    const int per_q = s_base + (int)(n_tiles - n_cut) * kvq;
    pv.ppre[0] = 0;
    pv.pj[0] = l_pj[0] = 0;
    for (int k = 0; k < kXcds; ++k) pv.hdr[k] = 0;  // the queues' claim counters
    pv.hdr[8] = nq;
    pv.hdr[9] = S;
    pv.hdr[10] = n_cut;
    pv.hdr[11] = nj;
    pv.hdr[12] = per_q;
    pv.hdr[14] = desc_off;
  }
  // Item descriptors, one per queue position (the same in every queue and
  // layer): {row tile, KV head in the queue | piece << 16, first and last key
  // tile of the piece}.  Cut row tiles are a prefix of the longest-first order,
  // so piece j of row tile i sits at pj[j] + kvl * cnt_j + i; uncut row tile i
  // at pj[nj] + kvl * (uncut count) + i - (cut count).  One thread per
  // position.  The last quarter of the queue (the part handed out last) is
  // reordered longest first, so the launch ends on its shortest items; the
  // order of equal lengths is immaterial (an item's descriptor alone fixes
  // its work and its output slots).
  __shared__ int l_bkt[256];
  if (tid < 256) l_bkt[tid] = 0;
  __syncthreads();
  int4* desc = (int4*)(plan + desc_off);
  const int p_end = s_base;
  const int nun = (int)(n_tiles - n_cut);
  const int per_q_all = p_end + nun * kvq;
  const int r0 = per_q_all - (per_q_all + 3) / 4;
  const bool sort_tail = per_q_all - r0 <= kPlanSortCap;
  auto put = [&](int pos, int4 d) {
    if (sort_tail && pos >= r0) l_desc[pos - r0] = d;
    else desc[pos] = d;
  };
  for (int pos = tid; pos < per_q_all; pos += 1024) {
    if (pos < p_end) {
      int lo = 0, up = nj;  // piece j: the last section starting at or before pos
      while (up - lo > 1) {
        const int mid = (lo + up) >> 1;
        if (l_pj[mid] <= pos) lo = mid;
        else up = mid;
      }
      const int cnt = (l_pj[lo + 1] - l_pj[lo]) / kvq;
      const int r = pos - l_pj[lo], kvl = r / cnt, i = r - kvl * cnt;
      const int b = lo * S, e = min((lo + 1) * S, nu[i]);  // the same key range for piece j of every row tile
      put(pos, make_int4(i, kvl | (lo << 16), b, e));
    } else {
      const int r = pos - p_end, kvl = r / nun, i = n_cut + (r - kvl * nun);
      put(pos, make_int4(i, kvl, 0, nu[i]));
    }
  }
  if (sort_tail) {  // (uniform)
    // counting sort of the tail by length (at most S key tiles), longest
    // first, in 256 buckets
    __syncthreads();
    const int nt = per_q_all - r0;
    int shift = 0;
    while ((S >> shift) > 255) ++shift;
    auto bucket = [&](int4 d) { return 255 - min((d.w - d.z) >> shift, 255); };
    for (int t = tid; t < nt; t += 1024) atomicAdd(&l_bkt[bucket(l_desc[t])], 1);
    __syncthreads();
    if (tid < 64) {  // exclusive scan of the 256 bucket counts by one wavefront
      int c4[4], tot = 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) tot += c4[q] = l_bkt[4 * tid + q];
      int incl = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(incl, o);
        if (tid >= o) incl += y;
      }
      int run = incl - tot;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        l_bkt[4 * tid + q] = run;
        run += c4[q];
      }
    }
    __syncthreads();
    for (int t = tid; t < nt; t += 1024) {
      const int4 d = l_desc[t];
      desc[r0 + atomicAdd(&l_bkt[bucket(d)], 1)] = d;
    }
  }
  // what the plan was made from, and its checksum, for the next call to compare
  __syncthreads();  // every part of the plan is written
  const uint2 c = plan_checksum(plan, n_tiles, nj, desc_off, per_q_all, red_u);
  if (tid == 0) {
    pv.hdr[16] = kPlanMagic;
    pv.hdr[17] = (int)n_tiles;
    pv.hdr[18] = RT;
    pv.hdr[19] = Hkv;
    pv.hdr[20] = part_cap;
    pv.hdr[21] = desc_off;
    pv.hdr[22] = (int)c.x;
    pv.hdr[23] = (int)c.y;
    pv.hdr[24] = 0;
  }
}

__global__ __launch_bounds__(1024) void plan_items(const PlanArgs p) {
  plan_body(p);
}

// The plan (workgroup 0) and the scatter of the call's fresh rows (the other
// workgroups) in one launch: the two are independent, and the attention that
// follows needs both.
template <int W, typename Rows>
__global__ __launch_bounds__(1024) void plan_scatter(const PlanArgs p, const Rows rows, const ScatterArgs sa) {
  if (blockIdx.x == 0) {
    plan_body(p);
    return;
  }
  scatter_body<W>(rows, sa, (int64_t)(blockIdx.x - 1) * 1024 + threadIdx.x, (int64_t)(gridDim.x - 1) * 1024);
}

// The fused rotary scatter (Eq. 2 at the global coordinates p' of the
// repair step): a workgroup takes kPrTok selected tokens of one layer, builds
// their cos/sin table in LDS (angles in float64, reduced modulo 2*pi, rounded
// to float32, as the re-basing kernels do; the call's first layer also keeps
// it in the workspace for the attention's queries), rotates their fresh keys
// into the cache rows and copies their fresh values.  Eight lanes per row,
// each holding the pairs (8j .. 8j+7) and (64 + 8j .. 64 + 8j+7).
constexpr int kPrTok = 32;   // selected tokens per workgroup
constexpr int kPrTabW = 65;  // LDS table row stride (float2): one pad entry spreads the banks
struct RopeRowsArgs {
  const uint16_t* k_pre;  // [L][H_kv][n][128]
  const uint16_t* v_new;  // [L][H_kv][n][128]
  const int32_t* sel;
  const int32_t* coords;  // [T][3]
  float2* tab;            // [n_sel][64]
  int64_t T, n, n_sel, cs1;
  int Hkv, lb, nblk;      // nblk: workgroups per layer
  int sec0, sec01;
  double theta[64];
};

template <typename Rows>
__device__ void rope_rows_body(const RopeRowsArgs& a, const Rows& rows, int blk, int lrel) {
  __shared__ float2 tab[kPrTok * kPrTabW];
  __shared__ int tok_of[kPrTok];
  const int tid = threadIdx.x;
  const int64_t m0 = (int64_t)blk * kPrTok;
  const int nm = (int)min<int64_t>(kPrTok, a.n_sel - m0);
  const int layer = a.lb + lrel;
  if (tid < kPrTok) {
    int t = -1;
    if (tid < nm) {
      const int64_t g = a.sel[m0 + tid];
      if (g >= a.cs1 && g < a.T) t = (int)g;  // out-of-contract index: the row is skipped
    }
    tok_of[tid] = t;
  }
  __syncthreads();
  for (int e = tid; e < kPrTok * 64; e += 1024) {
    const int r = e >> 6, i = e & 63;
    const int t = tok_of[r];
    float2 cs = make_float2(1.f, 0.f);
    if (t >= 0) cs = cos_sin_of((double)a.coords[(int64_t)t * 3 + axis_of(i, a.sec0, a.sec01)] * a.theta[i]);
    tab[r * kPrTabW + i] = cs;
    if (lrel == 0 && r < nm) a.tab[(m0 + r) * 64 + i] = cs;
  }
  __syncthreads();
  const int j = tid & 7;
  const int total = kPrTok * 2 * a.Hkv;  // rows: K of each KV head (rotated), then V (copied)
  for (int idx = tid >> 3; idx < total; idx += 128) {
    const int r = idx % kPrTok, kind = idx / kPrTok;
    const int t = tok_of[r];
    if (t < 0) continue;
    const bool is_k = kind < a.Hkv;
    const int h = is_k ? kind : kind - a.Hkv;
    const uint16_t* src = (is_k ? a.k_pre : a.v_new) + (((int64_t)layer * a.Hkv + h) * a.n + (t - a.cs1)) * 128;
    uint16_t* dst = (uint16_t*)rows.row(!is_k, (int64_t)layer * a.Hkv + h, t, 256);
    u32x4 wa = *(const u32x4*)(src + 8 * j), wb = *(const u32x4*)(src + 64 + 8 * j);
    if (is_k) {
      float c[8], sn[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float2 v = tab[r * kPrTabW + 8 * j + e];
        c[e] = v.x;
        sn[e] = v.y;
      }
      rotate8(wa, wb, c, sn);
    }
    *(u32x4*)(dst + 8 * j) = wa;
    *(u32x4*)(dst + 64 + 8 * j) = wb;
  }
}

// The plan (workgroup 0) and the fused rotary scatter of the call's fresh rows
// (the other workgroups: layer (b - 1) / nblk, tokens of block (b - 1) % nblk).
template <typename Rows>
__global__ __launch_bounds__(1024) void plan_rope_scatter(const PlanArgs p, const Rows rows, const RopeRowsArgs ra) {
  if (blockIdx.x == 0) {
    plan_body(p);
    return;
  }
  const int b = blockIdx.x - 1;
  rope_rows_body(ra, rows, b % ra.nblk, b / ra.nblk);
}

template <int G, typename Rows>
__global__ __launch_bounds__(kThreads) void sel_attn_mfma(const AttnArgs a, const Rows rows) {
  constexpr bool kPaged = !std::is_same<Rows, FlatRows>::value;
  constexpr int RW = 32 / G;       // selected rows per wavefront
  constexpr int RT = kWaves * RW;  // selected rows per workgroup tile
  // The V ring takes the low 64 KB of LDS, where the DS instruction's 16-bit
  // offset reaches every V operand read; the K ring above is read through
  // per-lane bases that carry the extra 64 KB (see koff).  LDS variables are
  // laid out in name order, hence lo_* below up_*.  (Any layout computes the
  // same; this one saves an address add per operand read.)
  __shared__ __attribute__((aligned(1024))) char lo_v0[kKT * kRow], lo_v1[kKT * kRow], lo_v2[kKT * kRow], lo_v3[kKT * kRow];
  __shared__ __attribute__((aligned(1024))) char up_k0[kKT * kRow], up_k1[kKT * kRow], up_k2[kKT * kRow], up_k3[kKT * kRow];
  auto kbuf = [&](auto B) -> char* {
    if constexpr (decltype(B)::value == 0) return up_k0;
    else if constexpr (decltype(B)::value == 1) return up_k1;
    else if constexpr (decltype(B)::value == 2) return up_k2;
    else return up_k3;
  };
  auto vbuf = [&](auto B) -> char* {
    if constexpr (decltype(B)::value == 0) return lo_v0;
    else if constexpr (decltype(B)::value == 1) return lo_v1;
    else if constexpr (decltype(B)::value == 2) return lo_v2;
    else return lo_v3;
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;

  // The workgroup stays resident and takes items one after another from its
  // XCD's queue (then from the others'), through one atomic counter per
  // queue.  The next item is claimed during an item's last key tiles and
  // started (its descriptor and first two key tiles) before the item's
  // results are written; its first two key tiles are fetched before its
  // queries are loaded.
  //
  // Registers are the limit of this kernel (two wavefronts per SIMD), so
  // nothing that only the per-item code needs is kept in registers across the
  // tile loop: the item's fields sit in LDS, the kernel arguments are read
  // again from the argument segment, and lane-derived addresses are formed
  // from a lane index read afresh (an opaque value the compiler cannot hoist
  // out of the item loop).
  __shared__ int s_claim[2];
  __shared__ int s_it[8];  // the current item: layer in call, row tile, KV head, piece, first and end key
  typedef const __attribute__((address_space(4))) AttnArgs* ArgPtr;  // the argument segment (scalar loads)
  const ArgPtr argp = (ArgPtr)__builtin_amdgcn_kernarg_segment_ptr();
  auto args = [&]() -> AttnArgs {  // the arguments, read anew where they are used
    ArgPtr p = argp;
    asm volatile("" : "+s"(p));
    return *(const AttnArgs*)p;
  };
  auto it_field = [&](int k) { return __builtin_amdgcn_readfirstlane(s_it[k]); };  // (uniform)
  auto lane_id = []() {
    int l;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
    return l;
  };
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int jq;  // this workgroup's queue: workgroup b runs on XCD b mod 8, and the XCDs x = j (mod nq) share queue j
  {
    const PlanView pv = plan_view(a.plan, a.n_tiles);
    jq = (blockIdx.x % kXcds) % pv.hdr[8];
  }
  // A claim: the queue position got from this workgroup's queue, or, past
  // its end, the next queue's first free position (whole workgroup; thread 0
  // claims).  -1 when every queue is empty.
  auto claim_rest = [&](const AttnArgs& A, int got) -> int {
    const PlanView pv = plan_view(A.plan, A.n_tiles);
    const int nq = pv.hdr[8], total_q = pv.hdr[12] * A.layers;
    if (tid == 0) {
      int j = jq;
      for (int t = 1; got >= total_q && t < nq; ++t) {
        j = j + 1 == nq ? 0 : j + 1;
        got = atomicAdd(&pv.hdr[j], 1);
      }
      s_claim[0] = got < total_q ? got : -1;
      s_claim[1] = j;
    }
    __syncthreads();
    const int it = __builtin_amdgcn_readfirstlane(s_claim[0]);
    jq = __builtin_amdgcn_readfirstlane(s_claim[1]);
    __syncthreads();  // s_claim is reused by the next claim
    return it;
  };
  // Thread 0's claim of the next queue position, read later: the lane offset
  // the compiler cannot see is zero keeps it from turning the add into a
  // wavefront-wide atomic whose result it reads (and waits for) at once.
  auto claim_add = [&](int* ctr) -> int {
    int z;
    asm volatile("v_mov_b32 %0, 0" : "=v"(z));
    return atomicAdd(ctr + z, 1);
  };
  auto claim_one = [&](const AttnArgs& A) -> int {
    int got = 0;
    if (tid == 0) got = atomicAdd(&plan_view(A.plan, A.n_tiles).hdr[jq], 1);
    return claim_rest(A, got);
  };

  // Key tiles are fetched in ascending order.  A contiguous cache is one
  // buffer range per plane; in a paged cache every 64-key tile lies inside one
  // chunk (chunk starts are multiples of 64), and the range follows the chunk
  // of the tile being fetched.  Rows past a range read as zeros.
  const StageOffsets so = stage_offsets(wave, tid & 63);
  __amdgpu_buffer_rsrc_t rk, rv;
  int dma_c = 0, dma_first = 0, dma_next = 0x7fffffff;
  int64_t dma_plane = 0;
  auto use_chunk = [&](int c) {
    if constexpr (kPaged) {
      const int s0 = rows.start[c], len = rows.start[c + 1] - s0;
      rk = plane_rsrc(rows.k[c] + dma_plane * len * kRow, len);
      rv = plane_rsrc(rows.v[c] + dma_plane * len * kRow, len);
      dma_c = c;
      dma_first = s0;
      dma_next = c + 1 < rows.n ? rows.start[c + 1] : 0x7fffffff;
    }
  };
  auto fetch = [&](int kt, char* Kd, char* Vd) {
    if constexpr (kPaged) {
      if (kt >= dma_next) {
        int c = dma_c + 1;
        while (c + 1 < rows.n && rows.start[c + 1] <= kt) ++c;
        use_chunk(c);
      }
    }
    stage_dma(rk, rv, so, kt - dma_first, Kd, Vd, wave);
  };
  // An item's fields from its descriptor {row tile (longest-first order), KV
  // head in the queue | piece << 16, key tiles [b, e)} into s_it (thread 0),
  // then the buffer ranges of its plane and its key tiles 0 and 1 into ring
  // slots 0 and 1.  False for a damaged plan entry (never for a plan the
  // planning kernel wrote).
  auto start_item = [&](const AttnArgs& A, int item) -> bool {
    const PlanView pv = plan_view(A.plan, A.n_tiles);
    const int per_q = pv.hdr[12], nq = pv.hdr[8];
    const int lrel = item / per_q;
    const int4 dsc = *(const int4*)(A.plan + A.desc_off + 4 * (item - lrel * per_q));
    const int oi = dsc.x, kv = (dsc.y & 0xffff) * nq + jq;
    if (oi < 0 || oi >= A.n_tiles || kv >= A.Hkv || dsc.z < 0 || dsc.w < dsc.z) return false;
    const int key_begin = (int)min((int64_t)dsc.z * kKT, A.T);
    if (tid == 0) {
      s_it[0] = lrel;
      s_it[1] = oi;
      s_it[2] = kv;
      s_it[3] = dsc.y >> 16;
      s_it[4] = key_begin;
      s_it[5] = (int)min((int64_t)dsc.w * kKT, A.T);  // the last tile holds the row tile's last token
    }
    dma_plane = (int64_t)(A.lb + lrel) * A.Hkv + kv;
    if constexpr (kPaged) {
      use_chunk(__builtin_amdgcn_readfirstlane(rows.chunk_of(key_begin)));
    } else {
      rk = plane_rsrc(rows.k + dma_plane * A.T * kRow, A.T);
      rv = plane_rsrc(rows.v + dma_plane * A.T * kRow, A.T);
    }
    fetch(key_begin, up_k0, lo_v0);
    fetch(key_begin + kKT, up_k1, lo_v1);
    return true;
  };
  auto begin_next = [&](const AttnArgs& A, int got) {  // claims until an item starts; false when none is left
    int item = claim_rest(A, got);
    while (item >= 0 && !start_item(A, item)) item = claim_one(A);
    return item >= 0;
  };

  // per-lane LDS offsets of the MFMA operands
  int koff[8];  // K: row q, chunk 2s + hi  (row 32 + q has the same swizzle), plus kHiLds
  const int lane = tid & 63, q = lane & 31, hi = lane >> 5;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    koff[s] = q * kRow + 16 * ((2 * s + hi) ^ (q & 15));
    // opaque to constant folding, so that each read keeps this register as
    // its base and puts (slot - kHiLds) in the instruction's offset field
    asm("v_add_u32 %0, 0x10000, %1" : "=v"(koff[s]) : "v"(koff[s]));
  }
  const int L = lane & 15, dh = (lane >> 4) & 1;
  int voff[4];  // V transposing reads: rows 4hi + L/4 (+16ks, +8), dims 32d + 16dh + 4(L%4)
#pragma unroll
  for (int d = 0; d < 4; ++d)
    voff[d] = (4 * hi + (L >> 2)) * kRow + 16 * ((4 * d + 2 * dh + ((L & 3) >> 1)) ^ ((L >> 2) << 2)) + 8 * (L & 1);
  const float sc = a.scale_log2;
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

  if (!begin_next(a, tid == 0 ? atomicAdd(&plan_view(a.plan, a.n_tiles).hdr[jq], 1) : 0)) return;  // every queue is empty
  __syncthreads();  // s_it is written
  int got = 0;      // thread 0: the next claim, made during the item's last key tiles

  while (true) {
    int g_q = -1, g_wmin, g_wmax, key_begin, n_kt;
    bf16x8 qb[8];
    {
      const AttnArgs A = args();
      key_begin = it_field(4);
      const int lrel = it_field(0), oi = it_field(1), kv = it_field(2);
      const int key_end = it_field(5);
      n_kt = key_end > key_begin ? (key_end - key_begin + kKT - 1) / kKT : 0;
      const int ln = lane_id(), lq = ln & 31;
      const int64_t m = (A.n_tiles - 1 - oi) * RT + wave * RW + lq / G;
      const int h = kv * G + lq % G;
      // the selected token is loaded before key tile 2's DMA is issued, so
      // that the wait for it (and the query load behind it) does not also
      // wait for that DMA
      const int t = A.sel[min<int64_t>(m, A.n_sel - 1)];
      asm volatile("" ::: "memory");
      fetch(key_begin + 2 * kKT, up_k2, lo_v2);
      if (m < A.n_sel && t >= A.cs1 && t < A.T) g_q = t;
      // the wavefront's smallest and largest token: masking starts at the
      // tile that reaches past the smallest, arithmetic stops after the largest
      g_wmin = g_q >= 0 ? g_q : 0x7fffffff;
      g_wmax = g_q;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) {
        g_wmin = min(g_wmin, __shfl_xor(g_wmin, o));
        g_wmax = max(g_wmax, __shfl_xor(g_wmax, o));
      }
      g_wmin = __builtin_amdgcn_readfirstlane(g_wmin);
      g_wmax = __builtin_amdgcn_readfirstlane(g_wmax);
      if (g_q >= 0) {
        const int64_t qrow = A.q_by_slot ? ((int64_t)lrel * A.Hq + h) * A.n_sel + m
                                         : ((int64_t)(A.lb + lrel) * A.Hq + h) * A.n + (g_q - A.cs1);
        const uint16_t* qp = A.q + qrow * 128 + 8 * (ln >> 5);
#pragma unroll
        for (int s = 0; s < 8; ++s) qb[s] = *(const bf16x8*)(qp + 16 * s);
        if (A.rope_tab) {
          // pre-rotary query: qb[s] and qb[s + 4] hold elements d and d + 64
          // of the same rotary pairs (d = 16s + 8hi + x), rotated here with the
          // selected token's cos/sin (Eq. 2 at p') and rounded to bf16
          const float2* tb = A.rope_tab + m * 64 + 8 * (ln >> 5);
#pragma unroll
          for (int s = 0; s < 4; ++s) {
            float c[8], sn[8];
#pragma unroll
            for (int x = 0; x < 8; ++x) {
              const float2 v = tb[16 * s + x];
              c[x] = v.x;
              sn[x] = v.y;
            }
            u32x4 wa = __builtin_bit_cast(u32x4, qb[s]), wb = __builtin_bit_cast(u32x4, qb[s + 4]);
            rotate8(wa, wb, c, sn);
            qb[s] = __builtin_bit_cast(bf16x8, wa);
            qb[s + 4] = __builtin_bit_cast(bf16x8, wb);
          }
        }
      } else {
#pragma unroll
        for (int s = 0; s < 8; ++s) qb[s] = bf16x8{};
      }
    }

    f32x16 o[4];
#pragma unroll
    for (int d = 0; d < 4; ++d) o[d] = f32x16{};
    float m_use = -INFINITY, l_run = 0.f;

    // S^T = K Q^T for the tile in LDS buffer B
    auto qk = [&](auto B, f32x16& s0, f32x16& s1) {
      const char* K = kbuf(B);
      s0 = f32x16{};
      s1 = f32x16{};
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const bf16x8 k0 = *(const bf16x8*)(K - kHiLds + koff[s]);
        const bf16x8 k1 = *(const bf16x8*)(K - kHiLds + 32 * kRow + koff[s]);
        s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qb[s], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qb[s], s1, 0, 0, 0);
      }
    };

    // Causal mask and running max of the tile starting at key kt; rescales the
    // accumulators when the max grew by more than 2^8.
    auto mask_max = [&](int kt, f32x16& s0, f32x16& s1) {
      // accumulator register r of block b holds key kt + 32b + 8(r/4) + 4hi + r%4
      if (kt + kKT - 1 > g_wmin) {
        const int lim = g_q - kt - 4 * hi;
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int off = 8 * (rr >> 2) + (rr & 3);
          if (off > lim) s0[rr] = -INFINITY;
          if (off + 32 > lim) s1[rr] = -INFINITY;
        }
      }
      // max tree of three-input maxima (16 instructions), eight independent chains first
      float t8[8];
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) t8[rr] = fmaxf(fmaxf(s0[rr], s0[rr + 8]), s1[rr]);
      float t4[4];
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) t4[rr] = fmaxf(fmaxf(t8[2 * rr], t8[2 * rr + 1]), s1[rr + 8]);
      const float t2a = fmaxf(fmaxf(t4[0], t4[1]), s1[12]), t2b = fmaxf(fmaxf(t4[2], t4[3]), s1[13]);
      const float mx = fmaxf(fmaxf(fmaxf(t2a, t2b), s1[14]), s1[15]);
      const float mt = pair_max(mx) * sc;
      const bool need = mt > m_use + kRescaleLog2;
      if (__ballot(need)) {
        const float m_new = need ? mt : m_use;
        const float alpha = need ? __builtin_amdgcn_exp2f(m_use - m_new) : 1.f;
        l_run *= alpha;
#pragma unroll
        for (int d = 0; d < 4; ++d) o[d] *= alpha;
        m_use = m_new;
      }
    };

    // Probabilities of the current tile (buffer C), O^T += V^T P^T, and, in
    // the same straight-line block, k-steps 2..7 of S^T of the next tile
    // (buffer N; k-steps 0..1 were issued before the running max), so the
    // exponentials overlap the matrix instructions.
    auto qk_head = [&](auto N, f32x16& n0, f32x16& n1) {
      const char* K = kbuf(N);
      n0 = f32x16{};
      n1 = f32x16{};
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bf16x8 k0 = *(const bf16x8*)(K - kHiLds + koff[s]);
        const bf16x8 k1 = *(const bf16x8*)(K - kHiLds + 32 * kRow + koff[s]);
        n0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qb[s], n0, 0, 0, 0);
        n1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qb[s], n1, 0, 0, 0);
      }
      // operand reads two ahead of the products that use them
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // LDS reads
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
    };
    auto exp_pv_qk = [&](auto C, auto N, f32x16& s0, f32x16& s1, f32x16& n0, f32x16& n1) {
      const char* V = vbuf(C);
      const char* K = kbuf(N);
      // LLVM's MFMA / exponential interleave strategy for this block: measured
      // 1.4% fewer cycles per launch than the default schedule
      __builtin_amdgcn_iglp_opt(3);
      const float nm = m_use == -INFINITY ? 0.f : -m_use;
      bf16x8 pb[4];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        const f32x16& sv = ks < 2 ? s0 : s1;
        const int base = 8 * (ks & 1);
#pragma unroll
        for (int x = 0; x < 8; ++x) pb[ks][x] = (__bf16)__builtin_amdgcn_exp2f(fmaf(sv[base + x], sc, nm));
        if (ks < 3) {  // k-steps 2(ks+1), 2(ks+1)+1 of the next tile's S^T
#pragma unroll
          for (int s = 2 * ks + 2; s < 2 * ks + 4; ++s) {
            const bf16x8 k0 = *(const bf16x8*)(K - kHiLds + koff[s]);
            const bf16x8 k1 = *(const bf16x8*)(K - kHiLds + 32 * kRow + koff[s]);
            n0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qb[s], n0, 0, 0, 0);
            n1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qb[s], n1, 0, 0, 0);
          }
        }
#pragma unroll
        for (int d = 0; d < 4; ++d) {
          const char* vp = V + ks * 16 * kRow + voff[d];
          const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vp));
          const bf16x4 up = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vp + 8 * kRow));
          const bf16x8 va = __builtin_shufflevector(lo, up, 0, 1, 2, 3, 4, 5, 6, 7);
          o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[ks], o[d], 0, 0, 0);
        }
      }
      // row sum of the bf16 probabilities the PV product used
      float lsum = 0.f;
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const bf16x2 pp = {pb[ks][2 * x], pb[ks][2 * x + 1]};
          lsum = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, lsum, false);
        }
      l_run += lsum;
    };

    // One pipeline step: tile i sits in ring slot C, tile i+1 in slot N, and
    // tile i+3 is fetched by DMA into slot S (read last in step i-1).  Each
    // wavefront then waits only for the DMA of tile i+2 (its four newest
    // buffer loads, tile i+3's, may stay in flight) before the barrier.  Past
    // the end of the key range the fetched rows are never used and the
    // next-tile product is discarded, which keeps the step free of branches.
    // A wavefront whose rows all end before tile i skips the arithmetic.
    auto step = [&](auto C, auto N, auto S, int i, f32x16& c0, f32x16& c1, f32x16& n0, f32x16& n1) {
      const int kt = key_begin + i * kKT;
      fetch(kt + 3 * kKT, kbuf(S), vbuf(S));
      if (kt <= g_wmax) {
        qk_head(N, n0, n1);
        mask_max(kt, c0, c1);
        exp_pv_qk(C, N, c0, c1, n0, n1);
      }
      asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
      __builtin_amdgcn_s_barrier();
    };

    f32x16 sa0, sa1, sb0, sb1;
    // The next item is claimed at the start of the last group of four steps
    // that leaves at least two steps, so that the claim's round trip overlaps
    // them (an earlier claim would hold the item back from idle workgroups
    // for longer).
    const int claim_at = max(0, (n_kt - 2) & ~3);
    asm volatile("s_waitcnt vmcnt(4)" ::: "memory");  // tiles 0 and 1 and the queries have landed
    __builtin_amdgcn_s_barrier();
    qk(I0{}, sa0, sa1);
    for (int i = 0; i < n_kt; i += 4) {
      if (i == claim_at && tid == 0) got = claim_add(plan_view(args().plan, 0).hdr + jq);
      step(I0{}, I1{}, I3{}, i, sa0, sa1, sb0, sb1);
      if (i + 1 >= n_kt) break;
      step(I1{}, I2{}, I0{}, i + 1, sb0, sb1, sa0, sa1);
      if (i + 2 >= n_kt) break;
      step(I2{}, I3{}, I1{}, i + 2, sa0, sa1, sb0, sb1);
      if (i + 3 >= n_kt) break;
      step(I3{}, I0{}, I2{}, i + 3, sb0, sb1, sa0, sa1);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this item's DMA is complete
    __builtin_amdgcn_s_barrier();                     // and every wavefront is done with the ring

    // Epilogue.  The next item (claimed in the tile loop, or here if the item
    // had no key tiles) is started first: its descriptor, buffer ranges and
    // key tiles 0 and 1 into ring slots 0 and 1, while this item's results
    // pass through slots 2 and 3.
    const AttnArgs A = args();
    const PlanView pv = plan_view(A.plan, A.n_tiles);
    if (n_kt == 0 && tid == 0) got = claim_add(&pv.hdr[jq]);
    const int lrel = it_field(0), oi = it_field(1), kv = it_field(2), piece_f = it_field(3);
    const bool more = begin_next(A, got);
    const int layer = A.lb + lrel;
    const int nsp = pv.nsp[oi];
    const int piece = min(piece_f, nsp - 1);  // (a bound, as in start_item)
    const int64_t m0 = (A.n_tiles - 1 - oi) * RT;
    const bool valid = g_q >= 0;
    const int el = lane_id(), eq = el & 31, ehi = el >> 5;
    const int64_t m = m0 + wave * RW + eq / G;
    const int h = kv * G + eq % G;
    const float l_tot = pair_sum(l_run);
    // The wavefront's 32 result rows (query vector q, 256 bytes each) pass
    // through 8 KB of ring slots 2 and 3, so that every global store writes
    // four whole rows instead of 16-byte pieces of 32 rows.  In LDS, 16-byte
    // chunk c of row q sits at position c ^ (q & 15) (conflict-free writes of
    // the accumulator layout).
    char* tb = (wave < 2 ? up_k2 : wave < 4 ? up_k3 : wave < 6 ? lo_v2 : lo_v3) + (wave & 1) * (32 * kRow);
    auto put = [&](int c, u32x2 w) {  // chunk c = elements 8c..8c+7 of row q; this lane holds half hi
      *(u32x2*)(tb + eq * kRow + ((c ^ (eq & 15)) << 4) + 8 * ehi) = w;
    };
    auto get = [&](int row, int c) -> u32x4 { return *(const u32x4*)(tb + row * kRow + ((c ^ (row & 15)) << 4)); };
    // accumulator register r of d-block b holds dim 32b + 8(r/4) + 4hi + r%4
    if (nsp == 1) {
      const float inv = valid ? 1.f / l_tot : 0.f;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          u32x2 w;
          w[0] = pack_bf16x2(o[d][4 * rq] * inv, o[d][4 * rq + 1] * inv);
          w[1] = pack_bf16x2(o[d][4 * rq + 2] * inv, o[d][4 * rq + 3] * inv);
          put(4 * d + rq, w);
        }
      if (valid && A.lse && ehi == 0)
        A.lse[((int64_t)layer * A.Hq + h) * A.n_sel + m] = (m_use + __log2f(l_tot)) * kLn2;
      const uint64_t has_row = __ballot(valid);  // bit q: query vector q has an output row
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      // store s covers rows R = 4s .. 4s+3 in output order: head hh = R / RW, selected row j = R % RW
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int R = 4 * s + (el >> 4), c = el & 15;
        const int hh = R / RW, j = R % RW, qq = j * G + hh;
        const u32x4 v = get(qq, c);
        if ((has_row >> qq) & 1)
          *(u32x4*)(A.out + (((int64_t)layer * A.Hq + kv * G + hh) * A.n_sel + m0 + wave * RW + j) * 128 + 8 * c) = v;
      }
    } else {
      // The piece's output row O / sum, scaled by 2^-e so that its largest
      // magnitude lies in [0.5, 1), is kept in fp16 (11 significant bits
      // relative to that element; the scale keeps the bf16 range of V within
      // fp16's).
      const int64_t slot = (int64_t)lrel * A.part_cap + pv.ppre[oi] + kv * nsp + piece;  // < part_cap per layer
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      float amax = 0.f;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) amax = fmaxf(amax, fabsf(o[d][r]));
      amax = pair_max(amax) * inv;
      const int e = amax > 0.f ? min(max(__builtin_amdgcn_frexp_expf(amax), -100), 100) : 0;  // 2^-e stays normal
      const float sc_e = inv * __builtin_ldexpf(1.f, -e);
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int rq = 0; rq < 4; ++rq) {
          const f32x4 v4 = {o[d][4 * rq] * sc_e, o[d][4 * rq + 1] * sc_e, o[d][4 * rq + 2] * sc_e, o[d][4 * rq + 3] * sc_e};
          put(4 * d + rq, __builtin_bit_cast(u32x2, __builtin_convertvector(v4, f16x4)));
        }
      if (ehi == 0) {
        const f32x4 ml = {m_use, l_tot, (float)e, 0.f};
        *(f32x4*)(A.part_ml + (slot * kQPerWG + wave * 32 + eq) * 4) = ml;
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      uint16_t* pp = A.part + (slot * kQPerWG + wave * 32) * 128;  // the wavefront's 32 consecutive rows
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const int R = 4 * s + (el >> 4), c = el & 15;
        *(u32x4*)(pp + R * 128 + 8 * c) = get(R, c);
      }
    }
    // every wavefront is done with ring slots 2 and 3 before the next item's
    // key tile 2 is fetched there, and s_it holds the next item
    __syncthreads();
    if (!more) break;
  }
}

// Merge the pieces of every cut row tile, in piece order: one block per
// (row tile, KV head, wavefront's 32 query vectors) of each layer.
template <int G>
__global__ __launch_bounds__(256) void sel_attn_combine(const AttnArgs a) {
  constexpr int RW = 32 / G;
  constexpr int RT = kWaves * RW;
  const PlanView pv = plan_view(a.plan, a.n_tiles);
  const int w = blockIdx.x % kWaves;
  const int kvh = (blockIdx.x / kWaves) % a.Hkv;
  const int64_t oi = blockIdx.x / (kWaves * a.Hkv);  // longest-first order
  const int nsp = pv.nsp[oi];
  if (nsp == 1) return;  // not cut: written directly
  const int layer = a.lb + blockIdx.y;
  const int64_t slot0 = (int64_t)blockIdx.y * a.part_cap + pv.ppre[oi] + kvh * nsp;
  const int64_t m0 = (a.n_tiles - 1 - oi) * RT;
  // thread: query vector qv of the tile (row qv / G, head qv % G), dims 16 d16 .. 16 d16 + 15
  const int qv = 32 * w + (threadIdx.x >> 3), d16 = threadIdx.x & 7;
  const int64_t m = m0 + qv / G;
  if (m >= a.n_sel) return;
  const int t = a.sel[m];
  if (t < a.cs1 || t >= a.T) return;  // not a later-chunk token: no output (as in the direct path)
  const int h = kvh * G + qv % G;
  const float* ml0 = a.part_ml + (slot0 * kQPerWG + qv) * 4;
  const uint16_t* po0 = a.part + (slot0 * kQPerWG + qv) * 128 + 16 * d16;
  constexpr int64_t kSlotMl = kQPerWG * 4, kSlotPo = kQPerWG * 128;  // one partial slot apart
  float M = -INFINITY;
#pragma unroll 8
  for (int p = 0; p < nsp; ++p) M = fmaxf(M, ml0[p * kSlotMl]);
  float Lsum = 0.f;
  f32x4 acc[4] = {};
  // piece order, several pieces' loads in flight
#pragma unroll 4
  for (int p = 0; p < nsp; ++p) {
    const f32x4 ml = *(const f32x4*)(ml0 + p * kSlotMl);
    const float wgt = ml[0] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml[0] - M) * ml[1];
    Lsum += wgt;
    const float sw = wgt * __builtin_ldexpf(1.f, (int)ml[2]);
    const uint16_t* pp = po0 + p * kSlotPo;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const f16x4 po = *(const f16x4*)(pp + 4 * k);
      acc[k] += sw * __builtin_convertvector(po, f32x4);
    }
  }
  const float inv = 1.f / Lsum;
  uint16_t* op = a.out + (((int64_t)layer * a.Hq + h) * a.n_sel + m) * 128 + 16 * d16;
  u32x4 o0, o1;
  o0[0] = pack_bf16x2(acc[0][0] * inv, acc[0][1] * inv);
  o0[1] = pack_bf16x2(acc[0][2] * inv, acc[0][3] * inv);
  o0[2] = pack_bf16x2(acc[1][0] * inv, acc[1][1] * inv);
  o0[3] = pack_bf16x2(acc[1][2] * inv, acc[1][3] * inv);
  o1[0] = pack_bf16x2(acc[2][0] * inv, acc[2][1] * inv);
  o1[1] = pack_bf16x2(acc[2][2] * inv, acc[2][3] * inv);
  o1[2] = pack_bf16x2(acc[3][0] * inv, acc[3][1] * inv);
  o1[3] = pack_bf16x2(acc[3][2] * inv, acc[3][3] * inv);
  *(u32x4*)op = o0;
  *(u32x4*)(op + 8) = o1;
  if (a.lse && d16 == 0) a.lse[((int64_t)layer * a.Hq + h) * a.n_sel + m] = (M + __log2f(Lsum)) * kLn2;
}

// ============================================================== generic attention
struct GenAttnArgs {
  const void* q;
  const int32_t* sel;
  void* out;
  float* lse;
  int64_t T, n, n_sel;
  int cs1, Hq, Hkv, G, D, lb;
  int q_by_slot;
  float scale;
};

template <typename E>
__device__ __forceinline__ float gld(const E* p);
template <>
__device__ __forceinline__ float gld<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float gld<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <typename E>
__device__ __forceinline__ void gst(E* p, float x);
template <>
__device__ __forceinline__ void gst<float>(float* p, float x) { *p = x; }
template <>
__device__ __forceinline__ void gst<uint16_t>(uint16_t* p, float x) { *p = f32_to_bf16(x); }

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

template <typename E, typename Rows>
__global__ __launch_bounds__(64) void sel_attn_generic(const GenAttnArgs a, const Rows rows) {
  __shared__ float qs[512];
  __shared__ float ps[64];
  const int64_t m = blockIdx.x;
  const int h = blockIdx.y;
  const int layer = a.lb + blockIdx.z;
  const int lane = threadIdx.x;
  const int t = a.sel[m];
  if (t < a.cs1 || t >= a.T) return;  // out-of-contract index
  const int kv = h / a.G;
  const E* qp = (const E*)a.q + (a.q_by_slot ? ((int64_t)blockIdx.z * a.Hq + h) * a.n_sel + m
                                             : ((int64_t)layer * a.Hq + h) * a.n + (t - a.cs1)) * a.D;
  const int64_t plane = (int64_t)layer * a.Hkv + kv;
  const int rb = a.D * (int)sizeof(E);
  for (int d = lane; d < a.D; d += 64) qs[d] = gld(qp + d);
  __syncthreads();
  float acc[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) acc[j] = 0.f;
  float mrun = -INFINITY, lrun = 0.f;
  for (int j0 = 0; j0 <= t; j0 += 64) {
    const int j = j0 + lane;
    float s = -INFINITY;
    if (j <= t) {
      const E* kr = (const E*)rows.row(false, plane, j, rb);
      float dot = 0.f;
      for (int d = 0; d < a.D; ++d) dot = fmaf(qs[d], gld(kr + d), dot);
      s = dot * a.scale;
    }
    const float m_new = fmaxf(mrun, wave_max(s));
    const float alpha = mrun == -INFINITY ? 0.f : expf(mrun - m_new);
    const float p = j <= t ? expf(s - m_new) : 0.f;
    lrun = lrun * alpha + wave_sum(p);
#pragma unroll
    for (int x = 0; x < 8; ++x) acc[x] *= alpha;
    ps[lane] = p;
    __syncthreads();
    const int cnt = min(64, t + 1 - j0);
    for (int jj = 0; jj < cnt; ++jj) {
      const float pj = ps[jj];
      const E* vr = (const E*)rows.row(true, plane, j0 + jj, rb);
#pragma unroll
      for (int x = 0; x < 8; ++x) {
        const int d = lane + 64 * x;
        if (d < a.D) acc[x] = fmaf(pj, gld(vr + d), acc[x]);
      }
    }
    __syncthreads();
    mrun = m_new;
  }
  E* op = (E*)a.out + (((int64_t)layer * a.Hq + h) * a.n_sel + m) * a.D;
  const float inv = 1.f / lrun;
#pragma unroll
  for (int x = 0; x < 8; ++x) {
    const int d = lane + 64 * x;
    if (d < a.D) gst(op + d, acc[x] * inv);
  }
  if (a.lse && lane == 0) a.lse[((int64_t)layer * a.Hq + h) * a.n_sel + m] = mrun + logf(lrun);
}

// ============================================================== planning & launch
static int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// A piece has at least kMinPiece key tiles, so a row tile has at most
// ceil(ceil(T / 64) / kMinPiece) pieces (and at most kMaxPieces).
static int64_t plan_max_pieces(int64_t T) {
  return std::min<int64_t>(kMaxPieces, ((T + kKT - 1) / kKT + kMinPiece - 1) / kMinPiece);
}
// Items per queue and layer: at most one per row tile and KV head of the
// queue, plus the extra pieces of cut row tiles (bounded by part_cap).
static int64_t plan_per_q_bound(int64_t n_tiles, int Hkv, int part_cap) {
  const int nq = n_queues(Hkv);
  return (n_tiles * Hkv + part_cap + nq - 1) / nq;
}

AttnPlan plan_attention(const Geo& g, int64_t n_sel, int layers_per_call, int64_t max_part_slots) {
  AttnPlan p{};
  // (buffer loads address one [T][128] bf16 plane, plus three tiles of
  // look-ahead, with 32-bit byte offsets)
  p.mfma = g.dtype == CS_BF16 && g.D == 128 && g.G <= 32 && 32 % g.G == 0 && g.T <= (int64_t(1) << 23) - 256;
  if (!p.mfma || n_sel == 0) {
    p.ws_bytes_per_layer = 0;
    p.ws_fixed_bytes = 0;
    return p;
  }
  p.rows_per_tile = kWaves * (32 / g.G);
  p.n_tiles = (n_sel + p.rows_per_tile - 1) / p.rows_per_tile;
  // Partial slots: the plan keeps the total under kPartCap per layer by
  // enlarging the pieces.
  const int64_t max_pieces = plan_max_pieces(g.T);
  // the plan counts key tiles of a layer, and items of a call, in 32-bit integers
  if (p.n_tiles * ((g.T + kKT - 1) / kKT) * g.Hkv >= (int64_t(1) << 31) ||
      p.n_tiles * g.Hkv * std::max<int64_t>(1, max_pieces) * std::max(1, layers_per_call) >= (int64_t(1) << 31)) {
    p.mfma = false;
    p.ws_bytes_per_layer = 0;
    p.ws_fixed_bytes = 0;
    return p;
  }
  p.part_cap = (int)std::min<int64_t>(std::min<int64_t>(kPartCap, std::max<int64_t>(max_part_slots, 0)),
                                      p.n_tiles * g.Hkv * (max_pieces > 1 ? max_pieces : 0));
  // a cut row tile fills at least 2 H_kv slots: fewer slots allow no cut at all
  if (p.part_cap < 2 * g.Hkv) p.part_cap = 0;
  // item descriptors (4 ints each) after the plan's arrays, one per queue position
  const int64_t per_q_bound = plan_per_q_bound(p.n_tiles, g.Hkv, p.part_cap);
  p.desc_off = (int)((plan_ints(p.n_tiles, max_pieces) + 3) / 4 * 4);
  p.ws_fixed_bytes = ((p.desc_off + 4 * per_q_bound) * sizeof(int) + 255) / 256 * 256;
  p.ws_bytes_per_layer = (size_t)p.part_cap * kQPerWG * (128 * sizeof(uint16_t) + 4 * sizeof(float));
  return p;
}

// Workgroups of the attention launch (resident, one per CU, each taking items
// until the queues are empty; no more than there are items) and of the
// combine launch.
static int64_t mfma_grid(const AttnArgs& a) {
  // items per queue and layer: at most one per row tile and KV head of the
  // queue, plus the extra pieces of cut row tiles (bounded by part_cap)
  const int nq = n_queues(a.Hkv);
  const int64_t items = (a.n_tiles * a.Hkv + a.part_cap + nq - 1) / nq * nq * a.layers;
  return std::min<int64_t>(kPlanCUs, items);
}
static int64_t combine_grid(const AttnArgs& a) {
  // cut row tiles lead the longest-first order, and each fills at least
  // 2 H_kv partial slots
  return std::min<int64_t>(a.n_tiles, a.part_cap / (2 * a.Hkv)) * a.Hkv * kWaves;
}

static int64_t plan_scatter_blocks(const ScatterArgs& sa) {
  return 1 + std::min<int64_t>((scatter_items(sa) + 1023) / 1024, 16384);
}

template <int G, typename Rows>
static void launch_mfma_g(const AttnArgs& a, const Rows& rows, const ScatterArgs* sa, const RopeRowsArgs* ra,
                          hipStream_t s) {
  static_assert(sizeof(AttnArgs) + sizeof(Rows) <= 4096, "kernel arguments within 4 KB");
  static_assert(sizeof(PlanArgs) + sizeof(Rows) + sizeof(ScatterArgs) <= 4096, "kernel arguments within 4 KB");
  static_assert(sizeof(PlanArgs) + sizeof(Rows) + sizeof(RopeRowsArgs) <= 4096, "kernel arguments within 4 KB");
  PlanArgs pa;
  pa.sel = a.sel;
  pa.n_sel = a.n_sel;
  pa.n_tiles = a.n_tiles;
  pa.T = a.T;
  pa.RT = kWaves * (32 / G);
  pa.Hkv = a.Hkv;
  pa.part_cap = a.part_cap;
  pa.desc_off = a.desc_off;
  pa.pj_cap = (int)plan_max_pieces(a.T) + 1;
  pa.desc_cap = (int)(4 * plan_per_q_bound(a.n_tiles, a.Hkv, a.part_cap));
  pa.plan = a.plan;
  if (ra) {
    TraceScope tr("plan_rope_scatter", s);
    const unsigned blocks = (unsigned)(1 + (int64_t)ra->nblk * a.layers);
    CS_LAUNCH(tr, plan_rope_scatter<Rows>, dim3(blocks), dim3(1024), 0, s, pa, rows, *ra);
  } else if (sa) {
    TraceScope tr("plan_scatter", s);
    const unsigned blocks = (unsigned)plan_scatter_blocks(*sa);
    if (scatter_word(*sa) == 16)
      CS_LAUNCH(tr, (plan_scatter<16, Rows>), dim3(blocks), dim3(1024), 0, s, pa, rows, *sa);
    else
      CS_LAUNCH(tr, (plan_scatter<4, Rows>), dim3(blocks), dim3(1024), 0, s, pa, rows, *sa);
  } else {
    TraceScope tr("plan_items", s);
    CS_LAUNCH(tr, plan_items, dim3(1), dim3(1024), 0, s, pa);
  }
  {
    TraceScope tr("sel_attn_mfma", s);
    CS_LAUNCH(tr, (sel_attn_mfma<G, Rows>), dim3((unsigned)mfma_grid(a)), dim3(kThreads), 0, s, a, rows);
  }
  if (a.part_cap > 0) {
    TraceScope tr("sel_attn_combine", s);
    CS_LAUNCH(tr, sel_attn_combine<G>, dim3((unsigned)combine_grid(a), a.layers), dim3(256), 0, s, a);
  }
}

template <typename Rows>
static cs_status launch_mfma(int G, const AttnArgs& a, const Rows& rows, const ScatterArgs* sa,
                             const RopeRowsArgs* ra, hipStream_t s) {
  switch (G) {
    case 1: launch_mfma_g<1>(a, rows, sa, ra, s); break;
    case 2: launch_mfma_g<2>(a, rows, sa, ra, s); break;
    case 4: launch_mfma_g<4>(a, rows, sa, ra, s); break;
    case 8: launch_mfma_g<8>(a, rows, sa, ra, s); break;
    case 16: launch_mfma_g<16>(a, rows, sa, ra, s); break;
    case 32: launch_mfma_g<32>(a, rows, sa, ra, s); break;
    default: return fail(CS_ERR_UNSUPPORTED, "MFMA attention needs H_q/H_kv dividing 32");
  }
  return CS_OK;
}

template <typename Rows>
static void launch_generic(const Geo& g, const GenAttnArgs& a, const Rows& rows, int64_t n_sel, int layers,
                           hipStream_t s) {
  static_assert(sizeof(GenAttnArgs) + sizeof(Rows) <= 4096, "kernel arguments within 4 KB");
  TraceScope tr("sel_attn_generic", s);
  if (g.dtype == CS_BF16)
    CS_LAUNCH(tr, (sel_attn_generic<uint16_t, Rows>), dim3((unsigned)n_sel, g.Hq, layers), dim3(64), 0, s, a,
                       rows);
  else
    CS_LAUNCH(tr, (sel_attn_generic<float, Rows>), dim3((unsigned)n_sel, g.Hq, layers), dim3(64), 0, s, a,
                       rows);
}

size_t rope_table_bytes(int64_t n_sel) { return ((size_t)n_sel * 64 * sizeof(float2) + 255) / 256 * 256; }

bool chunks_tile_aligned(const Geo& g) {
  for (int c = 0; c < g.N; ++c)
    if (g.cs[c] % kKT) return false;
  return true;
}

cs_status launch_attention(const Geo& g, const AttnPlan& p, const CacheView& cv, int lb, int le,
                           const int32_t* sel, int64_t n_sel, const void* qf, bool q_by_slot, void* out, float* lse,
                           void* ws, hipStream_t s, bool check_only, const ScatterJob* job, const RopeJob* rope) {
  const int layers = le - lb;
  ScatterArgs sa;
  if (job) sa = scatter_args(g, lb, le, sel, n_sel, job->kf, job->vf);
  RopeRowsArgs ra;
  if (rope) {  // (MFMA path only: bf16, head_dim 128)
    ra.k_pre = (const uint16_t*)rope->k_pre;
    ra.v_new = (const uint16_t*)rope->v_new;
    ra.sel = sel;
    ra.coords = rope->coords;
    ra.tab = (float2*)rope->tab;
    ra.T = g.T;
    ra.n = g.n;
    ra.n_sel = n_sel;
    ra.cs1 = g.cs1;
    ra.Hkv = g.Hkv;
    ra.lb = lb;
    ra.nblk = (int)((n_sel + kPrTok - 1) / kPrTok);
    ra.sec0 = g.sec[0];
    ra.sec01 = g.sec[0] + g.sec[1];
    for (int i = 0; i < 64; ++i) ra.theta[i] = rope->theta[i];
  }
  if (p.mfma) {
    if (cv.paged && !chunks_tile_aligned(g))
      return fail(CS_ERR_UNSUPPORTED, "a paged cache needs chunk starts that are multiples of 64 on the MFMA path");
    AttnArgs a;
    a.q = (const uint16_t*)qf;
    a.sel = sel;
    a.out = (uint16_t*)out;
    a.lse = lse;
    a.plan = (int*)ws;
    a.part = (uint16_t*)((char*)ws + p.ws_fixed_bytes);
    a.part_ml = (float*)(a.part + (size_t)layers * p.part_cap * kQPerWG * 128);
    a.T = g.T;
    a.n = g.n;
    a.n_sel = n_sel;
    a.n_tiles = p.n_tiles;
    a.cs1 = (int)g.cs1;
    a.Hq = g.Hq;
    a.Hkv = g.Hkv;
    a.lb = lb;
    a.layers = layers;
    a.part_cap = p.part_cap;
    a.q_by_slot = q_by_slot ? 1 : 0;
    a.desc_off = p.desc_off;
    a.rope_tab = rope ? (const float2*)rope->tab : nullptr;
    a.scale_log2 = (float)(1.4426950408889634 / sqrt((double)g.D));
    cs_status stg = check_grid(mfma_grid(a), 1, 1, kThreads, "selective attention");
    if (!stg && rope) stg = check_grid(1 + (int64_t)ra.nblk * layers, 1, 1, 1024, "rotary scatter");
    if (!stg && a.part_cap > 0) stg = check_grid(combine_grid(a), layers, 1, 256, "partial combine");
    if (stg || check_only) return stg;
    const ScatterArgs* sp = job ? &sa : nullptr;
    const RopeRowsArgs* rp = rope ? &ra : nullptr;
    const cs_status st = cv.paged ? launch_mfma(g.G, a, cv.pages<kMaxPages>(g), sp, rp, s)
                                  : launch_mfma(g.G, a, cv.flat(g), sp, rp, s);
    if (st) return st;
    return check_launch("selective attention launch");
  }
  GenAttnArgs a;
  a.q = qf;
  a.q_by_slot = q_by_slot ? 1 : 0;
  a.sel = sel;
  a.out = out;
  a.lse = lse;
  a.T = g.T;
  a.n = g.n;
  a.n_sel = n_sel;
  a.cs1 = (int)g.cs1;
  a.Hq = g.Hq;
  a.Hkv = g.Hkv;
  a.G = g.G;
  a.D = g.D;
  a.lb = lb;
  a.scale = (float)(1.0 / sqrt((double)g.D));
  const cs_status stg = check_grid(n_sel, g.Hq, layers, 64, "selective attention");
  if (stg || check_only) return stg;
  if (job) {  // the scatter first: the attention reads the repaired rows
    if (cv.paged) launch_scatter_rows(sa, cv.pages<kMaxPages>(g), s);
    else launch_scatter_rows(sa, cv.flat(g), s);
  }
  if (cv.paged) launch_generic(g, a, cv.pages<kMaxPages>(g), n_sel, layers, s);
  else launch_generic(g, a, cv.flat(g), n_sel, layers, s);
  return check_launch("generic attention launch");
}

}  // namespace cs
