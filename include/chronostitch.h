/*
 * chronostitch.h -- C ABI of the ChronoStitch KV-composition hot path for
 * AMD Instinct MI355X (gfx950).
 *
 * The method (ChronoStitch, Section 2) composes independently prefilled
 * visual KV caches: stored post-rotary keys are moved from local chunk
 * coordinates to a global three-axis (t, h, w) mRoPE timeline by a delta
 * rotation (Eq. 3); later-chunk tokens are ranked by the deviation of their
 * recomputed scoring-layer key (Eq. 5); the top rho fraction is recomputed,
 * attending causally over the composed cache (Eq. 1), and their fresh keys
 * and values are scattered back.
 *
 * Conventions shared by every entry point
 *  - All functions are extern "C", take plain pointers and sizes, and never
 *    throw.  They return CS_OK or an error code; cs_last_error() then gives
 *    a human-readable message (thread-local, valid until the next call on
 *    the same thread).
 *  - Argument errors are detected before anything is enqueued and before any
 *    HIP runtime call, so a rejected call leaves device memory untouched.
 *    The same holds for a call whose kernel launches would exceed the GPU's
 *    grid limits (caches of tens of millions of tokens per call): every launch
 *    of the call is sized first, and such a call returns CS_ERR_UNSUPPORTED.
 *  - DEVICE pointers are device memory of the current HIP device; HOST
 *    pointers are read (or written) before the call returns, except the host
 *    chunk data of compose_load_rebase_k_paged, which its enqueued copies
 *    read (the pointer arrays themselves are read before it returns).  The caller
 *    owns every buffer; the library allocates no device memory.  Scratch
 *    memory is a caller-provided workspace sized by the *_workspace query.
 *  - Device work is asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream).  Outputs in device memory are valid once the stream has
 *    reached the enqueued work.  Host outputs are written synchronously.
 *  - Calls are re-entrant for distinct buffers and streams.  Inputs must not
 *    alias outputs except for the documented in-place caches.
 *  - Tensor layouts are dense, row-major, with the last index contiguous:
 *      caches      [L][H_kv][T][D]   chunks are contiguous token ranges, so
 *                                    the concatenation of the chunk caches is
 *                                    the layout itself (the *_paged calls
 *                                    take one buffer per chunk instead)
 *      fresh Q     [L][H_q][n][D]    row r <-> token chunk_start[1] + r
 *      fresh K, V  [L][H_kv][n][D]   row r <-> token chunk_start[1] + r
 *    where n = T - chunk_start[1] is the number of later-chunk tokens.
 *  - Element type of every K/V/Q/O tensor is geometry.dtype; bf16 values are
 *    rounded to nearest even.
 */
#ifndef CHRONOSTITCH_H
#define CHRONOSTITCH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CS_OK = 0,
  CS_ERR_INVALID_ARGUMENT = 1,   /* a pointer, size or value is out of its documented range */
  CS_ERR_UNSUPPORTED = 2,        /* a valid request this library does not implement           */
  CS_ERR_WORKSPACE_TOO_SMALL = 3,/* workspace_bytes is below the *_workspace query's answer    */
  CS_ERR_HIP = 4                 /* a HIP runtime call or kernel launch failed                 */
} cs_status;

typedef enum { CS_F32 = 0, CS_BF16 = 1 } cs_dtype;

/* Geometry of a composed cache (Section 3 gives the model's: 36 layers,
 * 16 query heads, 2 KV heads, head dim 128, mRoPE sections 16/24/24).
 *   n_q_heads % n_kv_heads == 0; query head h reads KV head h / (n_q_heads/n_kv_heads).
 *   head_dim even, 2 <= head_dim <= 512.
 *   sections: rotary pairs on the t, h, w axes, in that order; they sum to
 *     head_dim/2.  Pair i is the element pair (i, i + head_dim/2) and rotates
 *     with axis t for i < s_t, h for i < s_t + s_h, w otherwise (Eq. 2).
 *   rope_base: theta_i = rope_base^(-2i/head_dim) when inv_freq is NULL.
 *   inv_freq: HOST [head_dim/2] float64 theta_i overriding rope_base, or NULL.
 *   chunk_start: HOST [n_chunks + 1], 0 = s_0 < s_1 < ... < s_N = n_tokens;
 *     chunk c owns tokens [s_c, s_{c+1}).  n_tokens < 2^31.             */
typedef struct {
  int32_t n_layers;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t sections[3];
  int32_t dtype;               /* cs_dtype */
  double rope_base;
  const double* inv_freq;
  int64_t n_tokens;
  int32_t n_chunks;
  const int64_t* chunk_start;
} cs_geometry;

/* ---------------------------------------------------------------------------
 * compose_rebase_k -- Section 2, Eq. 3 (three-axis delta rotation).
 *
 * Gives chunk c the global coordinates p' = p + Delta_c and rotates every
 * stored post-rotary key of the chunk, in place, by R(Delta): pair i turns by
 * Delta_c[sigma(i)] * theta_i, so a key stored as f(x, p) becomes f(x, p').
 * Angles are formed in float64 and reduced modulo 2*pi before the cos/sin
 * table is rounded to float32, so offsets of 1e5 and beyond stay accurate.
 * Chunks with Delta_c = (0,0,0) are not touched (bit-identical).  Values are
 * never rotated, so there is no V argument.
 *
 *   g             geometry (HOST)
 *   k_cache       DEVICE [L][H_kv][T][D] keys, post-rotary at local
 *                 coordinates on entry and at global coordinates on return
 *   chunk_offsets HOST int32 [n_chunks][3]: (dt, dh, dw) = p' - p of chunk c
 *   local_coords  HOST int32 [T][3] token coordinates (t, h, w), or NULL
 *   global_coords HOST int32 [T][3] output p' = p + Delta_c, or NULL; needs
 *                 local_coords.  Written before the call returns.
 *   stream        hipStream_t or NULL
 * Errors: CS_ERR_INVALID_ARGUMENT for a bad geometry, a NULL k_cache or
 * chunk_offsets, or global_coords without local_coords.                    */
cs_status compose_rebase_k(const cs_geometry* g, void* k_cache,
                           const int32_t* chunk_offsets,
                           const int32_t* local_coords, int32_t* global_coords,
                           void* stream);

/* ---------------------------------------------------------------------------
 * compose_rebase_k_tokens -- Eq. 3 with one offset per token (the position
 * policies compared in Section 3 and Table 1).
 *
 * Rotates every stored post-rotary key, in place, by its own token's offset:
 * pair i of token t turns by Delta_t[sigma(i)] * theta_i, so f(x, p_t) becomes
 * f(x, p_t + Delta_t).  With Delta_t equal to the chunk offset for every token
 * of a chunk this is compose_rebase_k; a per-token offset expresses policies
 * such as scalar re-basing, which moves token j of the composed cache to
 * (j, j, j).  Angles are formed in float64 and reduced modulo 2*pi as in
 * compose_rebase_k.  Tokens with Delta_t = (0,0,0) are not touched.
 *
 *   g              geometry (HOST)
 *   k_cache        DEVICE [L][H_kv][T][D] keys, rotated in place
 *   token_offsets  DEVICE int32 [T][3]: (dt, dh, dw) = p' - p of every token
 *                  (read on the device; contents are not checked)
 *   stream         hipStream_t or NULL
 * Errors: CS_ERR_INVALID_ARGUMENT for a bad geometry or a NULL pointer,
 * CS_ERR_HIP for a launch failure.                                          */
cs_status compose_rebase_k_tokens(const cs_geometry* g, void* k_cache,
                                  const int32_t* token_offsets, void* stream);

/* ---------------------------------------------------------------------------
 * score_deviation_topk -- Section 2, Eq. 5 and the top-rho selection after it.
 *
 * For every later-chunk token t in [s_1, T):
 *   delta_t = || k_fresh[:, t - s_1, :] - k_cache[score_layer][:, t, :] ||_2
 * over all H_kv x D elements, accumulated in float64 and rounded once to
 * float32.  Then selects the k = n_select(rho, n) largest float32 scores,
 * lower token index first among equal scores, and writes their token indices
 * in ascending order.  n_select(rho, n) = 0 if rho == 0, else
 * min(n, ceil(rho * n - 1e-9)).
 *
 *   g             geometry (HOST)
 *   k_cache       DEVICE [L][H_kv][T][D] keys, already re-based
 *   score_layer   layer whose keys are compared, 0 <= score_layer < L (the
 *                 paper scores layer 1)
 *   k_fresh       DEVICE [H_kv][n][D] recomputed keys at score_layer,
 *                 post-rotary at global coordinates
 *   rho           repair fraction in [0, 1]
 *   scores        DEVICE float32 [n] output delta_t, or NULL (then the
 *                 workspace holds them)
 *   sel_idx       DEVICE int32 [k] output, ascending token indices in [s_1, T);
 *                 may be NULL when k == 0
 *   n_sel         HOST int64 output k (computed on the host; no device sync)
 *   workspace     DEVICE scratch of workspace_bytes, >= the query's answer
 * Errors: CS_ERR_INVALID_ARGUMENT (bad geometry, rho outside [0,1] or NaN,
 * score_layer out of range, NULL required pointer), CS_ERR_WORKSPACE_TOO_SMALL.
 * Scores must be finite (NaN ranking is undefined).                       */
cs_status score_deviation_topk_workspace(const cs_geometry* g, size_t* bytes);
cs_status score_deviation_topk(const cs_geometry* g, const void* k_cache,
                               int32_t score_layer, const void* k_fresh,
                               double rho, float* scores, int32_t* sel_idx,
                               int64_t* n_sel, void* workspace,
                               size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * selective_attend_scatter_rope -- selective_attend_scatter with the rotary
 * embedding of the recomputed rows fused in (Eq. 2 at the global coordinates
 * p' of Section 2).
 *
 * The recompute of a selected token applies RoPE at its global coordinate;
 * here the caller hands over the PRE-rotary fresh queries and keys and the
 * global coordinates, and only the selected rows are rotated: for each layer,
 *   1. K row of selected token t (every KV head): f(k_pre, p'_t), rounded to
 *      the storage dtype, scattered into the cache; V rows are scattered as in
 *      selective_attend_scatter;
 *   2. Q row (every query head): f(q_pre, p'_t), rounded to the storage
 *      dtype;
 *   3. attention exactly as in selective_attend_scatter.
 * For bf16 with head_dim 128 the rotations run inside the attention's own
 * launches (the keys while they are scattered, the queries as the attention
 * loads them) from a cos/sin table of the selected tokens kept in the
 * workspace; otherwise the rotated queries pass through the workspace.
 * The result equals selective_attend_scatter on q_fresh = f(q_pre, p') and
 * k_fresh = f(k_pre, p') rounded the same way.  Angles are formed in float64
 * and reduced modulo 2*pi (float32 cos/sin), as in compose_rebase_k.
 *
 *   q_pre          DEVICE [L][H_q][n][D] pre-rotary fresh queries
 *   k_pre          DEVICE [L][H_kv][n][D] pre-rotary fresh keys
 *   v_fresh        DEVICE [L][H_kv][n][D] fresh values
 *   coords         DEVICE int32 [T][3] global coordinates p' of every token
 *                  (compose_rebase_k's global_coords, copied to the device)
 *   workspace      DEVICE, >= selective_attend_scatter_rope_workspace() for
 *                  the same n_sel and n_layers_per_call >= layer_end -
 *                  layer_begin: the attention's partials plus, for bf16 with
 *                  head_dim 128, the cos/sin table (n_sel x D/2 x 8 bytes),
 *                  otherwise the rotated queries (n_layers x H_q x n_sel x D
 *                  elements); the work plan is kept from call to call as in
 *                  selective_attend_scatter's workspace
 *   other arguments as for selective_attend_scatter.
 * Errors: CS_ERR_INVALID_ARGUMENT, CS_ERR_WORKSPACE_TOO_SMALL, CS_ERR_HIP. */
cs_status selective_attend_scatter_rope_workspace(const cs_geometry* g, int64_t n_sel,
                                                  int32_t n_layers_per_call,
                                                  size_t* bytes);
cs_status selective_attend_scatter_rope(const cs_geometry* g, void* k_cache,
                                        void* v_cache, int32_t layer_begin,
                                        int32_t layer_end, const int32_t* sel_idx,
                                        int64_t n_sel, const void* q_pre,
                                        const void* k_pre, const void* v_fresh,
                                        const int32_t* coords, void* out,
                                        float* lse, void* workspace,
                                        size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * selective_attend_scatter -- Section 2, Eq. 1 and the repair step.
 *
 * For each layer l in [layer_begin, layer_end):
 *   1. scatter: k_cache[l][h][sel_idx[m]] <- k_fresh[l][h][sel_idx[m] - s_1]
 *      and the same for V; every other row is unchanged.
 *   2. attend: for slot m (token t = sel_idx[m]) and query head h
 *      (KV head kv = h / (H_q/H_kv)), with q = q_fresh[l][h][t - s_1],
 *        out[l][h][m] = softmax_j(q . K[l][kv][j] / sqrt(D)) V[l][kv][j],
 *      j = 0 .. t (causal in cache order, self included), over the
 *      post-scatter cache.  Softmax and accumulation run in float32.
 *      lse[l][h][m] = log(sum_j exp(q . K[l][kv][j] / sqrt(D))).
 * Layers are independent, so one call over many layers equals one call per
 * layer; per-layer calls mirror the model's layer-by-layer recompute.
 *
 *   g              geometry (HOST)
 *   k_cache,v_cache DEVICE [L][H_kv][T][D], rows sel_idx overwritten in place
 *   layer_begin, layer_end  0 <= begin <= end <= L
 *   sel_idx        DEVICE int32 [n_sel], strictly ascending, in [s_1, T)
 *                  (as written by score_deviation_topk).  Not checked unless
 *                  the environment variable CS_DEBUG_VALIDATE is "1": then a
 *                  violation returns CS_ERR_INVALID_ARGUMENT before anything
 *                  else is enqueued, at the cost of a synchronisation of the
 *                  stream (a debugging aid; such calls must not overlap on one
 *                  GPU).  Unchecked, an index outside [s_1, T) is skipped and
 *                  an unsorted list gives wrong outputs, never an access
 *                  outside the caller's buffers.
 *   n_sel          0 <= n_sel <= n
 *   q_fresh        DEVICE [L][H_q][n][D] fresh queries (post-rotary, global)
 *   k_fresh,v_fresh DEVICE [L][H_kv][n][D] fresh keys / values
 *   out            DEVICE [L][H_q][n_sel][D] output, slot order of sel_idx
 *   lse            DEVICE float32 [L][H_q][n_sel] output, or NULL
 *   workspace      DEVICE scratch, >= selective_attend_scatter_workspace()
 *                  for the same n_sel and n_layers_per_call >= layer_end -
 *                  layer_begin (the size grows with the layer count); no
 *                  initial contents needed.  The call leaves its work plan at
 *                  the start of the workspace; a later call that finds there
 *                  a plan made from the same inputs (the row tiles' last
 *                  selected tokens, the row-tile and KV-head counts, the
 *                  partial-slot budget), whose checksum holds, keeps it
 *                  instead of planning again, so the layer calls of one
 *                  composition plan once.  Any other contents are
 *                  overwritten: the caller may use the workspace for anything
 *                  between calls.
 * Errors: CS_ERR_INVALID_ARGUMENT, CS_ERR_WORKSPACE_TOO_SMALL, CS_ERR_HIP. */
cs_status selective_attend_scatter_workspace(const cs_geometry* g, int64_t n_sel,
                                             int32_t n_layers_per_call,
                                             size_t* bytes);
cs_status selective_attend_scatter(const cs_geometry* g, void* k_cache,
                                   void* v_cache, int32_t layer_begin,
                                   int32_t layer_end, const int32_t* sel_idx,
                                   int64_t n_sel, const void* q_fresh,
                                   const void* k_fresh, const void* v_fresh,
                                   void* out, float* lse, void* workspace,
                                   size_t workspace_bytes, void* stream);

/* ---------------------------------------------------------------------------
 * selective_attend_scatter_noalloc -- selective_attend_scatter for callers
 * that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the same scatter and
 * attention with no workspace argument.  It calls no hipMalloc, hipFree or
 * other allocating routine (kernel tracing is off for its launches).
 *
 * Its plan and partial results live in a 64 MiB array of device memory that
 * the library holds on every GPU it runs on until the process ends; its
 * device address is looked up once per GPU, on the first call with that GPU
 * current.  Every call on a GPU shares that GPU's array: calls that overlap
 * on one GPU (two streams, two threads) race and give wrong results.  Nothing
 * needs clearing between calls; the plan left in the array is kept by a later
 * call with the same inputs, as in a workspace.
 *
 * When the call's plan and partials would exceed the array, the key pieces
 * of long row tiles are made longer (fewer partials), so the output then
 * differs from selective_attend_scatter's by rounding only (same tolerance);
 * within the limit it is bit-identical.  A call whose plan alone exceeds the
 * array returns CS_ERR_UNSUPPORTED before anything is enqueued (this needs
 * several million selected rows).
 *
 * Arguments, layouts and the other errors are those of
 * selective_attend_scatter (contiguous cache only).                        */
cs_status selective_attend_scatter_noalloc(const cs_geometry* g, void* k_cache,
                                           void* v_cache, int32_t layer_begin,
                                           int32_t layer_end, const int32_t* sel_idx,
                                           int64_t n_sel, const void* q_fresh,
                                           const void* k_fresh, const void* v_fresh,
                                           void* out, float* lse, void* stream);

/* ---------------------------------------------------------------------------
 * Paged cache (Section 2: every chunk is prefilled and stored on its own, and
 * the stored caches are concatenated after re-basing, the step listed after
 * Eq. 6).  The *_paged calls
 * take the cache as the chunks' own buffers instead of one composed buffer,
 * so chunks loaded from storage are used where they landed:
 *   k_chunks, v_chunks   HOST arrays of geometry.n_chunks DEVICE pointers;
 *                        chunk c's keys (values) are [L][H_kv][len_c][D],
 *                        len_c = chunk_start[c+1] - chunk_start[c], dense,
 *                        row-major.  The arrays are read before the call
 *                        returns; the buffers are used in place.
 * Every other argument, the workspace sizes (the contiguous *_workspace
 * queries apply), the outputs and the errors are those of the contiguous call
 * of the same name, and the results are bit-identical to that call on the
 * concatenation of the chunks.
 * Limits: n_chunks <= 128 when dtype is CS_BF16 and head_dim is 128, <= 64
 * otherwise (else CS_ERR_UNSUPPORTED).  The attention calls on the bf16 /
 * head_dim 128 path read whole 64-key tiles from one chunk, so they need every
 * chunk_start to be a multiple of 64 (else CS_ERR_UNSUPPORTED).  A NULL array
 * or NULL chunk pointer is CS_ERR_INVALID_ARGUMENT.                          */
cs_status compose_rebase_k_paged(const cs_geometry* g, void* const* k_chunks,
                                 const int32_t* chunk_offsets,
                                 const int32_t* local_coords,
                                 int32_t* global_coords, void* stream);
cs_status compose_rebase_k_tokens_paged(const cs_geometry* g, void* const* k_chunks,
                                        const int32_t* token_offsets, void* stream);

/* compose_load_rebase_k_paged -- the chunks' load from host memory with the
 * re-basing of Eq. 3 done during the load (Section 2: chunks come back from
 * storage and are re-based before they are concatenated), so that the
 * rotation hides under the transfer of the values.
 *
 * Every chunk's keys are copied from the host to k_chunks[c] on copy_stream,
 * then every chunk's values to v_chunks[c]; once the keys have landed, stream
 * re-bases them exactly as compose_rebase_k_paged would (chunks with a zero
 * offset are copied only) while the values are still in transfer.  The
 * copies start after the work
 * enqueued on stream before the call, and when stream reaches the end of the
 * call's work every copy is complete: the call is one step of stream, and
 * later work on stream sees the whole composed cache.
 *   k_host, v_host  HOST arrays of n_chunks HOST pointers, chunk c's keys
 *                   (values) as [L][H_kv][len_c][D]; page-locked memory
 *                   (hipHostMalloc) lets the copies overlap the re-basing,
 *                   pageable memory works but serialises them.  Read before
 *                   the call's work completes on stream: keep them unchanged
 *                   until then.
 *   copy_stream     the stream of the copies; NULL or equal to stream: one
 *                   stream does everything in order.
 *   k_chunks, v_chunks, chunk_offsets, stream: as for compose_rebase_k_paged
 *                   (the destination buffers' prior contents are overwritten).
 * The results are bit-identical to copying the chunks and then calling
 * compose_rebase_k_paged.  Errors: those of compose_rebase_k_paged, plus
 * CS_ERR_INVALID_ARGUMENT for a NULL host array or chunk pointer. */
cs_status compose_load_rebase_k_paged(const cs_geometry* g, void* const* k_chunks,
                                      void* const* v_chunks, const void* const* k_host,
                                      const void* const* v_host,
                                      const int32_t* chunk_offsets,
                                      void* copy_stream, void* stream);
cs_status score_deviation_topk_paged(const cs_geometry* g, void* const* k_chunks,
                                     int32_t score_layer, const void* k_fresh,
                                     double rho, float* scores, int32_t* sel_idx,
                                     int64_t* n_sel, void* workspace,
                                     size_t workspace_bytes, void* stream);
cs_status selective_attend_scatter_paged(const cs_geometry* g, void* const* k_chunks,
                                         void* const* v_chunks, int32_t layer_begin,
                                         int32_t layer_end, const int32_t* sel_idx,
                                         int64_t n_sel, const void* q_fresh,
                                         const void* k_fresh, const void* v_fresh,
                                         void* out, float* lse, void* workspace,
                                         size_t workspace_bytes, void* stream);
cs_status selective_attend_scatter_rope_paged(const cs_geometry* g, void* const* k_chunks,
                                              void* const* v_chunks, int32_t layer_begin,
                                              int32_t layer_end, const int32_t* sel_idx,
                                              int64_t n_sel, const void* q_pre,
                                              const void* k_pre, const void* v_fresh,
                                              const int32_t* coords, void* out, float* lse,
                                              void* workspace, size_t workspace_bytes,
                                              void* stream);

/* Thread-local text describing the last non-OK status on this thread. */
const char* cs_last_error(void);

/* ---------------------------------------------------------------------------
 * Kernel tracing (measurement aid, off by default).
 * While enabled, every kernel the library launches carries a pair of
 * hipEvents that its own dispatch stamps at the kernel's start and end
 * (hipExtLaunchKernel: no extra packets on the stream, so tracing leaves the
 * timeline as it is).  cs_trace_collect() synchronises those events and
 * accumulates, per kernel name, the number of launches and their total
 * duration.  The trace state is shared by all threads and guarded by a
 * lock; a kernel's events reach the collector once its launch is enqueued,
 * so a collect running beside launches on other threads never waits on a
 * half-enqueued pair.  A collect that fails keeps the launches it had not
 * reached.
 *
 * cs_trace_only(names) narrows tracing to the kernels named in a
 * comma-separated list (NULL or "": every kernel); the list is copied.  The
 * events cost the GPU a few microseconds per traced launch, so a caller that
 * needs one kernel's durations can leave the others untraced. */
cs_status cs_trace_enable(int32_t on);
cs_status cs_trace_only(const char* names);
cs_status cs_trace_collect(void);
int32_t cs_trace_count(void);
cs_status cs_trace_get(int32_t i, const char** name, int64_t* launches,
                       double* total_ms);
void cs_trace_reset(void);

#ifdef __cplusplus
}
#endif

#endif /* CHRONOSTITCH_H */
