/*
 * hga.h -- C ABI of the MI355X (gfx950) routed-attention path of
 * Hierarchical Global Attention (HGA).
 *
 * The five calls follow the paper's statement of the problem.  Its tiered
 * K/V store (Sec. 4.3) exposes four operations -- append a closed chunk,
 * read chunk summaries, fetch group summaries, gather exact token K/V --
 * and the routed module then runs exact-token attention (Sec. 3.4):
 *
 *   hga_build_summaries  mixed-RoPE chunk and group key summaries (Sec. 3.1, 3.2)
 *   hga_route_chunks     query-chunk -> chunk scoring, top-K_c (Sec. 3.3)
 *   hga_route_groups     group refinement inside the chosen chunks, top-K_g (Sec. 3.3)
 *   hga_route            both routing stages in one launch, same outputs
 *   hga_build_summaries_qbar  summaries and the routing query means in one launch
 *   hga_route_qbar       hga_route's selection stages from a given q_bar
 *   hga_gather_kv        copy the routed groups' exact token K/V (Sec. 4.3)
 *   hga_attend           exact causal softmax attention, Eq. (1), over the
 *                        current chunk, the always-visible chunks and the
 *                        routed groups (Sec. 3.3, 3.4)
 *
 * Conventions shared by every call
 * --------------------------------
 * - Tensors are row-major "BHND": [batch, heads, tokens, head_dim] with
 *   head_dim contiguous.  Q and K arrive already rotated by RoPE at their
 *   absolute positions (rotate-half pairing: dimension p pairs with
 *   p + head_dim/2).  Chunk c is tokens [c*chunk, (c+1)*chunk).
 * - Query head h reads KV head h / (n_q_heads / n_kv_heads) (GQA, Sec. 2);
 *   routing is per KV head and shared by its query heads.
 * - Element type of Q, K, V, the routed buffers and the output: the plan's
 *   dtype (fp32 or bf16).  Summaries and query means are fp32; indices are
 *   int32, ascending, padded with -1.
 * - Every buffer is owned by the caller; the calls allocate nothing.
 *   Pointers are device pointers unless stated otherwise.  Tensor pointers
 *   must be 16-byte aligned, index pointers 4-byte aligned.
 * - Every call is asynchronous on `stream` (a hipStream_t; NULL = the
 *   legacy default stream) and must run with the plan's device current.
 *   All argument checks happen on the host before anything is launched; a
 *   failing check launches nothing and returns a negative hga_status.
 * - Error strings: hga_last_error() returns the message of the last failing
 *   call on the calling thread.  No C++ exception crosses this interface.
 * - The library keeps no state between calls besides the plan, so calls on
 *   different streams may overlap as long as their buffers do not -- except
 *   hga_route_qbar calls on one plan, which may share the plan's routing
 *   workspace (and hga_attend_split_static calls on one device).
 */
#ifndef HGA_H
#define HGA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    HGA_OK = 0,
    HGA_EINVAL = -1,        /* invalid argument: null pointer, size or id out of range */
    HGA_EUNSUPPORTED = -2,  /* valid by the method but outside what the kernels cover  */
    HGA_EALIGN = -3,        /* misaligned pointer                                       */
    HGA_EHIP = -4           /* a HIP runtime call failed (no device, launch failure...) */
} hga_status;

typedef enum { HGA_F32 = 0, HGA_BF16 = 1 } hga_dtype;

/* Routing configuration (Sec. 3.1-3.3).  Field meaning and accepted values:
 *   batch, n_q_heads, n_kv_heads  >= 1, n_q_heads % n_kv_heads == 0,
 *                                 n_q_heads / n_kv_heads <= 16
 *   head_dim        64 or 128
 *   chunk           C, the chunk length: 64 (Sec. 3.1)
 *   group           g_s, the group length: 8, 16 or 32 (divides chunk)
 *   keep_first      F: the first F chunks are always visible (attention sinks)
 *   keep_last       L: the last L closed chunks are always visible
 *   force_prev      1: the preceding chunk is force-included when L == 0
 *                   (Sec. 3.3 "Deterministic visibility"); 0: not included
 *   topk_chunks     K_c in [1, 512]: chunks kept by chunk routing
 *   topk_groups     K_g in [1, 512]: groups opened by group refinement
 *   hf_pairs_chunk  number of high-frequency RoPE pairs for chunk summaries;
 *   hf_pairs_group  ... for group summaries.  -1 selects the rule "pair p is
 *                   high-frequency when its wavelength 2*pi*base^(2p/d) is at
 *                   most the span" (Sec. 3.2 gives no threshold).  The resolved
 *                   values must satisfy hf_pairs_chunk >= hf_pairs_group (the
 *                   rule always does; HGA_EUNSUPPORTED otherwise).
 *   dtype           hga_dtype of Q/K/V/routed buffers/output
 *   rope_base       RoPE base (> 1), theta_p = base^(-2p/head_dim)
 *
 * Visible closed chunks of query chunk c ("D_c"): chunks [0, min(F, c)) and
 * [max(0, c - W), c) with W = max(L, force_prev ? 1 : 0).  Routable middle
 * ("M_c"): chunks [F, c - W).  Chunk routing keeps min(K_c, |M_c|) chunks;
 * group refinement opens min(K_g, (chunk/group) * that) groups. */
typedef struct {
    int32_t batch;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t chunk;
    int32_t group;
    int32_t keep_first;
    int32_t keep_last;
    int32_t force_prev;
    int32_t topk_chunks;
    int32_t topk_groups;
    int32_t hf_pairs_chunk;
    int32_t hf_pairs_group;
    int32_t dtype;
    double rope_base;
} hga_params;

typedef struct hga_plan hga_plan;

/* Validate `params`, compute the summary phase tables in double precision on
 * the host (stored as fp32) and upload them to the current device.  The plan
 * owns that device memory (a few tens of KiB) and a routing workspace of
 * 512 KiB (see hga_route_qbar), and is bound to the device current at
 * creation.  *plan is set only on HGA_OK.  Returns HGA_EINVAL /
 * HGA_EUNSUPPORTED for bad params before touching the device, HGA_EHIP if
 * there is no usable device. */
hga_status hga_plan_create(const hga_params* params, hga_plan** plan);

/* Release the plan's device memory.  NULL is accepted.  The caller must not
 * destroy a plan while work that uses it is still queued. */
hga_status hga_plan_destroy(hga_plan* plan);

/* Copy the plan's resolved parameters (hf_pairs_* filled in) to *out. */
hga_status hga_plan_params(const hga_plan* plan, hga_params* out);

/* Mixed-RoPE chunk and group key summaries (Sec. 3.2), the store's "append
 * a newly closed chunk" (Sec. 4.3).
 *
 * For each chunk c in [chunk_begin, chunk_end) and each (batch, KV head):
 *   chunk_sum[c]  = mean over the chunk's tokens of R(phi_p(o)) k_rot[t]
 *   group_sum[g]  = the same over each of the chunk/group groups g of c
 * where o = t - span start, phi_p(o) = 0 for the high-frequency pairs
 * (rotated keys are averaged) and ((span-1)/2 - o) * theta_p for the others
 * (which equals averaging the raw keys and rotating at the span's middle).
 *
 *   k_rot        [batch, n_kv_heads, k_tokens, head_dim] plan dtype; its
 *                token 0 is the first token of chunk k_chunk0
 *   chunk_sum    fp32 [batch, n_kv_heads, table_chunks, head_dim]
 *   group_sum    fp32 [batch, n_kv_heads, table_chunks * chunk/group, head_dim]
 * Requires k_chunk0 <= chunk_begin <= chunk_end <= table_chunks and
 * (chunk_end - k_chunk0) * chunk <= k_tokens.  Rows of other chunks are not
 * written.  An empty range is a no-op. */
hga_status hga_build_summaries(const hga_plan* plan, const void* k_rot, int64_t k_tokens,
                               int32_t k_chunk0, int32_t chunk_begin, int32_t chunk_end,
                               float* chunk_sum, float* group_sum, int32_t table_chunks,
                               void* stream);

/* Chunk-level content routing (Sec. 3.3), the store's "read chunk
 * summaries".  For query chunk c = q_chunk0 + i and KV head j:
 *   qbar[i]       = mean of q_rot over the chunk's tokens and the query
 *                   heads of KV head j (chunk-shared routing, Sec. 1)
 *   chunk_idx[i]  = the min(K_c, |M_c|) chunks of M_c with the largest
 *                   qbar . chunk_sum[c'] (unscaled dot product), lowest
 *                   chunk id first among equal scores; ascending, -1 padded
 *
 *   q_rot      [batch, n_q_heads, n_q_chunks * chunk, head_dim] plan dtype:
 *              the tokens of chunks q_chunk0 .. q_chunk0 + n_q_chunks - 1
 *   chunk_sum  fp32 [batch, n_kv_heads, table_chunks, head_dim]; only rows of
 *              middle chunks are read
 *   qbar       fp32 out [batch, n_kv_heads, n_q_chunks, head_dim]
 *   chunk_idx  int32 out [batch, n_kv_heads, n_q_chunks, topk_chunks]
 * Requires q_chunk0 >= 0, n_q_chunks >= 0 and q_chunk0 + n_q_chunks - 1 <=
 * table_chunks.  HGA_EUNSUPPORTED when a query chunk has more than 262144
 * (2^18) middle chunks. */
hga_status hga_route_chunks(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                            int32_t n_q_chunks, const float* chunk_sum, int32_t table_chunks,
                            float* qbar, int32_t* chunk_idx, void* stream);

/* Group refinement (Sec. 3.3), the store's "fetch group summaries".  The
 * candidates of query chunk c are the groups (chunk/group) * c' + i of every
 * chunk c' listed in chunk_idx[i]; the min(K_g, #candidates) groups with the
 * largest qbar . group_sum are kept, globally across the chunks, lowest group
 * id first among equal scores; ascending, -1 padded.
 *
 *   qbar, chunk_idx  as written by hga_route_chunks (chunk ids distinct)
 *   group_sum        fp32 [batch, n_kv_heads, table_chunks * chunk/group, head_dim]
 *   group_idx        int32 out [batch, n_kv_heads, n_q_chunks, topk_groups]
 * chunk_idx entries outside [0, min(c, table_chunks)) are ignored like -1. */
hga_status hga_route_groups(const hga_plan* plan, const float* qbar, const int32_t* chunk_idx,
                            int32_t q_chunk0, int32_t n_q_chunks, const float* group_sum,
                            int32_t table_chunks, int32_t* group_idx, void* stream);

/* Both routing stages of Sec. 3.3 in one launch: writes exactly what
 * hga_route_chunks followed by hga_route_groups on the same arguments writes
 * (qbar, chunk_idx and group_idx bit-identical), without reading qbar or
 * chunk_idx back from memory.  Arguments, layouts, requirements and errors
 * are those of the two calls. */
hga_status hga_route(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                     int32_t n_q_chunks, const float* chunk_sum, const float* group_sum,
                     int32_t table_chunks, float* qbar, int32_t* chunk_idx, int32_t* group_idx,
                     void* stream);

/* hga_build_summaries and the q_bar reduction of hga_route_chunks (Sec. 3.3:
 * the mean of q_rot over each query chunk's tokens and the query heads of its
 * KV head) in one launch: the two read different tensors (K and Q) and do
 * not depend on each other.  chunk_sum/group_sum receive exactly what
 * hga_build_summaries writes, and qbar exactly what hga_route_chunks (or
 * hga_route) writes for the same query rows.
 *
 *   k_rot .. table_chunks   as for hga_build_summaries
 *   q_rot                   [batch, n_q_heads, n_q_chunks * chunk, head_dim]
 *                           plan dtype (query chunks q_chunk0 ..)
 *   qbar                    fp32 out [batch, n_kv_heads, n_q_chunks, head_dim]
 * Requirements and errors: those of hga_build_summaries, plus q_chunk0 >= 0
 * and n_q_chunks >= 0.  Either part may be empty. */
hga_status hga_build_summaries_qbar(const hga_plan* plan, const void* k_rot, int64_t k_tokens,
                                    int32_t k_chunk0, int32_t chunk_begin, int32_t chunk_end,
                                    float* chunk_sum, float* group_sum, int32_t table_chunks,
                                    const void* q_rot, int32_t q_chunk0, int32_t n_q_chunks,
                                    float* qbar, void* stream);

/* The selection stages of hga_route (chunk scores and top-K_c, group
 * refinement and top-K_g, Sec. 3.3) from a given q_bar, e.g. the one
 * hga_build_summaries_qbar wrote; chunk_idx and group_idx are exactly what
 * hga_route writes when it computes the same q_bar itself.  qbar is read
 * only.  Arguments, layouts, requirements and errors are those of
 * hga_route.  A launch of at most 16 query chunks x KV heads x batch with
 * 256..4096 middle chunks spreads each unit's table scan over several
 * workgroups whose keys meet in the plan's routing workspace: two such calls
 * on one plan must not run at the same time (keep a plan's routing calls on
 * one stream, or use one plan per stream); the workspace is left ready for
 * the next call. */
hga_status hga_route_qbar(const hga_plan* plan, const float* qbar, int32_t q_chunk0,
                          int32_t n_q_chunks, const float* chunk_sum, const float* group_sum,
                          int32_t table_chunks, int32_t* chunk_idx, int32_t* group_idx,
                          void* stream);

/* Gather the exact token K/V of the routed groups (Sec. 4.3, "gathering
 * exact token K/V for the selected chunks or groups").  Slot s of query chunk
 * c = q_chunk0 + i receives tokens [g*group, (g+1)*group) of group
 * g = group_idx[i][s]; slots with g outside [0, c*chunk/group) or beyond
 * src_tokens are zero-filled.
 *
 *   k_src, v_src  [batch, n_kv_heads, src_tokens, head_dim] plan dtype.  With
 *                 src_on_host == 0 they are device pointers.  With
 *                 src_on_host == 1 they are pinned host allocations made with
 *                 hipHostMalloc (mapped); the kernel reads them directly over
 *                 the host link (the paper's RAM-backed cold tier) -- only the
 *                 routed groups cross it.
 *   k_routed, v_routed  out [batch, n_kv_heads, n_q_chunks, topk_groups*group,
 *                 head_dim] plan dtype (device) */
hga_status hga_gather_kv(const hga_plan* plan, const int32_t* group_idx, int32_t q_chunk0,
                         int32_t n_q_chunks, const void* k_src, const void* v_src,
                         int64_t src_tokens, int32_t src_on_host, void* k_routed,
                         void* v_routed, void* stream);

/* Exact-token attention (Sec. 3.4) with the causal softmax of Eq. (1).  For
 * query head h, KV head j = h / (n_q_heads / n_kv_heads), and token t of
 * query chunk c = q_chunk0 + i, the softmax of q.k / sqrt(head_dim) runs over
 *   - the tokens of the visible closed chunks D_c (sinks and recent window),
 *   - the valid rows of the routed buffers (slots s with group_idx[i][s] in
 *     [0, c*chunk/group)),
 *   - the tokens u <= t of the current chunk c,
 * and out = sum_u p_u v_u.  lse = natural-log log-sum-exp of the logits.
 *
 *   q_rot       [batch, n_q_heads, n_q_chunks*chunk, head_dim] plan dtype
 *   k_res,v_res resident K/V [batch, n_kv_heads, res_tokens, head_dim].
 *               res_slot == NULL: chunk c' is at tokens [c'*chunk, ...) and
 *               (q_chunk0 + n_q_chunks) * chunk <= res_tokens is required.
 *               res_slot != NULL: device int32 [q_chunk0 + n_q_chunks]; chunk
 *               c' is at tokens [res_slot[c']*chunk, ...).  Only the entries
 *               of chunks in D_c and of c itself are read; if one is outside
 *               [0, res_tokens/chunk) the rows of that query chunk are NaN.
 *   k_routed, v_routed, group_idx  as produced by hga_gather_kv/route_groups
 *   out         [batch, n_q_heads, n_q_chunks*chunk, head_dim] plan dtype
 *   lse         fp32 [batch, n_q_heads, n_q_chunks*chunk] or NULL
 * HGA_EUNSUPPORTED when one head's resident K/V (res_tokens rows) or the
 * query rows of one KV head span 0xfff00000 bytes or more. */
hga_status hga_attend(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                      int32_t n_q_chunks, const void* k_res, const void* v_res,
                      int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                      const void* v_routed, const int32_t* group_idx, void* out, float* lse,
                      void* stream);

/* hga_attend for measurement: the same work and results, and the attention
 * kernel's own dispatch records start_event when it begins and stop_event
 * when it ends (both hipEvent_t created by the caller; either may be NULL).
 * hipEventElapsedTime between them is the kernel's duration, without the
 * queue time that separate event records on the stream would add.  Same
 * arguments, requirements and errors as hga_attend otherwise. */
hga_status hga_attend_timed(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                            int32_t n_q_chunks, const void* k_res, const void* v_res,
                            int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                            const void* v_routed, const int32_t* group_idx, void* out, float* lse,
                            void* start_event, void* stop_event, void* stream);

/* hga_gather_kv for one query chunk c through a warm cache in device memory
 * (Sec. 4.3: the "warm" tier, a bounded LRU cache of recently routed token
 * K/V; here the cached unit is the routed group, the unit the gather moves).
 * Each (batch, KV head) owns a partition of n_slots slots; a routed group
 * whose slot still holds it is copied from the cache (a hit), every other
 * valid group from k_src/v_src into the least recently used slot and the
 * routed buffer (a miss).  k_routed/v_routed receive exactly what
 * hga_gather_kv(plan, group_idx, c, 1, k_src, v_src, src_tokens,
 * src_on_host, k_routed, v_routed, stream) writes.
 * Replacement: the victims are the slots with the oldest last-use tick
 * (never-used slots first, ties to the lowest slot), taken in ascending slot
 * order by the misses in routed order; hits and misses get `tick`.
 *   group_idx   device int32 [batch, n_kv_heads, 1, topk_groups]; ids outside
 *               [0, c*chunk/group) or past src_tokens are absent (zero rows);
 *               a repeated id gets its first occurrence's rows
 *   k_src,v_src [batch, n_kv_heads, src_tokens, head_dim], device memory
 *               (src_on_host = 0) or pinned mapped host memory (1);
 *               src_tokens >= c * chunk
 *   cache_k, cache_v  device [batch, n_kv_heads, n_slots, group, head_dim]
 *   n_slots     in [topk_groups, 8192] (so that a call never evicts a group
 *               it uses)
 *   slot_group  device int32 [batch, n_kv_heads, n_slots]: group held, -1 empty
 *   slot_used   device int32 [batch, n_kv_heads, n_slots]: tick of last use
 *   group_slot  device int32 [batch, n_kv_heads, map_groups]: slot holding
 *               the group or -1 (a new cache: every entry of the three maps -1)
 *   map_groups  groups per (batch, KV head) partition of group_slot, fixed for
 *               the lifetime of the maps (the partition stride), at least
 *               src_tokens / group: a history that grows between calls keeps
 *               its maps as long as it stays within this capacity
 *   entry_slot  device int32 [batch, n_kv_heads, topk_groups]: the call's
 *               copy plan (written, then read by its second kernel; no
 *               contents are needed before or kept after a call)
 *   tick        >= 0 and greater than every tick of an earlier call on the
 *               same maps (e.g. the block's position in the sequence)
 *   n_fetched   device int32 [batch, n_kv_heads] or NULL: groups read from
 *               k_src/v_src by this call (the misses)
 * The caller owns every buffer; calls on the same maps must be ordered (the
 * same stream).  HGA_EINVAL for an n_slots outside the range, a source
 * shorter than the causal past or longer than map_groups groups. */
hga_status hga_gather_kv_cached(const hga_plan* plan, const int32_t* group_idx, int32_t c,
                                const void* k_src, const void* v_src, int64_t src_tokens,
                                int32_t src_on_host, void* cache_k, void* cache_v,
                                int32_t n_slots, int32_t* slot_group, int32_t* slot_used,
                                int32_t* group_slot, int64_t map_groups, int32_t* entry_slot,
                                int32_t tick, void* k_routed, void* v_routed, int32_t* n_fetched,
                                void* stream);

/* hga_attend for launches with few units (a decode block, one block of a
 * block-sequential prefill), Sec. 3.4: each unit's key tiles (current chunk,
 * visible chunks, routed rows) are divided among up to 16 workgroups, each
 * of which leaves an unnormalised partial result (fp32 output sums, running
 * maximum and weight sum per query row) in `workspace`; a second kernel
 * merges them with the usual softmax rescaling.  The number of splits is
 * chosen from the unit count, the tile count and what the workspace holds.
 * out and lse equal hga_attend's up to fp32 summation order (the softmax is
 * the same; its sums are formed in a different order); with one split
 * (workspace_bytes below two splits' worth, the fp32 plan dtype, or one
 * query head per KV head) this runs hga_attend itself, bit for bit.
 *   workspace        device memory owned by the caller, 16-byte aligned,
 *                    not read before it is written; NULL with
 *                    workspace_bytes = 0 is allowed (one split)
 *   workspace_bytes  its size; hga_attend_split_workspace gives the most
 *                    any call with n_q_chunks query chunks uses
 * Other arguments, layouts, requirements and errors as hga_attend.  Calls
 * that share a workspace must not overlap in time. */
hga_status hga_attend_split(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                            int32_t n_q_chunks, const void* k_res, const void* v_res,
                            int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                            const void* v_routed, const int32_t* group_idx, void* out, float* lse,
                            void* workspace, int64_t workspace_bytes, void* stream);

/* Workspace bytes hga_attend_split uses at most for n_q_chunks query chunks
 * (16 splits of batch x n_kv_heads x n_q_chunks units, each
 * (n_q_heads/n_kv_heads)*chunk rows of head_dim + 2 floats).  -1 on a
 * NULL or invalid plan or n_q_chunks < 0. */
int64_t hga_attend_split_workspace(const hga_plan* plan, int32_t n_q_chunks);

/* hga_attend_split without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the split partial results go to a fixed
 * array of hga_static_scratch_bytes() (16 MiB) that the library holds on every
 * device it runs on, from the first plan created there until the process
 * ends.  The call allocates nothing and writes exactly what
 *   hga_attend_split(..., workspace = that array,
 *                    workspace_bytes = hga_static_scratch_bytes(), stream)
 * writes (same split count, same out and lse bit for bit).
 * Limit: where the split form applies (bf16 plan, several query heads per KV
 * head), HGA_EUNSUPPORTED when two splits of the call's units need more than
 * the array holds (2 * hga_attend_split_workspace(plan, n_q_chunks) / 16 bytes
 * above hga_static_scratch_bytes(); a decode block of 32/4 heads at d128 uses
 * 2 MiB).  Every call on one device shares that device's array: calls that
 * overlap in time on one device (different streams, or threads) race and
 * must be serialised by the caller.  Other arguments, layouts, requirements
 * and errors as hga_attend_split. */
hga_status hga_attend_split_static(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                                   int32_t n_q_chunks, const void* k_res, const void* v_res,
                                   int64_t res_tokens, const int32_t* res_slot,
                                   const void* k_routed, const void* v_routed,
                                   const int32_t* group_idx, void* out, float* lse, void* stream);

/* Size in bytes of the per-device array hga_attend_split_static uses. */
int64_t hga_static_scratch_bytes(void);

/* Backward of hga_attend (Sec. 3.4, Eq. (1)) for the prefill layout and the
 * bf16 plan dtype: the gradients of the attention outputs with respect to
 * the rotated queries and the resident keys and values, the routing held
 * fixed (it is not differentiable).  For query row i of query chunk c and
 * key x of its working set (visible chunks, the routed groups of group_idx
 * valid as in hga_attend, the current chunk's tokens u <= t), with
 * p = exp(q_i.k_x/sqrt(d) - lse_i), D_i = dout_i . out_i,
 * ds = p (dout_i . v_x - D_i):
 *   dq_i = sum_x ds k_x / sqrt(d)                  (written)
 *   dk_x += sum_i ds q_i / sqrt(d), dv_x += sum_i p dout_i   (accumulated)
 * A routed row is resident token g*group + o, so its gradients land there.
 *   q_rot, out, dout  [batch, n_q_heads, n_q_chunks*chunk, head_dim] bf16:
 *               out and lse are hga_attend's results for these inputs
 *   k_res,v_res [batch, n_kv_heads, res_tokens, head_dim] bf16, token-indexed
 *               ((q_chunk0 + n_q_chunks) * chunk <= res_tokens)
 *   group_idx   as for hga_attend
 *   lse         fp32 [batch, n_q_heads, n_q_chunks*chunk] (required)
 *   dq          fp32 like q_rot, written (with GQA groups beyond one
 *               workgroup's query rows the call first keeps D_i in dq's
 *               leading floats, then overwrites all of dq); must not
 *               overlap any other argument
 *   dk, dv      fp32 [batch, n_kv_heads, res_tokens, head_dim], ADDED INTO
 *               (zero them for a plain gradient; the sums over query units
 *               are fp32 atomic adds, so their order, and the last bits, may
 *               vary from call to call)
 * HGA_EUNSUPPORTED for an fp32 plan; other errors as hga_attend. */
hga_status hga_attend_backward(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                               int32_t n_q_chunks, const void* k_res, const void* v_res,
                               int64_t res_tokens, const int32_t* group_idx, const void* out,
                               const float* lse, const void* dout, float* dq, float* dk,
                               float* dv, void* stream);

/* hga_gather_kv followed by hga_attend_split, as one pass, for any layout
 * (Sec. 4.3 gather, Sec. 3.4 attention): the workgroups of a unit's routed
 * tiles copy the routed groups' rows straight from k_src/v_src (rows
 * g*group .. g*group+group-1 of group g, zeros for a padded or future id)
 * while those of its visible tiles already compute, and the staged rows are
 * written to k_routed/v_routed.  With the history in pinned host memory
 * (src_on_host = 1: a decode block) the copies over the host link overlap
 * the attention of the resident chunks instead of preceding it.
 * k_routed, v_routed, out and lse receive exactly what
 *   hga_gather_kv(plan, group_idx, q_chunk0, n_q_chunks, k_src, v_src,
 *                 src_tokens, src_on_host, k_routed, v_routed, stream);
 *   hga_attend_split(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res,
 *                    res_tokens, res_slot, k_routed, v_routed, group_idx,
 *                    out, lse, workspace, workspace_bytes, stream);
 * writes (the same split count: it depends only on the plan, the chunk
 * range and workspace_bytes).
 *   k_src, v_src  [batch, n_kv_heads, src_tokens, head_dim] plan dtype;
 *                 src_tokens >= (q_chunk0 + n_q_chunks - 1) * chunk (the
 *                 causal past of the last query chunk), else HGA_EINVAL
 *   src_on_host   0: device memory; 1: pinned, mapped host memory
 *                 (hipHostMalloc), read through its device mapping
 * Other arguments as hga_gather_kv and hga_attend_split; k_routed/v_routed
 * must not overlap any input.  k_routed = v_routed = NULL: the routed rows
 * are gathered into the kernel's tiles only and not written out (out and
 * lse unchanged); exactly one of them NULL is HGA_EINVAL. */
hga_status hga_gather_attend_split(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                                   int32_t n_q_chunks, const void* k_res, const void* v_res,
                                   int64_t res_tokens, const int32_t* res_slot,
                                   const void* k_src, const void* v_src, int64_t src_tokens,
                                   int32_t src_on_host, const int32_t* group_idx, void* k_routed,
                                   void* v_routed, void* out, float* lse, void* workspace,
                                   int64_t workspace_bytes, void* stream);

/* hga_gather_kv followed by hga_attend, for the prefill layout (resident
 * K/V indexed by token, no res_slot), as one pass: the attention copies each
 * routed group's rows straight from k_res/v_res (Sec. 4.3 gather, Sec. 3.4
 * attention), and the same staged rows are written to k_routed/v_routed.
 * k_routed, v_routed, out and lse receive exactly what
 *   hga_gather_kv(plan, group_idx, q_chunk0, n_q_chunks, k_res, v_res,
 *                 res_tokens, 0, k_routed, v_routed, stream);
 *   hga_attend(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
 *              NULL, k_routed, v_routed, group_idx, out, lse, stream);
 * writes, without reading the routed rows back from k_routed/v_routed.
 * start_event/stop_event (hipEvent_t, either may be NULL) are recorded by
 * the attention kernel's dispatch as in hga_attend_timed (for the fp32 plan
 * dtype the gather runs as its own kernel first, outside the events).
 * Arguments, layouts, requirements and errors are those of the two calls;
 * k_routed/v_routed must not overlap any input.
 * k_routed = v_routed = NULL: the gather's rows go to the attention's
 * on-chip tiles only and are not written to memory (for a caller that needs
 * the output, not the gathered copies: no routed-buffer traffic, 2 bytes x
 * head_dim x 2 per routed row and unit); out and lse are bit-identical to
 * the call with buffers (for the fp32 plan dtype the attention kernel then
 * reads the routed rows from k_res/v_res itself, and no gather kernel runs).
 * Exactly one of them NULL is HGA_EINVAL. */
hga_status hga_gather_attend(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                             int32_t n_q_chunks, const void* k_res, const void* v_res,
                             int64_t res_tokens, const int32_t* group_idx, void* k_routed,
                             void* v_routed, void* out, float* lse, void* start_event,
                             void* stop_event, void* stream);

/* One 64-token block of a block-sequential prefill (the paper's block
 * processing with incremental store appends, Sec. 4.3): for query chunk c,
 *   hga_route(plan, q_block, c, 1, chunk_sum, group_sum, table_chunks,
 *             qbar, chunk_idx, group_idx, stream);
 *   hga_gather_attend(plan, q_block, c, 1, k_res, v_res, res_tokens,
 *                     group_idx, k_routed, v_routed, out, lse, NULL, NULL, stream);
 *   hga_build_summaries(plan, k_res, res_tokens, 0, c, c + 1, chunk_sum,
 *                       group_sum, table_chunks, stream);
 * i.e. the block routes against the summaries of the chunks closed before
 * it, attends, and then appends its own chunk's summaries.  Every argument
 * is checked before the first launch.
 *
 *   q_block      [batch, n_q_heads, chunk, head_dim] plan dtype: the block's
 *                queries (query chunk c)
 *   k_res, v_res [batch, n_kv_heads, res_tokens, head_dim], token-indexed
 *                (res_tokens >= (c + 1) * chunk)
 *   chunk_sum, group_sum  as for hga_build_summaries, table_chunks >= c + 1;
 *                rows of chunks < c are read, the rows of chunk c written
 *   qbar, chunk_idx, group_idx, k_routed, v_routed, out, lse  the outputs of
 *                the three calls for one query chunk ([.., 1, ..] shapes)
 *   workspace, workspace_bytes  NULL and 0: the attention is hga_gather_attend
 *                as above (outputs bit-identical to the bulk prefill's);
 *                otherwise it is hga_gather_attend_split with this workspace
 *                (k_src = k_res, device memory): the block's few units spread
 *                over more workgroups, out and lse equal to the bulk prefill's
 *                up to the split's summation order (routing, summaries and the
 *                routed buffers still bit-identical).  Owned by the caller;
 *                hga_attend_split_workspace(plan, 1) bytes give the most splits.
 * Errors: those of the three calls. */
hga_status hga_block_step(const hga_plan* plan, const void* q_block, int32_t c,
                          const void* k_res, const void* v_res, int64_t res_tokens,
                          float* chunk_sum, float* group_sum, int32_t table_chunks, float* qbar,
                          int32_t* chunk_idx, int32_t* group_idx, void* k_routed, void* v_routed,
                          void* out, float* lse, void* workspace, int64_t workspace_bytes,
                          void* stream);

/* A block-sequential prefill of blocks 0 .. n_blocks-1: hga_block_step for
 * c = 0, 1, ... in order, all enqueued on `stream`.  Block c reads and
 * writes the c-th slice of each block-major buffer:
 *   q_blocks, out   [n_blocks][batch, n_q_heads, chunk, head_dim]
 *   lse             [n_blocks][batch, n_q_heads, chunk] fp32 or NULL
 *   qbar            [n_blocks][batch, n_kv_heads, 1, head_dim] fp32
 *   chunk_idx       [n_blocks][batch, n_kv_heads, 1, topk_chunks] int32
 *   group_idx       [n_blocks][batch, n_kv_heads, 1, topk_groups] int32
 *   k_routed, v_routed  [n_blocks][batch, n_kv_heads, 1, topk_groups*group, head_dim]
 * k_res/v_res hold the whole prompt's keys and values (token-indexed,
 * res_tokens >= n_blocks * chunk); the summary tables are built as the
 * blocks close.  Every block's outputs equal what the bulk prefill
 * (hga_build_summaries, then hga_route and hga_gather_attend over all chunks)
 * writes for the same query chunk.  Arguments are checked before the first
 * launch; an error returned by a later launch leaves the earlier blocks done.
 * workspace / workspace_bytes as for hga_block_step. */
hga_status hga_prefill_blocks(const hga_plan* plan, const void* q_blocks, int32_t n_blocks,
                              const void* k_res, const void* v_res, int64_t res_tokens,
                              float* chunk_sum, float* group_sum, int32_t table_chunks,
                              float* qbar, int32_t* chunk_idx, int32_t* group_idx,
                              void* k_routed, void* v_routed, void* out, float* lse,
                              void* workspace, int64_t workspace_bytes, void* stream);

/* The closed chunks that query chunk c sees besides its own (Sec. 3.3,
 * deterministic visibility): the first min(keep_first, c) chunks and the
 * recent window [max(0, c - W), c), W = max(keep_last, force_prev), in
 * ascending order, without repeats.  These are the chunks the attention
 * reads from the resident K/V for c (through res_slot when one is given),
 * so a caller that keeps a compact resident set takes it from here rather
 * than restating the rule.  Host-only: validates params as hga_plan_create
 * does, touches no device.
 *   params  the routing parameters (hf_pairs_* are not used)
 *   c       query chunk, >= 0
 *   chunks  out, int32[cap] (NULL when cap = 0): the ids, ascending
 *   cap     capacity of chunks
 * Returns the number of visible chunks (which may exceed cap: then only the
 * first cap are written), or a negative hga_status for invalid params or
 * c < 0. */
int32_t hga_visible_chunks(const hga_params* params, int32_t c, int32_t* chunks, int32_t cap);

/* Static description of a status code (never NULL). */
const char* hga_status_string(int32_t status);

/* Message of the last failing call on the calling thread ("" if none). */
const char* hga_last_error(void);

/* Library ABI version: (major << 16) | minor. */
int32_t hga_version(void);

#ifdef __cplusplus
}
#endif

#endif /* HGA_H */
