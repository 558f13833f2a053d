// Internal declarations shared by the host ABI and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "hga.h"

struct hga_plan {
    hga_params p;         // resolved: hf_pairs_* filled in
    int device;
    int max_lds;          // device limit on LDS bytes per workgroup
    int n_cu;             // compute units of the device
    float* phase_group;   // device [2][group][head_dim/2]: cos then sin of phi_p(o), span = group
    float* phase_psi;     // device [2][chunk/group][head_dim/2]: cos, sin of psi_g theta_p
    // routing workspace of the spread form (launches of a few units): keys
    // [kRouteSpreadUnits][kRouteSpreadCandidates], then one counter per unit
    // (zero between calls)
    uint64_t* route_keys;
    unsigned* route_count;
};

namespace hga {

// Most middle chunks a query chunk may have (2^18: a 16.7M-token context);
// beyond 1024 the routing streams the table and keeps no per-candidate list.
constexpr int kMaxChunkCandidates = 1 << 18;
constexpr int kMaxTopK = 512;
// Launches of at most this many units with this many middle chunks or fewer
// may take the spread routing form, whose keys live in the plan's workspace.
constexpr int kRouteSpreadUnits = 16;
constexpr int kRouteSpreadCandidates = 4096;
inline size_t route_workspace_bytes() {
    return sizeof(uint64_t) * kRouteSpreadUnits * kRouteSpreadCandidates +
           sizeof(unsigned) * kRouteSpreadUnits;
}

// Runs `set` (a kernel's one-time attribute setting, e.g. its dynamic LDS
// limit) once per device: function attributes belong to the kernel on each
// device, so a process that launches on several devices sets them on each.
// `done` holds one bit per device id below 64 (larger ids set every time).
template <typename F>
inline hipError_t once_per_device(std::atomic<uint64_t>& done, int device, F set) {
    const uint64_t bit = device >= 0 && device < 64 ? uint64_t(1) << device : 0;
    if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
    const hipError_t e = set();
    if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_release);
    return e;
}

// visible-window length W = max(L, force_prev ? 1 : 0)
inline int recent_window(const hga_params& p) {
    return p.keep_last > (p.force_prev ? 1 : 0) ? p.keep_last : (p.force_prev ? 1 : 0);
}

// Number of routable middle chunks of query chunk c: |[F, c - W)|.
inline int middle_count(const hga_params& p, int c) {
    int n = c - recent_window(p) - p.keep_first;
    return n > 0 ? n : 0;
}

// LDS a routing workgroup of one wavefront needs for `n_max` middle-chunk
// candidates, with or without the fused group refinement.
size_t route_lds_bytes(const hga_plan& plan, int n_max, bool groups);

// Kernel launchers; each returns hipSuccess or the launch error.
hipError_t launch_build_summaries(const hga_plan& plan, const void* k_rot, int64_t k_tokens,
                                  int k_chunk0, int chunk_begin, int chunk_end, float* chunk_sum,
                                  float* group_sum, int table_chunks, hipStream_t stream);

hipError_t launch_route_chunks(const hga_plan& plan, const void* q_rot, int q_chunk0,
                               int n_q_chunks, const float* chunk_sum, int table_chunks,
                               float* qbar, int32_t* chunk_idx, hipStream_t stream);

hipError_t launch_route(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                        const float* chunk_sum, const float* group_sum, int table_chunks,
                        float* qbar, int32_t* chunk_idx, int32_t* group_idx, hipStream_t stream);

// hga_route's selection stages from a given q_bar (it is read, not written).
hipError_t launch_route_from_qbar(const hga_plan& plan, const float* qbar, int q_chunk0,
                                  int n_q_chunks, const float* chunk_sum, const float* group_sum,
                                  int table_chunks, int32_t* chunk_idx, int32_t* group_idx,
                                  hipStream_t stream);

// Summaries of [chunk_begin, chunk_end) and q_bar of the query chunks in one
// launch (independent work items).
hipError_t launch_summaries_qbar(const hga_plan& plan, const void* k_rot, int64_t k_tokens,
                                 int k_chunk0, int chunk_begin, int chunk_end, float* chunk_sum,
                                 float* group_sum, int table_chunks, const void* q_rot,
                                 int q_chunk0, int n_q_chunks, float* qbar, hipStream_t stream);

hipError_t launch_route_groups(const hga_plan& plan, const float* qbar, const int32_t* chunk_idx,
                               int q_chunk0, int n_q_chunks, const float* group_sum,
                               int table_chunks, int32_t* group_idx, hipStream_t stream);

hipError_t launch_gather_kv(const hga_plan& plan, const int32_t* group_idx, int q_chunk0,
                            int n_q_chunks, const void* k_src, const void* v_src,
                            int64_t src_tokens, void* k_routed, void* v_routed,
                            hipStream_t stream);

// Gather of one query chunk's routed groups through a warm LRU cache of
// groups in device memory (one workgroup per (batch, KV head)).
size_t gather_cached_lds_bytes(const hga_plan& plan, int n_slots);
hipError_t launch_gather_kv_cached(const hga_plan& plan, const int32_t* group_idx, int c,
                                   const void* k_src, const void* v_src, int64_t src_tokens,
                                   void* cache_k, void* cache_v, int n_slots, int32_t* slot_group,
                                   int32_t* slot_used, int32_t* group_slot, int64_t n_groups,
                                   int tick, int32_t* entry_slot, void* k_routed, void* v_routed,
                                   int32_t* n_fetched, hipStream_t stream);

// start/stop (may be null) are recorded by the attention kernel's dispatch.
hipError_t launch_attend(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                         const void* k_res, const void* v_res, int64_t res_tokens,
                         const int32_t* res_slot, const void* k_routed, const void* v_routed,
                         const int32_t* group_idx, void* out, float* lse, hipEvent_t start,
                         hipEvent_t stop, hipStream_t stream);

// Device scratch the library holds on every device it runs on, for the
// allocation-free split attention (its partial results): 16 MiB, the most a
// decode block of 32 query heads over 4 KV heads at d128 uses for its splits.
constexpr int64_t kStaticScratchBytes = int64_t(16) << 20;
// Takes the array's device address for `device` (current) once; later calls
// return at once.
hipError_t static_scratch_init(int device);
// The address static_scratch_init recorded for `device`, or null.
void* static_scratch(int device);

// Attention with each unit's key tiles divided among several workgroups
// (bf16, r >= 2) whose partial results go to `workspace` and are merged by a
// second kernel; other configurations, or a workspace too small for two
// splits, run launch_attend.
constexpr int kMaxSplit = 16;  // at most the merge kernel's slots
int64_t attend_split_bytes_per_split(const hga_plan& plan, int n_q_chunks);
// Whether launch_attend_split may split these query chunks at all (bf16,
// several query heads per KV head); otherwise it runs launch_attend.
bool attend_split_applies(const hga_plan& plan);
hipError_t launch_attend_split(const hga_plan& plan, const void* q_rot, int q_chunk0,
                               int n_q_chunks, const void* k_res, const void* v_res,
                               int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                               const void* v_routed, const int32_t* group_idx, void* out,
                               float* lse, void* workspace, int64_t workspace_bytes,
                               hipStream_t stream);

// Backward of the attention (bf16): dq written, dk and dv (fp32, resident
// layout) accumulated into.
size_t attend_backward_lds_bytes(const hga_plan& plan);
hipError_t launch_attend_backward(const hga_plan& plan, const void* q_rot, int q_chunk0,
                                  int n_q_chunks, const void* k_res, const void* v_res,
                                  int64_t res_tokens, const int32_t* group_idx, const void* out,
                                  const float* lse, const void* dout, float* dq, float* dk,
                                  float* dv, hipStream_t stream);

// The gather fused into the split attention: routed rows copied from
// k_src / v_src (src_tokens rows per head, device memory or the device
// mapping of pinned host memory) and written to k_routed / v_routed; the
// visible and current chunks from k_res / v_res (res_slot as for
// launch_attend).
hipError_t launch_gather_attend_split(const hga_plan& plan, const void* q_rot, int q_chunk0,
                                      int n_q_chunks, const void* k_res, const void* v_res,
                                      int64_t res_tokens, const int32_t* res_slot,
                                      const void* k_src, const void* v_src, int64_t src_tokens,
                                      const int32_t* group_idx, void* k_routed, void* v_routed,
                                      void* out, float* lse, void* workspace,
                                      int64_t workspace_bytes, hipStream_t stream);

// The gather of the routed rows fused into the attention (prefill layout:
// resident K/V indexed by token, no slot map); writes k_routed / v_routed as
// launch_gather_kv does.  start/stop as for launch_attend.
hipError_t launch_gather_attend(const hga_plan& plan, const void* q_rot, int q_chunk0,
                                int n_q_chunks, const void* k_res, const void* v_res,
                                int64_t res_tokens, const int32_t* group_idx, void* k_routed,
                                void* v_routed, void* out, float* lse, hipEvent_t start,
                                hipEvent_t stop, hipStream_t stream);

}  // namespace hga
