// Gather of the routed groups' exact token K/V (Sec. 4.3, store operation
// "gather exact token K/V").
//
// A pure indexed copy: every thread moves 16-byte vectors of K and V from the
// source rows of its group to the contiguous routed buffer.  Consecutive
// threads take consecutive vectors of one destination row, so both the reads
// (one group = `group` contiguous source rows) and the writes are fully
// coalesced.  The source may be device memory or pinned host memory mapped
// into the device address space; in the latter case only the routed groups
// cross the host link.  Each thread issues all its loads before its stores.
#include "hga_device.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 4;

template <int D, int V>
__global__ __launch_bounds__(kThreads) void gather_kernel(
    const int32_t* __restrict__ group_idx, int q_chunk0, int n_q_chunks, int topk, int group,
    int gpc, const unsigned char* __restrict__ k_src, const unsigned char* __restrict__ v_src,
    int64_t src_tokens, unsigned char* __restrict__ k_out, unsigned char* __restrict__ v_out,
    int64_t total_vec, int elem_bytes) {
    constexpr int VPR = D / V;
    const int64_t row_bytes = static_cast<int64_t>(D) * elem_bytes;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
    const int rows_per_unit = topk * group;
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; base < total_vec;
         base += stride * kUnroll) {
        vec16 kv[kUnroll], vv[kUnroll];
        int64_t dst[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t idx = base + u * stride;
            dst[u] = -1;
            if (idx >= total_vec) continue;
            const int64_t row = idx / VPR;
            const int cv = static_cast<int>(idx % VPR);
            const int64_t unit = row / rows_per_unit;          // (b * n_kv + j) * n_q_chunks + i
            const int in_unit = static_cast<int>(row % rows_per_unit);
            const int s = in_unit / group, o = in_unit % group;
            const int i = static_cast<int>(unit % n_q_chunks);
            const int64_t bh = unit / n_q_chunks;
            const int g = group_idx[unit * topk + s];
            const int c = q_chunk0 + i;
            const bool ok = g >= 0 && g < c * gpc &&
                            static_cast<int64_t>(g + 1) * group <= src_tokens;
            dst[u] = row * row_bytes + cv * 16;
            if (ok) {
                const int64_t src = (bh * src_tokens + static_cast<int64_t>(g) * group + o) *
                                        row_bytes + cv * 16;
                kv[u] = load16(k_src + src);
                vv[u] = load16(v_src + src);
            } else {
                kv[u] = vec16{{0u, 0u, 0u, 0u}};
                vv[u] = kv[u];
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            if (dst[u] < 0) continue;
            store16(k_out + dst[u], kv[u]);
            store16(v_out + dst[u], vv[u]);
        }
    }
}

// ---- gather through a warm cache (Sec. 4.3 "warm" tier) ----------------
//
// One workgroup per (batch, KV head), which owns that head's cache
// partition: n_slots slots of `group` rows of K and V in device memory, the
// maps slot -> group (slot_group), group -> slot (group_slot) and the tick
// of each slot's last use (slot_used).  The maps are only written here and
// stay mutual inverses: group_slot[g] = v exactly when slot_group[v] = g.
// Bookkeeping, with every global read issued by the whole workgroup at once
// (two round trips):
//   1. the slot ticks and owners, and the routed ids of the query chunk
//      (ids outside [0, c*C/G) or past the source become absent; a repeated
//      id copies its first occurrence's rows); then each id's slot;
//   2. hits: ids that have a slot; the slot gets this call's tick;
//   3. victims for the misses: the least recently used slots (smallest
//      tick, then lowest slot; never-used slots first), chosen with the
//      selection code of the routing over keys ((~(tick + 1)) << 32 | ~slot);
//      a slot hit in this call is keyed 0, so with n_slots >= K_g it is
//      never chosen;
//   4. misses take the victims in ascending slot order, in routed order, and
//      the maps are updated.
// It leaves a copy plan per routed entry; a second kernel, spread over the
// chip, then copies: a miss from the source (pinned host memory through its
// device mapping, or device memory) into both its cache slot and the routed
// buffer, a hit from its cache slot into the routed buffer, an absent id as
// zeros.  No slot is both read and written in one call.
enum CacheKind { kAbsentId = 0, kHit = 1, kMiss = 2, kHitDup = 3, kMissDup = 4 };

constexpr int kCacheThreads = 1024;

// The copy plan of routed entry s (entry_slot[bh][s]): -1 absent (zero
// rows); v >= 0 a hit (rows from cache slot v); -2 - v a miss (rows from the
// source into slot v and the routed buffer); -2 - n_slots a repeated miss
// (rows from the source, routed buffer only).
__global__ __launch_bounds__(kCacheThreads) void cache_plan_kernel(
    const int32_t* __restrict__ group_idx, int c, int topk, int group, int gpc,
    int64_t src_tokens, int n_slots, int32_t* __restrict__ slot_group,
    int32_t* __restrict__ slot_used, int32_t* __restrict__ group_slot, int64_t n_groups,
    int tick, int32_t* __restrict__ entry_slot, int32_t* __restrict__ n_fetched) {
    extern __shared__ __align__(16) unsigned char smem[];
    uint64_t* keys = reinterpret_cast<uint64_t*>(smem);
    int* s_owner = reinterpret_cast<int*>(keys + n_slots);  // slot_group before this call
    int* s_gid = s_owner + n_slots;
    int* s_kind = s_gid + topk;
    int* s_slot = s_kind + topk;
    int* s_sel = s_slot + topk;
    int* s_scr = s_sel + topk;
    const int bh = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t* gi = group_idx + static_cast<int64_t>(bh) * topk;
    int32_t* sg = slot_group + static_cast<int64_t>(bh) * n_slots;
    int32_t* su = slot_used + static_cast<int64_t>(bh) * n_slots;
    int32_t* gs = group_slot + static_cast<int64_t>(bh) * n_groups;

    // 1. ticks, owners and ids, all requested together
    for (int v = tid; v < n_slots; v += kCacheThreads) {
        const int used = su[v], owner = sg[v];
        const uint32_t age = 0xffffffffu - static_cast<uint32_t>(used + 1);
        keys[v] = (static_cast<uint64_t>(age) << 32) | (0xffffffffu - static_cast<uint32_t>(v));
        s_owner[v] = owner;
    }
    for (int s = tid; s < topk; s += kCacheThreads) {
        const int g = gi[s];
        const bool ok = g >= 0 && g < c * gpc && static_cast<int64_t>(g + 1) * group <= src_tokens;
        s_gid[s] = ok ? g : -1;
    }
    __syncthreads();
    // each id's slot (-1: not cached), first occurrences only
    for (int s = tid; s < topk; s += kCacheThreads) {
        const int g = s_gid[s];
        int kind = kAbsentId, slot = -1;
        if (g >= 0) {
            int first = s;
            for (int t = 0; t < s; ++t)
                if (s_gid[t] == g) {
                    first = t;
                    break;
                }
            if (first != s) {
                kind = kHitDup;  // resolved once the first one has its slot
                slot = first;
            } else {
                const int v = gs[g];
                if (v >= 0 && v < n_slots) {
                    kind = kHit;
                    slot = v;
                } else {
                    kind = kMiss;
                }
            }
        }
        s_kind[s] = kind;
        s_slot[s] = slot;
    }
    __syncthreads();

    if (wave == 0) {
        // 2. hits keep their slots
        int n_miss = 0;
        for (int s0 = 0; s0 < topk; s0 += 64) {
            const int s = s0 + lane;
            const int kind = s < topk ? s_kind[s] : kAbsentId;
            if (kind == kHit) {
                const int v = s_slot[s];
                su[v] = tick;
                keys[v] = 0;  // never a victim in this call
            }
            const uint64_t mm = __ballot(kind == kMiss);
            if (kind == kMiss) s_slot[s] = n_miss + __popcll(mm & ((uint64_t(1) << lane) - 1));
            n_miss += __popcll(mm);
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        // 3. victims, 4. the misses take them
        if (n_miss > 0) wave_select_topk(keys, n_slots, n_miss, s_sel, s_scr, true);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        for (int s = lane; s < topk; s += 64) {
            if (s_kind[s] != kMiss) continue;
            const int v = s_sel[s_slot[s]];
            const int g = s_gid[s];
            const int old = s_owner[v];
            if (old >= 0 && old < n_groups) gs[old] = -1;
            sg[v] = g;
            gs[g] = v;
            su[v] = tick;
            s_slot[s] = v;
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        for (int s = lane; s < topk; s += 64) {
            if (s_kind[s] != kHitDup) continue;
            const int first = s_slot[s];
            s_kind[s] = s_kind[first] == kMiss ? kMissDup : kHitDup;
            s_slot[s] = s_slot[first];
        }
        if (lane == 0 && n_fetched) n_fetched[bh] = n_miss;
    }
    __syncthreads();
    for (int s = tid; s < topk; s += kCacheThreads) {
        const int kind = s_kind[s], v = s_slot[s];
        int code = -1;
        if (kind == kHit || kind == kHitDup) code = v;
        else if (kind == kMiss) code = -2 - v;
        else if (kind == kMissDup) code = -2 - n_slots;
        entry_slot[static_cast<int64_t>(bh) * topk + s] = code;
    }
}

// The copies of the plan, a grid-stride loop over 16-byte vectors of the
// routed rows (as gather_kernel), so the misses' reads of the source spread
// over the whole chip.
template <int D, int V>
__global__ __launch_bounds__(kThreads) void cache_copy_kernel(
    const int32_t* __restrict__ group_idx, const int32_t* __restrict__ entry_slot, int topk,
    int group, const unsigned char* __restrict__ k_src, const unsigned char* __restrict__ v_src,
    int64_t src_tokens, unsigned char* __restrict__ cache_k, unsigned char* __restrict__ cache_v,
    int n_slots, unsigned char* __restrict__ k_out, unsigned char* __restrict__ v_out,
    int64_t total_vec, int elem_bytes) {
    constexpr int VPR = D / V;
    const int64_t row_bytes = static_cast<int64_t>(D) * elem_bytes;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
    const int rows_per_unit = topk * group;
    for (int64_t base = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; base < total_vec;
         base += stride * kUnroll) {
        vec16 kv[kUnroll], vv[kUnroll];
        int64_t dst[kUnroll], cdst[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t idx = base + u * stride;
            dst[u] = -1;
            cdst[u] = -1;
            if (idx >= total_vec) continue;
            const int64_t row = idx / VPR;
            const int cv = static_cast<int>(idx % VPR);
            const int64_t bh = row / rows_per_unit;
            const int in_unit = static_cast<int>(row % rows_per_unit);
            const int s = in_unit / group, o = in_unit % group;
            const int code = entry_slot[bh * topk + s];
            dst[u] = row * row_bytes + cv * 16;
            kv[u] = vec16{{0u, 0u, 0u, 0u}};
            vv[u] = kv[u];
            if (code >= 0) {
                const int64_t src = ((bh * n_slots + code) * group + o) * row_bytes + cv * 16;
                kv[u] = load16(cache_k + src);
                vv[u] = load16(cache_v + src);
            } else if (code <= -2) {
                const int g = group_idx[bh * topk + s];
                const int64_t src = (bh * src_tokens + static_cast<int64_t>(g) * group + o) *
                                        row_bytes + cv * 16;
                kv[u] = load16(k_src + src);
                vv[u] = load16(v_src + src);
                const int v = -2 - code;
                if (v < n_slots) cdst[u] = ((bh * n_slots + v) * group + o) * row_bytes + cv * 16;
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            if (dst[u] < 0) continue;
            store16(k_out + dst[u], kv[u]);
            store16(v_out + dst[u], vv[u]);
            if (cdst[u] >= 0) {
                store16(cache_k + cdst[u], kv[u]);
                store16(cache_v + cdst[u], vv[u]);
            }
        }
    }
}

}  // namespace

size_t gather_cached_lds_bytes(const hga_plan& plan, int n_slots) {
    return (sizeof(uint64_t) + sizeof(int)) * static_cast<size_t>(n_slots) +
           5 * sizeof(int) * static_cast<size_t>(plan.p.topk_groups);
}

hipError_t launch_gather_kv_cached(const hga_plan& plan, const int32_t* group_idx, int c,
                                   const void* k_src, const void* v_src, int64_t src_tokens,
                                   void* cache_k, void* cache_v, int n_slots, int32_t* slot_group,
                                   int32_t* slot_used, int32_t* group_slot, int64_t n_groups,
                                   int tick, int32_t* entry_slot, void* k_routed, void* v_routed,
                                   int32_t* n_fetched, hipStream_t stream) {
    const hga_params& p = plan.p;
    const int eb = p.dtype == HGA_F32 ? 4 : 2;
    const int V = 16 / eb;
    const int units = p.batch * p.n_kv_heads;
    const size_t lds = gather_cached_lds_bytes(plan, n_slots);
    const int gpc = p.chunk / p.group;
    hipLaunchKernelGGL(cache_plan_kernel, dim3(units), dim3(kCacheThreads), lds, stream,
                       group_idx, c, p.topk_groups, p.group, gpc, src_tokens, n_slots, slot_group,
                       slot_used, group_slot, n_groups, tick, entry_slot, n_fetched);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t total_vec =
        static_cast<int64_t>(units) * p.topk_groups * p.group * (p.head_dim / V);
    int64_t blocks = (total_vec + kThreads * kUnroll - 1) / (kThreads * kUnroll);
    if (blocks > 65536) blocks = 65536;
    auto ks = static_cast<const unsigned char*>(k_src);
    auto vs = static_cast<const unsigned char*>(v_src);
    auto ck = static_cast<unsigned char*>(cache_k);
    auto cv = static_cast<unsigned char*>(cache_v);
    auto ko = static_cast<unsigned char*>(k_routed);
    auto vo = static_cast<unsigned char*>(v_routed);
#define HGA_CACHE_COPY(DD, VV)                                                                  \
    hipLaunchKernelGGL((cache_copy_kernel<DD, VV>), dim3(static_cast<unsigned>(blocks)),       \
                       dim3(kThreads), 0, stream, group_idx, entry_slot, p.topk_groups, p.group, \
                       ks, vs, src_tokens, ck, cv, n_slots, ko, vo, total_vec, eb)
    if (p.head_dim == 64) {
        if (V == 4) HGA_CACHE_COPY(64, 4); else HGA_CACHE_COPY(64, 8);
    } else {
        if (V == 4) HGA_CACHE_COPY(128, 4); else HGA_CACHE_COPY(128, 8);
    }
#undef HGA_CACHE_COPY
    return hipGetLastError();
}

hipError_t launch_gather_kv(const hga_plan& plan, const int32_t* group_idx, int q_chunk0,
                            int n_q_chunks, const void* k_src, const void* v_src,
                            int64_t src_tokens, void* k_routed, void* v_routed,
                            hipStream_t stream) {
    const hga_params& p = plan.p;
    const int eb = p.dtype == HGA_F32 ? 4 : 2;
    const int V = 16 / eb;
    const int64_t rows = static_cast<int64_t>(p.batch) * p.n_kv_heads * n_q_chunks *
                         p.topk_groups * p.group;
    const int64_t total_vec = rows * (p.head_dim / V);
    if (total_vec == 0) return hipSuccess;
    int64_t blocks = (total_vec + kThreads * kUnroll - 1) / (kThreads * kUnroll);
    if (blocks > 65536) blocks = 65536;
    const int gpc = p.chunk / p.group;
    auto ks = static_cast<const unsigned char*>(k_src);
    auto vs = static_cast<const unsigned char*>(v_src);
    auto ko = static_cast<unsigned char*>(k_routed);
    auto vo = static_cast<unsigned char*>(v_routed);
#define HGA_GATHER(DD, VV)                                                                        \
    hipLaunchKernelGGL((gather_kernel<DD, VV>), dim3(static_cast<unsigned>(blocks)),             \
                       dim3(kThreads), 0, stream, group_idx, q_chunk0, n_q_chunks, p.topk_groups, \
                       p.group, gpc, ks, vs, src_tokens, ko, vo, total_vec, eb)
    if (p.head_dim == 64) {
        if (V == 4) HGA_GATHER(64, 4); else HGA_GATHER(64, 8);
    } else {
        if (V == 4) HGA_GATHER(128, 4); else HGA_GATHER(128, 8);
    }
#undef HGA_GATHER
    return hipGetLastError();
}

}  // namespace hga
