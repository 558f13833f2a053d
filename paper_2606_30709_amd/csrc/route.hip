// Content-based routing (Sec. 3.3): query-chunk -> chunk scoring with top-K_c
// selection, then group refinement with top-K_g selection.
//
// One wavefront per (batch, KV head, query chunk) unit and up to four units
// per workgroup, each wave with its own LDS region.
// Scores are fp32 dot products in a fixed summation order,
// packed with their candidate id into 64-bit keys
// (larger score first, then lower id) held in LDS, and the wave extracts the top k by repeated wave-wide maxima: each lane
// keeps the best key of its own strided share, so a round costs one wave
// reduction plus one rescan of the winning lane's share.
#include "hga_device.hpp"
#include "hga_internal.hpp"
#include "qbar.hpp"

namespace hga {
namespace {

// Chunk-summary rows staged per LDS block, 64 at either head size: one row
// per lane of the scoring wavefront.  Taller blocks (128 rows at D = 64, one
// round trip for contexts up to 128 chunks) were measured slower: twice the
// prefetch registers and LDS per block, and a longer first load before the
// first scores.
constexpr int table_rows(int) { return 64; }

__device__ __forceinline__ void wave_sync_lds() {
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// x plus the value of the lane that DPP quad permutation kPerm names.
template <int kPerm>
__device__ __forceinline__ float add_quad(float x) {
    return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kPerm, 0xf, 0xf, false));
}

// Scores of 16 * NB candidates by one wavefront.  In each batch of 16, lane l
// works on candidate l/4, on float4 columns 4u + l%4 (u < D/16) of its table
// row, so one load instruction reads 64 contiguous bytes of each of 16 rows;
// all NB * D/16 loads are issued before any is used.  The four partial dot
// products of a row are added pairwise in a fixed order by quad exchanges
// ((p0 + p1) + (p2 + p3), the same value in all four lanes), so scores are
// bit-reproducible.  row_of(k) gives the table row, which is also the
// candidate id, of the batch's k-th candidate (callers clamp k to the last
// valid one); keys[k] is written for k < n_valid.
template <int D, int NB, typename RowOf>
__device__ __forceinline__ void batch_keys(const float* s_q, const float* table, RowOf row_of,
                                           int n_valid, uint64_t* keys) {
    constexpr int U = D / 16;
    const int lane = threadIdx.x & 63;
    const int cand = lane >> 2, qd = lane & 3;
    float4 x[NB][U];
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
        const float* row = table + static_cast<int64_t>(row_of(bb * 16 + cand)) * D;
#pragma unroll
        for (int u = 0; u < U; ++u) x[bb][u] = *reinterpret_cast<const float4*>(row + (4 * u + qd) * 4);
    }
    float4 qv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) qv[u] = *reinterpret_cast<const float4*>(s_q + (4 * u + qd) * 4);
#pragma unroll
    for (int bb = 0; bb < NB; ++bb) {
        float a = 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            a = fmaf(qv[u].x, x[bb][u].x, a);
            a = fmaf(qv[u].y, x[bb][u].y, a);
            a = fmaf(qv[u].z, x[bb][u].z, a);
            a = fmaf(qv[u].w, x[bb][u].w, a);
        }
        a = add_quad<0xb1>(a);  // quad_perm [1,0,3,2]
        a = add_quad<0x4e>(a);  // quad_perm [2,3,0,1]
        const int m = bb * 16 + cand;
        if (qd == 0 && m < n_valid) keys[m] = select_key(a, row_of(m));
    }
}

// Keys of candidates 0 .. n-1 (candidate m at table row row_of(m)), in
// batches of 64, 32 or 16 by what remains.
template <int D, typename RowOf>
__device__ __forceinline__ void score_candidates(const float* s_q, const float* table,
                                                 RowOf row_of, int n, uint64_t* keys) {
    for (int m0 = 0; m0 < n;) {
        const int rem = n - m0;
        auto ro = [&](int k) { return row_of(m0 + (k < rem ? k : rem - 1)); };
        if (D == 64 && rem > 32) {
            batch_keys<D, 4>(s_q, table, ro, rem, keys + m0);
            m0 += 64;
        } else if (rem > 16) {
            batch_keys<D, 2>(s_q, table, ro, rem, keys + m0);
            m0 += 32;
        } else {
            batch_keys<D, 1>(s_q, table, ro, rem, keys + m0);
            m0 += 16;
        }
    }
}

// Per-wave LDS carve-up, 16-byte aligned pieces.
struct WaveLds {
    float* q;        // [D]
    int* list;       // [n_list]
    int* sel;        // [topk]
    int* scr;        // [topk]
    uint64_t* keys;  // [n_keys]
};

__host__ __device__ inline size_t align16(size_t x) { return (x + 15) & ~size_t(15); }

__host__ __device__ inline size_t wave_lds_bytes(int d, int n_list, int topk, int n_keys) {
    return align16(sizeof(float) * d) + align16(sizeof(int) * n_list) +
           2 * align16(sizeof(int) * topk) + align16(sizeof(uint64_t) * (n_keys > 0 ? n_keys : 1));
}

__device__ inline WaveLds carve(unsigned char* base, int d, int n_list, int topk) {
    WaveLds w;
    size_t off = 0;
    w.q = reinterpret_cast<float*>(base + off);
    off += align16(sizeof(float) * d);
    w.list = reinterpret_cast<int*>(base + off);
    off += align16(sizeof(int) * n_list);
    w.sel = reinterpret_cast<int*>(base + off);
    off += align16(sizeof(int) * topk);
    w.scr = reinterpret_cast<int*>(base + off);
    off += align16(sizeof(int) * topk);
    w.keys = reinterpret_cast<uint64_t*>(base + off);
    return w;
}

// Query-chunk routing for up to four consecutive query chunks of one
// (batch, KV head), in a workgroup of four wavefronts.  Wavefront w < units
// owns query chunk w of the group and computes its q_bar; all four stage the
// chunk-summary table in LDS, table_rows(D) rows at a time (the next block's
// rows are loaded into registers while the current block is scored, and the
// first block's while q_bar is formed), and each owning wavefront scores its
// own middle chunks (one table row per lane and 64 rows; four partial dot
// products over the dimensions d = 0, 1, 2, 3 mod 4, each in order, added
// pairwise) and selects
// its top K_c.  With kGroups, the same wavefront goes on
// to group refinement of its chosen chunks (the work of route_groups_kernel,
// without a second launch or the q_bar/chunk_idx round trip through memory).
template <typename T, int D, bool kGroups, bool kQbarIn>
__global__ __launch_bounds__(256) void route_kernel(
    const T* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const float* __restrict__ chunk_sum,
    const float* __restrict__ group_sum, int table_chunks, float* __restrict__ qbar,
    int32_t* __restrict__ chunk_idx, int32_t* __restrict__ group_idx, int n_q_heads, int n_kv,
    int keep_first, int window, int topk, int topk_groups, int gpc_shift, int units_per_block,
    size_t wave_bytes) {
    constexpr int kThreads = 256;
    constexpr int TB = table_rows(D);       // table rows per LDS block
    constexpr int TS = D + 4;               // padded LDS row stride (floats)
    constexpr int F4 = D / 4;               // float4 per table row
    constexpr int PF = TB * F4 / kThreads;  // float4 per thread per table block
    static_assert(PF >= 1 && PF * kThreads == TB * F4, "table block split");
    extern __shared__ __align__(16) unsigned char smem_raw[];
    float* s_tab = reinterpret_cast<float*>(smem_raw);
    unsigned char* wave_base = smem_raw + align16(sizeof(float) * TB * TS);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int blocks_per_head = (n_q_chunks + units_per_block - 1) / units_per_block;
    const int bh = blockIdx.x / blocks_per_head;
    const int first_i = (blockIdx.x % blocks_per_head) * units_per_block;
    const int i = first_i + wave;
    const bool active = wave < units_per_block && i < n_q_chunks;
    const int gpc = 1 << gpc_shift;
    const int b = bh / n_kv, j = bh % n_kv;
    const int r = n_q_heads / n_kv;
    const int c = q_chunk0 + (active ? i : 0);
    const int64_t unit = static_cast<int64_t>(bh) * n_q_chunks + i;

    // Table rows [keep_first, hi) are needed by some wavefront of the group;
    // the descriptor covers exactly those, so loads past them return zeros.
    const int last_i = min(n_q_chunks, first_i + units_per_block) - 1;
    const int hi = q_chunk0 + last_i - window;
    const float* table = chunk_sum + static_cast<int64_t>(bh) * table_chunks * D;
    const buf_rsrc t_rsrc =
        make_rsrc(table, hi > 0 ? static_cast<uint32_t>(hi) * D * sizeof(float) : 0u);
    float4 pf[PF];
    auto fetch_block = [&](int r0) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int x = threadIdx.x + u * kThreads;
            const uint32_t off =
                (static_cast<uint32_t>(r0 + x / F4) * D + (x % F4) * 4) * sizeof(float);
            pf[u] = __builtin_bit_cast(float4, buf_load16(t_rsrc, off));
        }
    };
    if (keep_first < hi) fetch_block(keep_first);

    // 1. q_bar: computed here (mean over the r heads x chunk tokens) or read.
    WaveLds L{};
    if (active) {
        L = carve(wave_base + wave * wave_bytes, D, kGroups ? topk : 0,
                  kGroups && topk_groups > topk ? topk_groups : topk);
        if constexpr (kQbarIn) {
            for (int x = lane; x < D; x += 64) L.q[x] = qbar[unit * D + x];
            wave_sync_lds();
        } else {
            wave_query_mean<T, D>(q_rot, b, j, i, n_q_heads, r, n_q_chunks, L.q);
            wave_sync_lds();
            if (lane < D / 4) {
                const float4 v = *reinterpret_cast<const float4*>(L.q + lane * 4);
                *reinterpret_cast<float4*>(qbar + unit * D + lane * 4) = v;
            }
        }
    }

    // 2. score the middle chunks [keep_first, c - window) block by block.
    int n = c - window - keep_first;
    if (!active || n < 0) n = 0;
    for (int r0 = keep_first; r0 < hi; r0 += TB) {
        __syncthreads();                                 // the previous block is scored
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int x = threadIdx.x + u * kThreads;
            *reinterpret_cast<float4*>(s_tab + (x / F4) * TS + (x % F4) * 4) = pf[u];
        }
        __syncthreads();
        if (r0 + TB < hi) fetch_block(r0 + TB);
#pragma unroll
        for (int h = 0; h < TB / 64; ++h) {
            const int m = r0 - keep_first + h * 64 + lane;  // candidate ordinal of this lane
            if (m < n) {
                const float* row = s_tab + (h * 64 + lane) * TS;
                float a0 = 0.f, a1 = 0.f, a2 = 0.f, a3 = 0.f;
#pragma unroll
                for (int f = 0; f < F4; ++f) {
                    const float4 q = *reinterpret_cast<const float4*>(L.q + f * 4);
                    const float4 x = *reinterpret_cast<const float4*>(row + f * 4);
                    a0 = fmaf(q.x, x.x, a0);
                    a1 = fmaf(q.y, x.y, a1);
                    a2 = fmaf(q.z, x.z, a2);
                    a3 = fmaf(q.w, x.w, a3);
                }
                L.keys[m] = select_key((a0 + a1) + (a2 + a3), keep_first + m);
            }
        }
    }
    if (!active) return;
    wave_sync_lds();

    // 3. top-k chunks, ascending, -1 padded.
    const int k = n < topk ? n : topk;
    wave_select_topk(L.keys, n, k, L.sel, L.scr, true);  // ids keep_first + m
    wave_sync_lds();
    int32_t* out = chunk_idx + unit * topk;
    for (int t = lane; t < topk; t += 64) out[t] = t < k ? L.sel[t] : -1;
    if constexpr (!kGroups) return;

    // 4. group refinement of the chosen chunks.  When every candidate is
    // kept (K_g >= the candidates: the chunk-only variant, all groups of the
    // chosen chunks opened) the selection is the candidates in ascending
    // order, written without scoring.
    const int ng = k * gpc;
    int32_t* gout = group_idx + unit * topk_groups;
    if (ng <= topk_groups) {
        for (int t = lane; t < topk_groups; t += 64)
            gout[t] = t < ng ? L.sel[t >> gpc_shift] * gpc + (t & (gpc - 1)) : -1;
        return;
    }
    for (int t = lane; t < k; t += 64) L.list[t] = L.sel[t];
    wave_sync_lds();
    const float* gtab = group_sum + static_cast<int64_t>(bh) * table_chunks * gpc * D;
    score_candidates<D>(
        L.q, gtab, [&](int m) { return L.list[m >> gpc_shift] * gpc + (m & (gpc - 1)); }, ng,
        L.keys);
    wave_sync_lds();
    const int kg = topk_groups;
    wave_select_topk(L.keys, ng, kg, L.sel, L.scr, true);  // groups of ascending chunks
    wave_sync_lds();
    for (int t = lane; t < topk_groups; t += 64) gout[t] = L.sel[t];
}

template <int D>
__global__ __launch_bounds__(256) void route_groups_kernel(
    const float* __restrict__ qbar, const int32_t* __restrict__ chunk_idx, int q_chunk0,
    int n_q_chunks, const float* __restrict__ group_sum, int table_chunks,
    int32_t* __restrict__ group_idx, int n_units, int topk_chunks, int topk_groups, int gpc_shift,
    size_t wave_bytes) {
    const int gpc = 1 << gpc_shift;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int unit = blockIdx.x * (blockDim.x >> 6) + wave;
    if (unit >= n_units) return;
    WaveLds L = carve(smem_raw + wave * wave_bytes, D, topk_chunks, topk_groups);
    const int i = unit % n_q_chunks;
    const int bh = unit / n_q_chunks;
    const int c = q_chunk0 + i;
    const int limit = c < table_chunks ? c : table_chunks;

    for (int x = lane; x < D; x += 64) L.q[x] = qbar[static_cast<int64_t>(unit) * D + x];
    // valid chunk ids in order (a wave-wide compaction by ballot)
    const int32_t* row = chunk_idx + static_cast<int64_t>(unit) * topk_chunks;
    int nv = 0;
    for (int t0 = 0; t0 < topk_chunks; t0 += 64) {
        const int t = t0 + lane;
        const int cc = t < topk_chunks ? row[t] : -1;
        const bool ok = cc >= 0 && cc < limit;
        const uint64_t mask = __ballot(ok);
        const int pos = nv + __popcll(mask & ((uint64_t(1) << lane) - 1));
        if (ok) L.list[pos] = cc;
        nv += __popcll(mask);
    }
    wave_sync_lds();

    const int n = nv * gpc;
    int32_t* out = group_idx + static_cast<int64_t>(unit) * topk_groups;
    if (n <= topk_groups) {  // every candidate kept: ascending, no scores needed
        for (int t = lane; t < topk_groups; t += 64)
            out[t] = t < n ? L.list[t >> gpc_shift] * gpc + (t & (gpc - 1)) : -1;
        return;
    }
    const float* table = group_sum + static_cast<int64_t>(bh) * table_chunks * gpc * D;
    score_candidates<D>(
        L.q, table, [&](int m) { return L.list[m >> gpc_shift] * gpc + (m & (gpc - 1)); }, n,
        L.keys);
    wave_sync_lds();
    wave_select_topk(L.keys, n, topk_groups, L.sel, L.scr);
    wave_sync_lds();
    for (int t = lane; t < topk_groups; t += 64) out[t] = L.sel[t];
}

// Top-k by a whole workgroup of kThreads threads, for keys whose ids ascend
// with their position: writes the k ids with the largest keys to sel[0 .. k)
// in ascending order (0 < k <= n <= kMaxPer * kThreads); sel is complete
// when it returns.  Every thread must call it.  Short lists (n <= 256) go to
// wave 0's wave_select_topk.  Otherwise thread t holds keys t, t + kThreads,
// ... in registers and:
// 1. a lower bound L on the k-th largest score word is found, in one of two
//    forms.  For k <= kTopW * (waves): each wave hands over its
//    ceil(k / waves) largest words (one key removed per round) and wave 0
//    takes the k-th largest of those words, each of a different key.  For
//    larger k: each wave finds its own k-th largest word (bisection on ballot
//    counts; 0 if it holds fewer than k keys) and L is the largest of them.
//    Either way at least k keys have a word >= L, so every key of the top k
//    does;
// 2. the keys with word >= L (usually a few times k) are compacted in
//    position order, which keeps ids ascending;
// 3. wave 0 selects the top k of those with wave_select_topk.
// The result is the exact top k with wave_select_topk's tie rule.
template <int kThreads>
struct WgSelect {
    static constexpr int kMaxPer = 4;
    static constexpr int kTopW = 4;  // largest words each wave contributes to the bound
    uint32_t wave_t[kThreads / 64];
    int wave_cnt[kMaxPer][kThreads / 64];
    uint32_t cand[kTopW * (kThreads / 64)];
    uint32_t bound;
    int offset[kMaxPer * (kThreads / 64)];  // survivors before (pass, wave), position order
    int n_keep;
    uint64_t surv[kMaxPer * kThreads];
};

template <int kThreads>
__device__ __forceinline__ void wg_select_topk(uint64_t* keys, int n, int k, int* sel, int* scr,
                                               WgSelect<kThreads>* S) {
    constexpr int NW = kThreads / 64;
    constexpr int kMaxPer = WgSelect<kThreads>::kMaxPer;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    if (n <= 256) {
        if (wave == 0) wave_select_topk(keys, n, k, sel, scr, true);
        __syncthreads();
        return;
    }
    const int per = (n + kThreads - 1) / kThreads;  // keys per thread, 1 .. kMaxPer
    uint64_t key[kMaxPer];
    uint32_t hi[kMaxPer];
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
        const int x = tid + i * kThreads;
        key[i] = i < per && x < n ? keys[x] : 0;
        hi[i] = static_cast<uint32_t>(key[i] >> 32);  // 0 for no key: never >= a candidate
    }
    // A lower bound on the k-th largest score word.  With k <= kTopW * NW:
    // each wave hands over its `rounds` largest words (one key removed per
    // round), and the k-th largest of those rounds * NW words, each of a
    // different key, is found by wave 0.  Otherwise: the largest per-wave
    // k-th largest word.  Either way at least k keys reach the bound, so the
    // exact selection below sees every key of the result.
    constexpr int kTopW = WgSelect<kThreads>::kTopW;
    uint32_t bound = 0;
    if (k <= kTopW * NW) {
        // rounds: enough words for k candidates (one per key)
        const int rounds = (k + NW - 1) / NW;
        uint32_t used = 0;  // this thread's keys already handed over
#pragma unroll
        for (int rr = 0; rr < kTopW; ++rr) {
            if (rr >= rounds) break;
            uint32_t my = 0;
            int mi = -1;
#pragma unroll
            for (int i = 0; i < kMaxPer; ++i)
                if (i < per && !((used >> i) & 1u) && (mi < 0 || hi[i] > my)) {
                    my = hi[i];
                    mi = i;
                }
            const uint32_t m = wave_max_u32(my);
            const uint64_t holders = __ballot(mi >= 0 && my == m);
            if (lane == static_cast<int>(__builtin_ctzll(holders))) used |= 1u << mi;
            if (lane == 0) S->cand[rr * NW + wave] = m;
        }
        __syncthreads();
        if (wave == 0) {
            const uint32_t v = lane < rounds * NW ? S->cand[lane] : 0u;
            uint32_t t = 0;
            for (int bit = 31; bit >= 0; --bit) {
                const uint32_t c = t | (1u << bit);
                if (__popcll(__ballot(lane < rounds * NW && v >= c)) >= k) t = c;
            }
            if (lane == 0) S->bound = t;
        }
        __syncthreads();
        bound = S->bound;
    } else {
        uint32_t t_w = 0;
        for (int bit = 31; bit >= 0; --bit) {
            const uint32_t cand = t_w | (1u << bit);
            int cnt = 0;
#pragma unroll
            for (int i = 0; i < kMaxPer; ++i)
                if (i < per) cnt += __popcll(__ballot(hi[i] >= cand));
            if (cnt >= k) t_w = cand;
        }
        if (lane == 0) S->wave_t[wave] = t_w;
        __syncthreads();
#pragma unroll
        for (int w = 0; w < NW; ++w) bound = S->wave_t[w] > bound ? S->wave_t[w] : bound;
    }
    // word 0 marks an absent key (a score's word is never 0: that pattern
    // is a NaN), so it never passes, whatever the bound
    uint64_t km[kMaxPer];
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
        km[i] = i < per ? __ballot(hi[i] != 0 && hi[i] >= bound) : 0;
        if (lane == 0 && i < per) S->wave_cnt[i][wave] = __popcll(km[i]);
    }
    __syncthreads();
    // position order: pass i, then wave, then lane.  Wave 0 scans the
    // per * NW counts (one per lane) into exclusive offsets.
    static_assert(kMaxPer * NW <= 64, "one lane per (pass, wave)");
    if (wave == 0) {
        const int c0 = lane < per * NW ? S->wave_cnt[lane / NW][lane % NW] : 0;
        const int v = wave_incl_scan_add(c0);
        if (lane < per * NW) S->offset[lane] = v - c0;
        if (lane == 63) S->n_keep = v;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kMaxPer; ++i) {
        if (i >= per) break;
        if (hi[i] != 0 && hi[i] >= bound)
            S->surv[S->offset[i * NW + wave] + __popcll(km[i] & ((uint64_t(1) << lane) - 1))] = key[i];
    }
    __syncthreads();
    if (wave == 0) wave_select_topk(S->surv, S->n_keep, k, sel, scr, true);
    __syncthreads();
}

// q_bar from the chunk's r*64 query rows staged in LDS (row-major, D
// elements of T per row; rows a multiple of 64), by the first NRS * D
// threads of the workgroup:
// thread (rs, d) adds element d of rows rs, rs + NRS, ... in ascending order,
// the chain one lane of wave_mean_rows keeps for that element, then thread d
// adds the NRS partial sums in the same pairwise tree as its butterfly.  So
// the result is bit-identical to wave_mean_rows<T, D> over the same rows.
// `part` is LDS scratch of NRS * D floats; every thread must call it.
template <typename T, int D>
__device__ __forceinline__ void wg_mean_rows(const T* rows_lds, int rows, float* part, float* out) {
    constexpr int VPR = D / elem<T>::kVec;
    constexpr int NRS = 64 / VPR;
    constexpr int kU = 8;
    static_assert(64 % (NRS * kU) == 0, "rows (a multiple of 64) split evenly");
    const int tid = threadIdx.x;
    if (tid < NRS * D) {
        const int rs = tid / D, d = tid % D;
        float acc = 0.f;
        for (int row0 = rs; row0 < rows; row0 += NRS * kU) {
            float f[kU];
#pragma unroll
            for (int u = 0; u < kU; ++u) f[u] = elem<T>::to_f32(rows_lds[(row0 + u * NRS) * D + d]);
#pragma unroll
            for (int u = 0; u < kU; ++u) acc += f[u];
        }
        part[rs * D + d] = acc;
    }
    __syncthreads();
    if (tid < D) {
        float v[NRS];
#pragma unroll
        for (int x = 0; x < NRS; ++x) v[x] = part[x * D + tid];
#pragma unroll
        for (int step = 1; step < NRS; step <<= 1)
#pragma unroll
            for (int x = 0; x < NRS; x += 2 * step) v[x] = v[x] + v[x + step];
        out[tid] = v[0] * (1.0f / static_cast<float>(rows));
    }
}

// Launches with at most this many units route each unit with a whole
// workgroup (route_wide_kernel, for up to kWideMaxCandidates middle chunks:
// four keys per thread in its selection); larger ones pack four units per
// workgroup (route_kernel, up to kPackedMaxCandidates: sixteen keys per
// lane).  Longer candidate lists take route_long_kernel.
constexpr int kWideMaxUnits = 128;
constexpr int kWideMaxCandidates = WgSelect<1024>::kMaxPer * 1024;
constexpr int kPackedMaxCandidates = 1024;

// Steps 3 and 4 of the whole-workgroup routing, shared by route_wide_kernel
// and route_spread_kernel: the top K_c of the n chunk keys in L.keys (ids
// keep_first + m) to chunk_idx, then, with kGroups, the group refinement of
// the chosen chunks against L.q.  Every thread of the workgroup calls.
template <int D, bool kGroups>
__device__ __forceinline__ void wide_select_refine(const WaveLds& L, unsigned char* big, int n,
                                                   int unit, int bh,
                                                   const float* __restrict__ group_sum,
                                                   int table_chunks, int32_t* __restrict__ chunk_idx,
                                                   int32_t* __restrict__ group_idx, int topk,
                                                   int topk_groups, int gpc_shift) {
    constexpr int kThreads = 1024;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int gpc = 1 << gpc_shift;
    // 3. top-k chunks, ascending, -1 padded (the select's histograms reuse
    // the table region)
    auto* S = reinterpret_cast<WgSelect<kThreads>*>(big);
    const int k = n < topk ? n : topk;
    int32_t* out = chunk_idx + static_cast<int64_t>(unit) * topk;
    if (k > 0) wg_select_topk<kThreads>(L.keys, n, k, L.sel, L.scr, S);  // ids keep_first + m
    if (wave == 0) {
        for (int t = lane; t < topk; t += 64) out[t] = t < k ? L.sel[t] : -1;
        if constexpr (kGroups)
            for (int t = lane; t < k; t += 64) L.list[t] = L.sel[t];
    }
    if constexpr (!kGroups) return;

    // 4. group refinement (the chunk-only variant keeps every candidate:
    // ascending, written without scoring)
    const int ng = k * gpc;
    int32_t* gout = group_idx + static_cast<int64_t>(unit) * topk_groups;
    if (ng <= topk_groups) {
        if (wave == 0)
            for (int t = lane; t < topk_groups; t += 64)
                gout[t] = t < ng ? L.sel[t >> gpc_shift] * gpc + (t & (gpc - 1)) : -1;
        return;
    }
    __syncthreads();  // the chunk list is visible to every wave
    const float* gtab = group_sum + static_cast<int64_t>(bh) * table_chunks * gpc * D;
    for (int m0 = wave * 16; m0 < ng; m0 += 16 * (kThreads / 64)) {
        const int rem = ng - m0;
        batch_keys<D, 1>(
            L.q, gtab,
            [&](int kk) {
                const int m = m0 + (kk < rem ? kk : rem - 1);
                return L.list[m >> gpc_shift] * gpc + (m & (gpc - 1));
            },
            rem, L.keys + m0);
    }
    __syncthreads();
    wg_select_topk<kThreads>(L.keys, ng, topk_groups, L.sel, L.scr, S);  // groups of ascending chunks
    if (wave == 0)
        for (int t = lane; t < topk_groups; t += 64) gout[t] = L.sel[t];
}

// Routing of one unit by a whole workgroup of 16 wavefronts, for launches
// with too few units to fill the chip (a decode block, a block-sequential
// prefill step).  The outputs are bit-identical to route_kernel's: every
// score has the same arithmetic, only the work is spread wider.
// * q_bar: the chunk's r*64 query rows are staged in LDS by all threads at
//   once (one round trip instead of one per 16 rows), then wave 0 reduces
//   them with the shared fixed-order code.  The first table block is
//   requested before that, so it arrives while q_bar is formed.
// * chunk scores: the table goes through LDS in blocks of kWideRows rows
//   (coalesced 16-byte loads, the next block in registers while the current
//   one is scored).  Four lanes score one row: lane qd sums the dimensions
//   d = qd mod 4 in order, and the quad adds the four partial sums pairwise,
//   ((s0 + s1) + (s2 + s3)), the same operations as one lane doing all four.
//   Wave 0 selects the top K_c.
// * group scores: wave w scores candidates 16w .. 16w + 15 (+ 256 per
//   pass) with batch_keys, whose per-candidate arithmetic does not depend on
//   the batch; wave 0 selects the top K_g.
// LDS: the WaveLds pieces (keys for the larger candidate list), then one
// region at big_off that holds the staged query rows and then table blocks.
constexpr int kWideRows = 256;

template <typename T, int D, bool kGroups, bool kQbarIn>
__global__ __launch_bounds__(1024) void route_wide_kernel(
    const T* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const float* __restrict__ chunk_sum,
    const float* __restrict__ group_sum, int table_chunks, float* __restrict__ qbar,
    int32_t* __restrict__ chunk_idx, int32_t* __restrict__ group_idx, int n_q_heads, int n_kv,
    int keep_first, int window, int topk, int topk_groups, int gpc_shift, int big_off) {
    constexpr int kThreads = 1024;
    constexpr int F4 = D / 4;                     // float4 per table row
    constexpr int TS = D + 4;                     // padded LDS row stride (floats)
    constexpr int PF = kWideRows * F4 / kThreads; // float4 per thread per table block
    constexpr int VPR = D / elem<T>::kVec;        // 16-byte vectors per query row
    constexpr int QU = 8;                         // query-row loads in flight per thread
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int unit = blockIdx.x;
    const int bh = unit / n_q_chunks, i = unit % n_q_chunks;
    const int b = bh / n_kv, j = bh % n_kv, r = n_q_heads / n_kv;
    const int c = q_chunk0 + i;
    const int gpc = 1 << gpc_shift;
    WaveLds L = carve(smem_raw, D, kGroups ? topk : 0,
                      kGroups && topk_groups > topk ? topk_groups : topk);
    unsigned char* big = smem_raw + big_off;

    // the middle chunks [keep_first, keep_first + n); loads past them read zeros
    int n = c - window - keep_first;
    if (n < 0) n = 0;
    const float* table = chunk_sum + (static_cast<int64_t>(bh) * table_chunks + keep_first) * D;
    const buf_rsrc t_rsrc = make_rsrc(table, static_cast<uint32_t>(n) * D * sizeof(float));
    float4 pf[PF];
    auto fetch_block = [&](int r0) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int x = tid + u * kThreads;
            const uint32_t off =
                (static_cast<uint32_t>(r0 + x / F4) * D + (x % F4) * 4) * sizeof(float);
            pf[u] = __builtin_bit_cast(float4, buf_load16(t_rsrc, off));
        }
    };
    if (n > 0) fetch_block(0);

    // 1. q_bar
    if constexpr (kQbarIn) {
        if (tid < D / 4)
            *reinterpret_cast<float4*>(L.q + tid * 4) =
                *reinterpret_cast<const float4*>(qbar + static_cast<int64_t>(unit) * D + tid * 4);
    } else {
        constexpr int V = elem<T>::kVec;
        const int64_t qtok = static_cast<int64_t>(n_q_chunks) * 64;
        const T* qbase = query_chunk_base<T, D>(q_rot, b, j, i, n_q_heads, r, n_q_chunks);
        // the r heads' 64-token slices, from the first row of head 0 to the
        // last row of head r - 1
        const buf_rsrc q_rsrc = make_rsrc(
            qbase, static_cast<uint32_t>(((r - 1) * qtok + 64) * D * sizeof(T)));
        vec16* s_rows = reinterpret_cast<vec16*>(big);
        const int n_vec = r * 64 * VPR;
        for (int x = tid; x < n_vec; x += kThreads * QU) {
            vec16 t[QU];
#pragma unroll
            for (int u = 0; u < QU; ++u) {
                const int y = x + u * kThreads;
                const int row = y / VPR, cv = y % VPR;
                t[u] = buf_load16(q_rsrc, static_cast<uint32_t>(
                                              (((row >> 6) * qtok + (row & 63)) * D + cv * V) *
                                              sizeof(T)));
            }
#pragma unroll
            for (int u = 0; u < QU; ++u)
                if (x + u * kThreads < n_vec) s_rows[x + u * kThreads] = t[u];
        }
        __syncthreads();
        // partial sums after the staged rows, inside the same region
        wg_mean_rows<T, D>(reinterpret_cast<const T*>(s_rows), r * 64,
                           reinterpret_cast<float*>(s_rows + n_vec), L.q);
        __syncthreads();
        if (tid < D / 4)
            *reinterpret_cast<float4*>(qbar + static_cast<int64_t>(unit) * D + tid * 4) =
                *reinterpret_cast<const float4*>(L.q + tid * 4);
    }
    __syncthreads();  // q_bar in LDS; the staged rows are dead

    // 2. chunk scores, a block of kWideRows table rows at a time
    float* s_tab = reinterpret_cast<float*>(big);
    const int qd = lane & 3;
    const int rl = wave * 16 + (lane >> 2);  // this quad's row within a block
    float qv[F4];
#pragma unroll
    for (int f = 0; f < F4; ++f) qv[f] = L.q[4 * f + qd];
    for (int r0 = 0; r0 < n; r0 += kWideRows) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int x = tid + u * kThreads;
            *reinterpret_cast<float4*>(s_tab + (x / F4) * TS + (x % F4) * 4) = pf[u];
        }
        __syncthreads();
        if (r0 + kWideRows < n) fetch_block(r0 + kWideRows);
#pragma unroll
        for (int h = 0; h < kWideRows / 256; ++h) {
            const float* row = s_tab + (h * 256 + rl) * TS + qd;
            float a = 0.f;
#pragma unroll
            for (int f = 0; f < F4; ++f) a = fmaf(qv[f], row[4 * f], a);
            a = add_quad<0xb1>(a);  // (s0 + s1), (s2 + s3)
            a = add_quad<0x4e>(a);  // (s0 + s1) + (s2 + s3)
            const int m = r0 + h * 256 + rl;
            if (qd == 0 && m < n) L.keys[m] = select_key(a, keep_first + m);
        }
        __syncthreads();  // the block is scored before the next one is stored
    }

    wide_select_refine<D, kGroups>(L, big, n, unit, bh, group_sum, table_chunks, chunk_idx,
                                   group_idx, topk, topk_groups, gpc_shift);
}

// Routing from a given q_bar for a launch of a few units (a decode block),
// each unit's table scan spread over `parts` workgroups: one workgroup reads
// the table at a single compute unit's bandwidth, which bounds
// route_wide_kernel there.  Workgroup (unit, p) scores middle chunks
// [p*kSpreadRows, (p+1)*kSpreadRows) with route_wide_kernel's arithmetic (the
// same keys, bit for bit) and writes their keys to the plan's routing
// workspace; the unit's last workgroup to finish -- the one whose increment
// of the unit's device-scope counter completes it -- reads every key back,
// resets the counter for the next call, and selects and refines exactly as
// route_wide_kernel does.  One thread per workgroup makes the increment, an
// acquire-release atomic at device scope: it publishes the workgroup's keys
// (ordered before it by the workgroup barrier) and, in the last workgroup,
// makes every other workgroup's keys visible.
constexpr int kSpreadRows = 128;
static_assert(kRouteSpreadCandidates <= kWideMaxCandidates, "the last workgroup's selection");

template <int D, bool kGroups>
__global__ __launch_bounds__(1024) void route_spread_kernel(
    const float* __restrict__ qbar, int q_chunk0, int n_q_chunks,
    const float* __restrict__ chunk_sum, const float* __restrict__ group_sum, int table_chunks,
    int32_t* __restrict__ chunk_idx, int32_t* __restrict__ group_idx,
    uint64_t* __restrict__ ws_keys, unsigned* __restrict__ ws_count, int n_kv, int keep_first,
    int window, int topk, int topk_groups, int gpc_shift, int parts, int big_off) {
    constexpr int kThreads = 1024;
    constexpr int F4 = D / 4;                        // float4 per table row
    constexpr int TS = D + 4;                        // padded LDS row stride (floats)
    constexpr int PF = kSpreadRows * F4 / kThreads;  // float4 per thread
    static_assert(PF >= 1 && PF * kThreads == kSpreadRows * F4, "block split");
    extern __shared__ __align__(16) unsigned char smem_raw[];
    __shared__ int s_last;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int unit = blockIdx.x / parts, part = blockIdx.x % parts;
    const int bh = unit / n_q_chunks, i = unit % n_q_chunks;
    const int c = q_chunk0 + i;
    WaveLds L = carve(smem_raw, D, kGroups ? topk : 0,
                      kGroups && topk_groups > topk ? topk_groups : topk);
    unsigned char* big = smem_raw + big_off;

    int n = c - window - keep_first;
    if (n < 0) n = 0;
    const float* table = chunk_sum + (static_cast<int64_t>(bh) * table_chunks + keep_first) * D;
    const buf_rsrc t_rsrc = make_rsrc(table, static_cast<uint32_t>(n) * D * sizeof(float));
    const int r0 = part * kSpreadRows;
    float4 qin = make_float4(0.f, 0.f, 0.f, 0.f);
    if (tid < D / 4)
        qin = *reinterpret_cast<const float4*>(qbar + static_cast<int64_t>(unit) * D + tid * 4);
    float4 pf[PF];
#pragma unroll
    for (int u = 0; u < PF; ++u) {
        const int x = tid + u * kThreads;
        const uint32_t off = (static_cast<uint32_t>(r0 + x / F4) * D + (x % F4) * 4) * sizeof(float);
        pf[u] = __builtin_bit_cast(float4, buf_load16(t_rsrc, off));  // zeros past row n
    }
    if (tid < D / 4) *reinterpret_cast<float4*>(L.q + tid * 4) = qin;
    float* s_tab = reinterpret_cast<float*>(big);
#pragma unroll
    for (int u = 0; u < PF; ++u) {
        const int x = tid + u * kThreads;
        *reinterpret_cast<float4*>(s_tab + (x / F4) * TS + (x % F4) * 4) = pf[u];
    }
    __syncthreads();
    // scores of the block's rows: quad rl scores row rl (route_wide_kernel's
    // per-row arithmetic), keys to the workspace
    const int qd = lane & 3;
    const int rl = wave * 16 + (lane >> 2);
    uint64_t* keys = ws_keys + static_cast<int64_t>(unit) * kRouteSpreadCandidates;
    if (rl < kSpreadRows) {
        const float* row = s_tab + rl * TS + qd;
        float a = 0.f;
#pragma unroll
        for (int f = 0; f < F4; ++f) a = fmaf(L.q[4 * f + qd], row[4 * f], a);
        a = add_quad<0xb1>(a);  // (s0 + s1), (s2 + s3)
        a = add_quad<0x4e>(a);  // (s0 + s1) + (s2 + s3)
        const int m = r0 + rl;
        if (qd == 0 && m < n) keys[m] = select_key(a, keep_first + m);
    }
    // The workgroup's keys happen before thread 0's increment (the barrier),
    // which releases them at device scope; the increment that completes the
    // count acquires every other workgroup's.
    __syncthreads();
    if (tid == 0)
        s_last = __hip_atomic_fetch_add(ws_count + unit, 1u, __ATOMIC_ACQ_REL,
                                        __HIP_MEMORY_SCOPE_AGENT) ==
                 static_cast<unsigned>(parts - 1);
    __syncthreads();
    if (!s_last) return;
    for (int m = tid; m < n; m += kThreads) L.keys[m] = keys[m];
    if (tid == 0) ws_count[unit] = 0u;  // every workgroup of the unit has counted
    __syncthreads();
    wide_select_refine<D, kGroups>(L, big, n, unit, bh, group_sum, table_chunks, chunk_idx,
                                   group_idx, topk, topk_groups, gpc_shift);
}

// Routing of units with more middle chunks than the other kernels hold as
// key lists (long contexts: the exhaustive scan of the summary table the
// paper names as its limit, Sec. 3.6 and Sec. 7), one workgroup of
// kLongThreads per unit.  The table streams through LDS in blocks of
// kLongRows rows (the next block in registers while the current one is
// scored); a quad scores a row with the arithmetic of the other kernels
// (lane qd sums the dimensions d = qd mod 4 in order, the quad adds the four
// sums pairwise), so every score, and hence every key, is bit-identical to
// theirs.  Only keys above the running cut are kept, in an LDS buffer of
// kLongCap keys; when it cannot take another block, an exact selection
// (long_select) reduces it to its k largest keys and the k-th becomes the
// cut.  Keys are unique (score word, then the complemented id), so selecting
// by key value is the lowest-index tie rule.  The group stage scores its
// candidates with batch_keys into the same buffer and selects the same way.
constexpr int kLongThreads = 512;
constexpr int kLongRows = kLongThreads / 4;   // one table row per quad
constexpr int kLongCap = 4096;                // >= every group list (K_c * chunk/group)
constexpr int kLongPer = kLongCap / kLongThreads;
static_assert(kLongCap >= kMaxTopK + kLongRows, "a reduced buffer takes a further block");

struct LongCtl {
    uint64_t cut;                           // keys above it are kept
    int n;                                  // keys in the buffer
    int cnt[2][kLongThreads / 64];          // per-wave counts of a bisection step
};

// The k largest of the n keys of buf (0 < k <= n <= kLongCap), left in
// buf[0 .. k) in no particular order; returns the k-th largest key.  The
// k-th largest key T is found bit by bit from the top (T grows by a bit
// while at least k keys are >= it: one count per step, summed over the
// waves through LDS), then the keys >= T, exactly k of them, are compacted.
// Every thread must call it; the buffer is complete when it returns.
__device__ uint64_t long_select(uint64_t* buf, int n, int k, LongCtl* ctl) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    constexpr int NW = kLongThreads / 64;
    uint64_t key[kLongPer];
#pragma unroll
    for (int i = 0; i < kLongPer; ++i) {
        const int x = tid + i * kLongThreads;
        key[i] = x < n ? buf[x] : 0;  // 0 is below every key
    }
    uint64_t T = 0;
    for (int bit = 63; bit >= 0; --bit) {
        const uint64_t c = T | (uint64_t(1) << bit);
        int cnt = 0;
#pragma unroll
        for (int i = 0; i < kLongPer; ++i) cnt += __popcll(__ballot(key[i] >= c));
        const int par = bit & 1;
        if (lane == 0) ctl->cnt[par][wave] = cnt;
        __syncthreads();
        int tot = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) tot += ctl->cnt[par][w];
        if (tot >= k) T = c;
    }
    // every thread holds its keys; the buffer is rewritten from the start
    if (tid == 0) ctl->n = 0;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kLongPer; ++i) {
        const bool keep = key[i] >= T && key[i] != 0;
        const uint64_t m = __ballot(keep);
        int base = 0;
        if (lane == 0 && m) base = atomicAdd(&ctl->n, __popcll(m));
        base = __shfl(base, 0);
        if (keep) buf[base + __popcll(m & ((uint64_t(1) << lane) - 1))] = key[i];
    }
    __syncthreads();
    return T;
}

// The ids of buf[0 .. k) (k <= kLongThreads), ascending, to sel.
__device__ __forceinline__ void long_sorted_ids(const uint64_t* buf, int k, int* sel) {
    const int tid = threadIdx.x;
    if (tid < k) {
        const int id = key_index(buf[tid]);
        int rank = 0;
        for (int t = 0; t < k; ++t) rank += key_index(buf[t]) < id;
        sel[rank] = id;
    }
    __syncthreads();
}

template <typename T, int D, bool kGroups, bool kQbarIn>
__global__ __launch_bounds__(kLongThreads) void route_long_kernel(
    const T* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const float* __restrict__ chunk_sum,
    const float* __restrict__ group_sum, int table_chunks, float* __restrict__ qbar,
    int32_t* __restrict__ chunk_idx, int32_t* __restrict__ group_idx, int n_q_heads, int n_kv,
    int keep_first, int window, int topk, int topk_groups, int gpc_shift) {
    constexpr int F4 = D / 4;                       // float4 per table row
    constexpr int TS = D + 4;                       // padded LDS row stride (floats)
    constexpr int PF = kLongRows * F4 / kLongThreads;  // float4 per thread per block
    __shared__ __align__(16) float s_q[D];
    __shared__ __align__(16) float s_tab[kLongRows * TS];
    __shared__ uint64_t s_buf[kLongCap];
    __shared__ int s_sel[kMaxTopK];
    __shared__ int s_list[kMaxTopK];
    __shared__ LongCtl ctl;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int unit = blockIdx.x;
    const int bh = unit / n_q_chunks, i = unit % n_q_chunks;
    const int b = bh / n_kv, j = bh % n_kv, r = n_q_heads / n_kv;
    const int c = q_chunk0 + i;
    const int gpc = 1 << gpc_shift;

    int n = c - window - keep_first;  // middle chunks [keep_first, keep_first + n)
    if (n < 0) n = 0;
    const float* table = chunk_sum + (static_cast<int64_t>(bh) * table_chunks + keep_first) * D;
    const buf_rsrc t_rsrc = make_rsrc(table, static_cast<uint32_t>(n) * D * sizeof(float));
    float4 pf[PF];
    auto fetch_block = [&](int r0) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int x = tid + u * kLongThreads;
            const uint32_t off =
                (static_cast<uint32_t>(r0 + x / F4) * D + (x % F4) * 4) * sizeof(float);
            pf[u] = __builtin_bit_cast(float4, buf_load16(t_rsrc, off));
        }
    };
    if (n > 0) fetch_block(0);

    // 1. q_bar (wave 0 forms it with the packed kernel's code, or reads it)
    if (tid == 0) {
        ctl.cut = 0;
        ctl.n = 0;
    }
    if constexpr (kQbarIn) {
        if (tid < D / 4)
            *reinterpret_cast<float4*>(s_q + tid * 4) =
                *reinterpret_cast<const float4*>(qbar + static_cast<int64_t>(unit) * D + tid * 4);
    } else {
        if (wave == 0) {
            wave_query_mean<T, D>(q_rot, b, j, i, n_q_heads, r, n_q_chunks, s_q);
            wave_sync_lds();
            if (lane < D / 4)
                *reinterpret_cast<float4*>(qbar + static_cast<int64_t>(unit) * D + lane * 4) =
                    *reinterpret_cast<const float4*>(s_q + lane * 4);
        }
    }
    __syncthreads();

    // 2. chunk scores, a block of kLongRows rows at a time; keys above the
    // cut are appended to the buffer, which is reduced to the top k whenever
    // it could not take another block
    const int k = n < topk ? n : topk;
    const int qd = lane & 3;
    const int rl = tid >> 2;  // this quad's row within a block
    float qv[F4];
#pragma unroll
    for (int f = 0; f < F4; ++f) qv[f] = s_q[4 * f + qd];
    for (int r0 = 0; r0 < n; r0 += kLongRows) {
#pragma unroll
        for (int u = 0; u < PF; ++u) {
            const int x = tid + u * kLongThreads;
            *reinterpret_cast<float4*>(s_tab + (x / F4) * TS + (x % F4) * 4) = pf[u];
        }
        __syncthreads();
        if (r0 + kLongRows < n) fetch_block(r0 + kLongRows);
        const float* row = s_tab + rl * TS + qd;
        float a = 0.f;
#pragma unroll
        for (int f = 0; f < F4; ++f) a = fmaf(qv[f], row[4 * f], a);
        a = add_quad<0xb1>(a);  // (s0 + s1), (s2 + s3)
        a = add_quad<0x4e>(a);  // (s0 + s1) + (s2 + s3)
        const int m = r0 + rl;
        const uint64_t key = select_key(a, keep_first + m);
        const bool keep = qd == 0 && m < n && key > ctl.cut;
        const uint64_t mm = __ballot(keep);
        int base = 0;
        if (lane == 0 && mm) base = atomicAdd(&ctl.n, __popcll(mm));
        base = __shfl(base, 0);
        if (keep) s_buf[base + __popcll(mm & ((uint64_t(1) << lane) - 1))] = key;
        __syncthreads();  // the block is scored and appended
        const int nb = ctl.n;
        if (nb > kLongCap - kLongRows) {
            const uint64_t cut = long_select(s_buf, nb, k, &ctl);
            if (tid == 0) ctl.cut = cut;
            __syncthreads();
        }
    }

    // 3. top-k chunks, ascending, -1 padded
    int32_t* out = chunk_idx + static_cast<int64_t>(unit) * topk;
    if (k > 0) {
        const int nb = ctl.n;
        if (nb > k) long_select(s_buf, nb, k, &ctl);
        long_sorted_ids(s_buf, k, s_sel);
    }
    for (int t = tid; t < topk; t += kLongThreads) out[t] = t < k ? s_sel[t] : -1;
    if constexpr (!kGroups) return;

    // 4. group refinement of the chosen chunks (every candidate kept when
    // the budget covers them: ascending, written without scoring)
    const int ng = k * gpc;
    int32_t* gout = group_idx + static_cast<int64_t>(unit) * topk_groups;
    if (ng <= topk_groups) {
        for (int t = tid; t < topk_groups; t += kLongThreads)
            gout[t] = t < ng ? s_sel[t >> gpc_shift] * gpc + (t & (gpc - 1)) : -1;
        return;
    }
    for (int t = tid; t < k; t += kLongThreads) s_list[t] = s_sel[t];
    __syncthreads();
    const float* gtab = group_sum + static_cast<int64_t>(bh) * table_chunks * gpc * D;
    for (int m0 = wave * 16; m0 < ng; m0 += 16 * (kLongThreads / 64)) {
        const int rem = ng - m0;
        batch_keys<D, 1>(
            s_q, gtab,
            [&](int kk) {
                const int m = m0 + (kk < rem ? kk : rem - 1);
                return s_list[m >> gpc_shift] * gpc + (m & (gpc - 1));
            },
            rem, s_buf + m0);
    }
    __syncthreads();
    long_select(s_buf, ng, topk_groups, &ctl);
    long_sorted_ids(s_buf, topk_groups, s_sel);
    for (int t = tid; t < topk_groups; t += kLongThreads) gout[t] = s_sel[t];
}

// Up to four waves per workgroup, as many as the LDS budget allows.
int waves_per_block(size_t wave_bytes, int max_lds) {
    int w = static_cast<int>(static_cast<size_t>(max_lds) / wave_bytes);
    return w < 1 ? 1 : (w > 4 ? 4 : w);
}

// LDS of the fused routing block: the staged table block plus one region per
// wavefront (q_bar, chunk list, selection, keys for the larger of the two
// candidate lists).
struct RouteGeom {
    size_t wave_bytes;
    size_t total;
    int units_per_block;
};

inline RouteGeom route_geom(const hga_plan& plan, int n_max, bool groups) {
    const hga_params& p = plan.p;
    const int gpc = p.chunk / p.group;
    const int nk = groups && p.topk_chunks * gpc > n_max ? p.topk_chunks * gpc : n_max;
    const int ntop = groups && p.topk_groups > p.topk_chunks ? p.topk_groups : p.topk_chunks;
    RouteGeom g;
    g.wave_bytes = wave_lds_bytes(p.head_dim, groups ? p.topk_chunks : 0, ntop, nk);
    const size_t tab = align16(sizeof(float) * table_rows(p.head_dim) * (p.head_dim + 4));
    g.units_per_block = 4;
    while (g.units_per_block > 1 &&
           tab + g.units_per_block * g.wave_bytes > static_cast<size_t>(plan.max_lds))
        g.units_per_block >>= 1;
    g.total = tab + g.units_per_block * g.wave_bytes;
    return g;
}


// LDS of route_wide_kernel: the WaveLds pieces (keys for the larger
// candidate list), then one region (at the returned offset) for the staged
// query rows of the chunk and then the table blocks.
struct WideGeom {
    size_t big_off;
    size_t total;
};

inline WideGeom route_wide_geom(const hga_plan& plan, int n_max, bool groups, bool qbar_in) {
    const hga_params& p = plan.p;
    const int gpc = p.chunk / p.group;
    const int nk = groups && p.topk_chunks * gpc > n_max ? p.topk_chunks * gpc : n_max;
    const int ntop = groups && p.topk_groups > p.topk_chunks ? p.topk_groups : p.topk_chunks;
    const size_t elem_bytes = p.dtype == HGA_F32 ? 4 : 2;
    const size_t rows = qbar_in ? 0
                                : static_cast<size_t>(p.n_q_heads / p.n_kv_heads) * p.chunk *
                                      p.head_dim * elem_bytes;
    const size_t part = qbar_in ? 0 : sizeof(float) * 8 * p.head_dim;  // wg_mean_rows partials
    const size_t tab = sizeof(float) * kWideRows * (p.head_dim + 4);
    size_t big = rows + part > tab ? rows + part : tab;
    if (big < sizeof(WgSelect<1024>)) big = sizeof(WgSelect<1024>);  // the selection, after scoring
    WideGeom g;
    g.big_off = wave_lds_bytes(p.head_dim, groups ? p.topk_chunks : 0, ntop, nk);
    g.total = g.big_off + align16(big);
    return g;
}

template <typename T, int D, bool kGroups, bool kQbarIn>
hipError_t launch_route_t(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                          const float* chunk_sum, const float* group_sum, int table_chunks,
                          float* qbar, int32_t* chunk_idx, int32_t* group_idx, hipStream_t stream) {
    const hga_params& p = plan.p;
    const int n_max = middle_count(p, q_chunk0 + n_q_chunks - 1);
    const int units = p.batch * p.n_kv_heads * n_q_chunks;
    const int gpc = p.chunk / p.group;
    const int gpc_shift = gpc == 8 ? 3 : (gpc == 4 ? 2 : 1);
    // a few units with long tables: the scan spread over several workgroups
    // per unit (q_bar given; the keys in the plan's workspace)
    if (kQbarIn && units <= kRouteSpreadUnits && n_max >= 2 * kSpreadRows &&
        n_max <= kRouteSpreadCandidates && plan.route_keys) {
        const WideGeom wg = route_wide_geom(plan, n_max, kGroups, true);
        const size_t tab = sizeof(float) * kSpreadRows * (D + 4);
        const size_t total = wg.big_off + (tab > wg.total - wg.big_off ? tab : wg.total - wg.big_off);
        if (total + 64 <= static_cast<size_t>(plan.max_lds)) {  // + the static flag
            const int parts = (n_max + kSpreadRows - 1) / kSpreadRows;
            hipLaunchKernelGGL((route_spread_kernel<D, kGroups>), dim3(units * parts), dim3(1024),
                               total, stream, qbar, q_chunk0, n_q_chunks, chunk_sum, group_sum,
                               table_chunks, chunk_idx, group_idx, plan.route_keys,
                               plan.route_count, p.n_kv_heads, p.keep_first, recent_window(p),
                               p.topk_chunks, p.topk_groups, gpc_shift, parts,
                               static_cast<int>(wg.big_off));
            return hipGetLastError();
        }
    }
    if (units <= kWideMaxUnits && n_max <= kWideMaxCandidates) {
        const WideGeom wg = route_wide_geom(plan, n_max, kGroups, kQbarIn);
        if (wg.total <= static_cast<size_t>(plan.max_lds)) {
            hipLaunchKernelGGL((route_wide_kernel<T, D, kGroups, kQbarIn>), dim3(units),
                               dim3(1024), wg.total, stream, static_cast<const T*>(q_rot),
                               q_chunk0, n_q_chunks, chunk_sum, group_sum, table_chunks, qbar,
                               chunk_idx, group_idx, p.n_q_heads, p.n_kv_heads, p.keep_first,
                               recent_window(p), p.topk_chunks, p.topk_groups, gpc_shift,
                               static_cast<int>(wg.big_off));
            return hipGetLastError();
        }
    }
    if (n_max > kPackedMaxCandidates) {
        hipLaunchKernelGGL((route_long_kernel<T, D, kGroups, kQbarIn>), dim3(units),
                           dim3(kLongThreads), 0, stream, static_cast<const T*>(q_rot), q_chunk0,
                           n_q_chunks, chunk_sum, group_sum, table_chunks, qbar, chunk_idx,
                           group_idx, p.n_q_heads, p.n_kv_heads, p.keep_first, recent_window(p),
                           p.topk_chunks, p.topk_groups, gpc_shift);
        return hipGetLastError();
    }
    const RouteGeom g = route_geom(plan, n_max, kGroups);
    const int upb = g.units_per_block < n_q_chunks ? g.units_per_block : n_q_chunks;
    const int blocks = p.batch * p.n_kv_heads * ((n_q_chunks + upb - 1) / upb);
    hipLaunchKernelGGL((route_kernel<T, D, kGroups, kQbarIn>), dim3(blocks), dim3(256), g.total,
                       stream,
                       static_cast<const T*>(q_rot), q_chunk0, n_q_chunks, chunk_sum, group_sum,
                       table_chunks, qbar, chunk_idx, group_idx, p.n_q_heads, p.n_kv_heads,
                       p.keep_first, recent_window(p), p.topk_chunks, p.topk_groups, gpc_shift, upb,
                       g.wave_bytes);
    return hipGetLastError();
}

template <bool kGroups, bool kQbarIn>
hipError_t launch_route_any(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                            const float* chunk_sum, const float* group_sum, int table_chunks,
                            float* qbar, int32_t* chunk_idx, int32_t* group_idx,
                            hipStream_t stream) {
    const hga_params& p = plan.p;
    if (p.dtype == HGA_F32) {
        if (p.head_dim == 64)
            return launch_route_t<float, 64, kGroups, kQbarIn>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                                      group_sum, table_chunks, qbar, chunk_idx,
                                                      group_idx, stream);
        return launch_route_t<float, 128, kGroups, kQbarIn>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                                   group_sum, table_chunks, qbar, chunk_idx,
                                                   group_idx, stream);
    }
    if (p.head_dim == 64)
        return launch_route_t<bf16_t, 64, kGroups, kQbarIn>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                                   group_sum, table_chunks, qbar, chunk_idx,
                                                   group_idx, stream);
    return launch_route_t<bf16_t, 128, kGroups, kQbarIn>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                                group_sum, table_chunks, qbar, chunk_idx,
                                                group_idx, stream);
}

template <int D>
hipError_t launch_groups_t(const hga_plan& plan, const float* qbar, const int32_t* chunk_idx,
                           int q_chunk0, int n_q_chunks, const float* group_sum, int table_chunks,
                           int32_t* group_idx, hipStream_t stream) {
    const hga_params& p = plan.p;
    const int gpc = p.chunk / p.group;
    const size_t wb = wave_lds_bytes(D, p.topk_chunks, p.topk_groups, p.topk_chunks * gpc);
    const int wpb = waves_per_block(wb, plan.max_lds);
    const int n_units = p.batch * p.n_kv_heads * n_q_chunks;
    const int blocks = (n_units + wpb - 1) / wpb;
    hipLaunchKernelGGL((route_groups_kernel<D>), dim3(blocks), dim3(64 * wpb), wb * wpb, stream,
                       qbar, chunk_idx, q_chunk0, n_q_chunks, group_sum, table_chunks, group_idx,
                       n_units, p.topk_chunks, p.topk_groups, gpc == 8 ? 3 : (gpc == 4 ? 2 : 1), wb);
    return hipGetLastError();
}

}  // namespace

size_t route_lds_bytes(const hga_plan& plan, int n_max, bool groups) {
    // beyond the packed kernel's lists: route_long_kernel, whose LDS does not
    // depend on the candidate count
    if (n_max > kPackedMaxCandidates) {
        const int d = plan.p.head_dim;
        return sizeof(float) * d + sizeof(float) * kLongRows * (d + 4) +
               sizeof(uint64_t) * kLongCap + 2 * sizeof(int) * kMaxTopK + sizeof(LongCtl);
    }
    // otherwise the smallest packed configuration (one wavefront per block)
    // must fit
    const hga_params& p = plan.p;
    const int gpc = p.chunk / p.group;
    const int nk = groups && p.topk_chunks * gpc > n_max ? p.topk_chunks * gpc : n_max;
    const int ntop = groups && p.topk_groups > p.topk_chunks ? p.topk_groups : p.topk_chunks;
    return align16(sizeof(float) * table_rows(p.head_dim) * (p.head_dim + 4)) +
           wave_lds_bytes(p.head_dim, groups ? p.topk_chunks : 0, ntop, nk);
}

hipError_t launch_route_chunks(const hga_plan& plan, const void* q_rot, int q_chunk0,
                               int n_q_chunks, const float* chunk_sum, int table_chunks,
                               float* qbar, int32_t* chunk_idx, hipStream_t stream) {
    return launch_route_any<false, false>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum, nullptr,
                                          table_chunks, qbar, chunk_idx, nullptr, stream);
}

hipError_t launch_route(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                        const float* chunk_sum, const float* group_sum, int table_chunks,
                        float* qbar, int32_t* chunk_idx, int32_t* group_idx, hipStream_t stream) {
    return launch_route_any<true, false>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum, group_sum,
                                         table_chunks, qbar, chunk_idx, group_idx, stream);
}

hipError_t launch_route_from_qbar(const hga_plan& plan, const float* qbar, int q_chunk0,
                                  int n_q_chunks, const float* chunk_sum, const float* group_sum,
                                  int table_chunks, int32_t* chunk_idx, int32_t* group_idx,
                                  hipStream_t stream) {
    return launch_route_any<true, true>(plan, nullptr, q_chunk0, n_q_chunks, chunk_sum, group_sum,
                                        table_chunks, const_cast<float*>(qbar), chunk_idx,
                                        group_idx, stream);
}

hipError_t launch_route_groups(const hga_plan& plan, const float* qbar, const int32_t* chunk_idx,
                               int q_chunk0, int n_q_chunks, const float* group_sum,
                               int table_chunks, int32_t* group_idx, hipStream_t stream) {
    if (plan.p.head_dim == 64)
        return launch_groups_t<64>(plan, qbar, chunk_idx, q_chunk0, n_q_chunks, group_sum,
                                   table_chunks, group_idx, stream);
    return launch_groups_t<128>(plan, qbar, chunk_idx, q_chunk0, n_q_chunks, group_sum,
                                table_chunks, group_idx, stream);
}

}  // namespace hga
