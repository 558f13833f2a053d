// Content-based routing (Sec. 3.3): query-chunk -> chunk scoring with top-K_c
// selection, then group refinement with top-K_g selection.
//
// One wavefront per (batch, KV head, query chunk) unit and up to four units
// per workgroup, each wave with its own LDS region and no workgroup barrier.
// Scores are fp32 dot products (coalesced row reads, a fixed DPP row sum),
// packed with their candidate id into 64-bit keys
// (larger score first, then lower id) held in LDS, and the wave extracts the top k by repeated wave-wide maxima: each lane
// keeps the best key of its own strided share, so a round costs one wave
// reduction plus one rescan of the winning lane's share.
#include "hga_device.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

__device__ __forceinline__ void wave_sync_lds() {
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

// x + x from the lane n below within each 16-lane row (lanes below n add 0).
template <int kCtrl>
__device__ __forceinline__ float add_row_shr(float x) {
    return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), kCtrl, 0xf, 0xf, true));
}

// Scores of 64 candidates by one wavefront, coalesced: the 16 lanes of row
// g = lane/16 read the rows of candidates 16g .. 16g+15, one table row per
// instruction (lane p takes float4 p, and p+16 for D = 128), form partial
// dot products with q_bar (broadcast from LDS), and a DPP prefix sum over the
// row (shifts 1, 2, 4, 8) leaves each candidate's complete score in lane 15
// of the row.  The summation order is fixed, so scores are bit-reproducible.
// Lane 15 of each row writes the keys of its 16 candidates; row_of(k) gives
// the table row (and candidate id) of the batch's k-th candidate, valid(k)
// whether it exists.
template <int D, typename RowOf>
__device__ __forceinline__ void batch_keys(const float* s_q, const float* table, RowOf row_of,
                                           int n_valid, uint64_t* keys) {
    constexpr int F4 = D / 64;  // float4 per lane per row
    const int lane = threadIdx.x & 63;
    const int grp = lane >> 4, p = lane & 15;
    float4 qv[F4];
#pragma unroll
    for (int f = 0; f < F4; ++f) qv[f] = *reinterpret_cast<const float4*>(s_q + (p + 16 * f) * 4);
    float part[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const float* row = table + static_cast<int64_t>(row_of(grp * 16 + k)) * D;
        float a = 0.f;
#pragma unroll
        for (int f = 0; f < F4; ++f) {
            const float4 x = *reinterpret_cast<const float4*>(row + (p + 16 * f) * 4);
            a = fmaf(qv[f].x, x.x, a);
            a = fmaf(qv[f].y, x.y, a);
            a = fmaf(qv[f].z, x.z, a);
            a = fmaf(qv[f].w, x.w, a);
        }
        part[k] = a;
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        float x = part[k];
        x = add_row_shr<0x111>(x);  // row_shr:1
        x = add_row_shr<0x112>(x);  // row_shr:2
        x = add_row_shr<0x114>(x);  // row_shr:4
        x = add_row_shr<0x118>(x);  // row_shr:8
        part[k] = x;
    }
    if (p == 15) {
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const int m = grp * 16 + k;
            if (m < n_valid) keys[m] = select_key(part[k], row_of(m));
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

template <typename T, int D>
__global__ __launch_bounds__(256) void route_chunks_kernel(
    const T* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const float* __restrict__ chunk_sum,
    int table_chunks, float* __restrict__ qbar, int32_t* __restrict__ chunk_idx, int n_q_heads,
    int n_kv, int n_units, int keep_first, int window, int topk, size_t wave_bytes) {
    constexpr int chunk = 64;
    constexpr int V = elem<T>::kVec;
    constexpr int VPR = D / V;              // 16-byte vectors per row
    constexpr int NRS = 64 / VPR;           // row slots per wave
    constexpr int UNROLL = 8;
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int unit = blockIdx.x * (blockDim.x >> 6) + wave;
    if (unit >= n_units) return;
    WaveLds L = carve(smem_raw + wave * wave_bytes, D, 0, topk);
    const int i = unit % n_q_chunks;
    const int bh = unit / n_q_chunks;
    const int b = bh / n_kv, j = bh % n_kv;
    const int r = n_q_heads / n_kv;
    const int c = q_chunk0 + i;

    // 1. q_bar: mean over the r heads x chunk tokens, fixed summation order.
    const int cv = lane % VPR, rs = lane / VPR;
    float acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = 0.f;
    const int rows = r * chunk;
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * chunk;
    const T* qbase = q_rot + ((static_cast<int64_t>(b) * n_q_heads + j * r) * qtok +
                              static_cast<int64_t>(i) * chunk) * D + cv * V;
    for (int row0 = rs; row0 < rows; row0 += NRS * UNROLL) {
        vec16 x[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int row = row0 + u * NRS;
            const int hh = row >> 6, tt = row & 63;
            x[u] = row < rows ? load16(qbase + (hh * qtok + tt) * D) : vec16{{0u, 0u, 0u, 0u}};
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            float f[V];
            elem<T>::unpack(x[u], f);
#pragma unroll
            for (int e = 0; e < V; ++e) acc[e] += f[e];
        }
    }
#pragma unroll
    for (int m = VPR; m < 64; m <<= 1)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] += __shfl_xor(acc[e], m, 64);
    const float inv = 1.0f / static_cast<float>(rows);
    if (rs == 0) {
#pragma unroll
        for (int e = 0; e < V; ++e) L.q[cv * V + e] = acc[e] * inv;
    }
    wave_sync_lds();
    if (lane < VPR) {
        float* out = qbar + static_cast<int64_t>(unit) * D + cv * V;
#pragma unroll
        for (int e = 0; e < V; ++e) out[e] = L.q[cv * V + e];
    }

    // 2. score the middle chunks [keep_first, c - window).
    int n = c - window - keep_first;
    if (n < 0) n = 0;
    const float* table = chunk_sum + static_cast<int64_t>(bh) * table_chunks * D;
    for (int m0 = 0; m0 < n; m0 += 64) {
        const int last = n - 1 - m0;
        batch_keys<D>(L.q, table, [&](int k) { return keep_first + m0 + min(k, last); }, n - m0,
                      L.keys + m0);
    }
    wave_sync_lds();

    // 3. top-k, ascending, -1 padded.
    const int k = n < topk ? n : topk;
    wave_select_topk(L.keys, n, k, L.sel, L.scr);
    wave_sync_lds();
    int32_t* out = chunk_idx + static_cast<int64_t>(unit) * topk;
    for (int t = lane; t < topk; t += 64) out[t] = t < k ? L.sel[t] : -1;
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
    const float* table = group_sum + static_cast<int64_t>(bh) * table_chunks * gpc * D;
    for (int m0 = 0; m0 < n; m0 += 64) {
        const int last = n - 1 - m0;
        auto row_of = [&](int k) {
            const int mm = m0 + min(k, last);
            return L.list[mm >> gpc_shift] * gpc + (mm & (gpc - 1));
        };
        batch_keys<D>(L.q, table, row_of, n - m0, L.keys + m0);
    }
    wave_sync_lds();
    const int k = n < topk_groups ? n : topk_groups;
    wave_select_topk(L.keys, n, k, L.sel, L.scr);
    wave_sync_lds();
    int32_t* out = group_idx + static_cast<int64_t>(unit) * topk_groups;
    for (int t = lane; t < topk_groups; t += 64) out[t] = t < k ? L.sel[t] : -1;
}

// Up to four waves per workgroup, as many as the LDS budget allows.
int waves_per_block(size_t wave_bytes, int max_lds) {
    int w = static_cast<int>(static_cast<size_t>(max_lds) / wave_bytes);
    return w < 1 ? 1 : (w > 4 ? 4 : w);
}

template <typename T, int D>
hipError_t launch_chunks_t(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                           const float* chunk_sum, int table_chunks, float* qbar,
                           int32_t* chunk_idx, hipStream_t stream) {
    const hga_params& p = plan.p;
    const int n_max = middle_count(p, q_chunk0 + n_q_chunks - 1);
    const size_t wb = wave_lds_bytes(D, 0, p.topk_chunks, n_max);
    const int wpb = waves_per_block(wb, plan.max_lds);
    const int n_units = p.batch * p.n_kv_heads * n_q_chunks;
    const int blocks = (n_units + wpb - 1) / wpb;
    hipLaunchKernelGGL((route_chunks_kernel<T, D>), dim3(blocks), dim3(64 * wpb), wb * wpb, stream,
                       static_cast<const T*>(q_rot), q_chunk0, n_q_chunks, chunk_sum,
                       table_chunks, qbar, chunk_idx, p.n_q_heads, p.n_kv_heads, n_units,
                       p.keep_first, recent_window(p), p.topk_chunks, wb);
    return hipGetLastError();
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

size_t route_chunks_lds_bytes(const hga_plan& plan, int n_max) {
    return wave_lds_bytes(plan.p.head_dim, 0, plan.p.topk_chunks, n_max);
}

hipError_t launch_route_chunks(const hga_plan& plan, const void* q_rot, int q_chunk0,
                               int n_q_chunks, const float* chunk_sum, int table_chunks,
                               float* qbar, int32_t* chunk_idx, hipStream_t stream) {
    const hga_params& p = plan.p;
    if (p.dtype == HGA_F32) {
        if (p.head_dim == 64)
            return launch_chunks_t<float, 64>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                              table_chunks, qbar, chunk_idx, stream);
        return launch_chunks_t<float, 128>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                           table_chunks, qbar, chunk_idx, stream);
    }
    if (p.head_dim == 64)
        return launch_chunks_t<bf16_t, 64>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                           table_chunks, qbar, chunk_idx, stream);
    return launch_chunks_t<bf16_t, 128>(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                        table_chunks, qbar, chunk_idx, stream);
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
