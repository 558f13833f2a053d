// Content-based routing (Sec. 3.3): query-chunk -> chunk scoring with top-K_c
// selection, then group refinement with top-K_g selection.
//
// One workgroup per (batch, KV head, query chunk).  Scores are fp32 dot
// products reduced in a fixed order, packed with their candidate id into
// 64-bit keys (larger score first, then lower id) held in LDS, and one
// wavefront extracts the top k by repeated wave-wide maxima.  Each lane keeps
// the best key of its own strided share, so a round costs one wave reduction
// plus one rescan of the winning lane's share.
#include "hga_device.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

constexpr int kThreads = 256;
constexpr int kLanesPerCand = 16;  // lanes cooperating on one dot product

// Dot product of the LDS query mean with a global fp32 row of length D, by the
// 16 lanes of a lane group; every lane of the group returns the sum.
template <int D>
__device__ __forceinline__ float group_dot(const float* s_q, const float* row, int part) {
    constexpr int PER = D / kLanesPerCand;  // 4 or 8 floats per lane
    float acc = 0.f;
#pragma unroll
    for (int v = 0; v < PER / 4; ++v) {
        const float4 x = *reinterpret_cast<const float4*>(row + part * PER + v * 4);
        const float* q = s_q + part * PER + v * 4;
        acc = fmaf(q[0], x.x, acc);
        acc = fmaf(q[1], x.y, acc);
        acc = fmaf(q[2], x.z, acc);
        acc = fmaf(q[3], x.w, acc);
    }
#pragma unroll
    for (int m = kLanesPerCand / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
    return acc;
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void route_chunks_kernel(
    const T* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const float* __restrict__ chunk_sum,
    int table_chunks, float* __restrict__ qbar, int32_t* __restrict__ chunk_idx, int n_q_heads,
    int n_kv, int chunk, int keep_first, int window, int topk) {
    constexpr int V = elem<T>::kVec;
    constexpr int VPR = D / V;              // 16-byte vectors per row
    constexpr int NRS = kThreads / VPR;     // row slots
    extern __shared__ __align__(16) unsigned char smem_raw[];
    float* s_part = reinterpret_cast<float*>(smem_raw);   // [NRS][D]
    float* s_q = s_part + NRS * D;                        // [D]
    int* s_sel = reinterpret_cast<int*>(s_q + D);         // [topk]
    int* s_scr = s_sel + topk;                            // [topk]
    uint64_t* s_keys = reinterpret_cast<uint64_t*>(
        smem_raw + ((sizeof(float) * (NRS * D + D) + sizeof(int) * 2 * topk + 15) & ~size_t(15)));

    const int i = blockIdx.x;
    const int bh = blockIdx.y;
    const int b = bh / n_kv, j = bh % n_kv;
    const int r = n_q_heads / n_kv;
    const int tid = threadIdx.x;
    const int c = q_chunk0 + i;

    // 1. q_bar: mean over the r heads x chunk tokens, fixed summation order.
    {
        const int cv = tid % VPR, rs = tid / VPR;
        float acc[V];
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] = 0.f;
        const int rows = r * chunk;
        const int64_t qtok = static_cast<int64_t>(n_q_chunks) * chunk;
        for (int row = rs; row < rows; row += NRS) {
            const int hh = row / chunk, tt = row % chunk;
            const T* src = q_rot + ((static_cast<int64_t>(b) * n_q_heads + j * r + hh) * qtok +
                                    static_cast<int64_t>(i) * chunk + tt) * D + cv * V;
            float x[V];
            elem<T>::unpack(load16(src), x);
#pragma unroll
            for (int e = 0; e < V; ++e) acc[e] += x[e];
        }
#pragma unroll
        for (int e = 0; e < V; ++e) s_part[rs * D + cv * V + e] = acc[e];
    }
    __syncthreads();
    if (tid < D) {
        float s = 0.f;
        for (int rs = 0; rs < NRS; ++rs) s += s_part[rs * D + tid];
        s *= 1.0f / static_cast<float>(r * chunk);
        s_q[tid] = s;
        qbar[(static_cast<int64_t>(bh) * n_q_chunks + i) * D + tid] = s;
    }
    __syncthreads();

    // 2. score the middle chunks [keep_first, c - window).
    int n = c - window - keep_first;
    if (n < 0) n = 0;
    const float* table = chunk_sum + static_cast<int64_t>(bh) * table_chunks * D;
    {
        const int part = tid % kLanesPerCand;
        for (int m = tid / kLanesPerCand; m < n; m += kThreads / kLanesPerCand) {
            const int cand = keep_first + m;
            const float s = group_dot<D>(s_q, table + static_cast<int64_t>(cand) * D, part);
            if (part == 0) s_keys[m] = select_key(s, cand);
        }
    }
    __syncthreads();

    // 3. top-k by wave 0, ascending, -1 padded.
    if (tid < 64) {
        const int k = n < topk ? n : topk;
        wave_select_topk(s_keys, n, k, s_sel, s_scr);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        int32_t* out = chunk_idx + (static_cast<int64_t>(bh) * n_q_chunks + i) * topk;
        for (int t = tid; t < topk; t += 64) out[t] = t < k ? s_sel[t] : -1;
    }
}

template <int D>
__global__ __launch_bounds__(kThreads) void route_groups_kernel(
    const float* __restrict__ qbar, const int32_t* __restrict__ chunk_idx, int q_chunk0,
    int n_q_chunks, const float* __restrict__ group_sum, int table_chunks,
    int32_t* __restrict__ group_idx, int topk_chunks, int topk_groups, int gpc) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    float* s_q = reinterpret_cast<float*>(smem_raw);      // [D]
    int* s_chunks = reinterpret_cast<int*>(s_q + D);      // [topk_chunks]
    int* s_sel = s_chunks + topk_chunks;                  // [topk_groups]
    int* s_scr = s_sel + topk_groups;                     // [topk_groups]
    int* s_nvalid = s_scr + topk_groups;                  // [1]
    uint64_t* s_keys = reinterpret_cast<uint64_t*>(
        smem_raw + ((sizeof(float) * D + sizeof(int) * (topk_chunks + 2 * topk_groups + 1) + 15) &
                    ~size_t(15)));

    const int i = blockIdx.x;
    const int bh = blockIdx.y;
    const int tid = threadIdx.x;
    const int c = q_chunk0 + i;
    const int limit = c < table_chunks ? c : table_chunks;

    if (tid < D) s_q[tid] = qbar[(static_cast<int64_t>(bh) * n_q_chunks + i) * D + tid];
    if (tid == 0) {
        const int32_t* row = chunk_idx + (static_cast<int64_t>(bh) * n_q_chunks + i) * topk_chunks;
        int nv = 0;
        for (int t = 0; t < topk_chunks; ++t) {
            const int cc = row[t];
            if (cc >= 0 && cc < limit) s_chunks[nv++] = cc;
        }
        *s_nvalid = nv;
    }
    __syncthreads();
    const int n = *s_nvalid * gpc;
    const float* table = group_sum + static_cast<int64_t>(bh) * table_chunks * gpc * D;
    {
        const int part = tid % kLanesPerCand;
        for (int m = tid / kLanesPerCand; m < n; m += kThreads / kLanesPerCand) {
            const int g = s_chunks[m / gpc] * gpc + m % gpc;
            const float s = group_dot<D>(s_q, table + static_cast<int64_t>(g) * D, part);
            if (part == 0) s_keys[m] = select_key(s, g);
        }
    }
    __syncthreads();
    if (tid < 64) {
        const int k = n < topk_groups ? n : topk_groups;
        wave_select_topk(s_keys, n, k, s_sel, s_scr);
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        int32_t* out = group_idx + (static_cast<int64_t>(bh) * n_q_chunks + i) * topk_groups;
        for (int t = tid; t < topk_groups; t += 64) out[t] = t < k ? s_sel[t] : -1;
    }
}

template <typename T, int D>
hipError_t launch_chunks_t(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                           const float* chunk_sum, int table_chunks, float* qbar,
                           int32_t* chunk_idx, hipStream_t stream) {
    const hga_params& p = plan.p;
    constexpr int V = elem<T>::kVec;
    constexpr int NRS = kThreads / (D / V);
    const int window = recent_window(p);
    const int n_max = middle_count(p, q_chunk0 + n_q_chunks - 1);
    const size_t head = (sizeof(float) * (NRS * D + D) + sizeof(int) * 2 * p.topk_chunks + 15) &
                        ~size_t(15);
    const size_t lds = head + sizeof(uint64_t) * (n_max > 0 ? n_max : 1);
    dim3 grid(n_q_chunks, p.batch * p.n_kv_heads);
    hipLaunchKernelGGL((route_chunks_kernel<T, D>), grid, dim3(kThreads), lds, stream,
                       static_cast<const T*>(q_rot), q_chunk0, n_q_chunks, chunk_sum,
                       table_chunks, qbar, chunk_idx, p.n_q_heads, p.n_kv_heads, p.chunk,
                       p.keep_first, window, p.topk_chunks);
    return hipGetLastError();
}

template <int D>
hipError_t launch_groups_t(const hga_plan& plan, const float* qbar, const int32_t* chunk_idx,
                           int q_chunk0, int n_q_chunks, const float* group_sum, int table_chunks,
                           int32_t* group_idx, hipStream_t stream) {
    const hga_params& p = plan.p;
    const int gpc = p.chunk / p.group;
    const size_t head = (sizeof(float) * D + sizeof(int) * (p.topk_chunks + 2 * p.topk_groups + 1) +
                         15) & ~size_t(15);
    const size_t lds = head + sizeof(uint64_t) * p.topk_chunks * gpc;
    dim3 grid(n_q_chunks, p.batch * p.n_kv_heads);
    hipLaunchKernelGGL((route_groups_kernel<D>), grid, dim3(kThreads), lds, stream, qbar,
                       chunk_idx, q_chunk0, n_q_chunks, group_sum, table_chunks, group_idx,
                       p.topk_chunks, p.topk_groups, gpc);
    return hipGetLastError();
}

}  // namespace

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
