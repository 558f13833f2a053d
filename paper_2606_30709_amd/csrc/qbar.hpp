// The routing query of a query chunk (Sec. 3.3; chunk-shared routing,
// Sec. 1): q_bar = the mean of the r*64 rotated query rows of KV head j over
// the chunk's 64 tokens and the r query heads that share the head.
#pragma once

#include "hga_device.hpp"

namespace hga {

// One wavefront reduces the r*64 rows of one query chunk in a fixed order:
// lane (rs, cv) adds the 16-byte column block cv of rows rs, rs + NRS, ...
// (UNROLL reads in flight), then a butterfly over the row slots adds the
// partial sums; the lanes with rs == 0 write out[0 .. D) (any address
// space).  row_vec(row, cv) returns that 16-byte block of row `row` (row =
// head * 64 + token) from wherever the rows are held.  Each lane adds its
// rows in ascending order whatever kUnroll (the reads in flight) is, so
// q_bar depends only on the shapes: it is bit-identical wherever this runs
// and wherever the rows are read from.
template <typename T, int D, int kUnroll = 16, typename RowVec>
__device__ __forceinline__ void wave_mean_rows(int rows, RowVec row_vec, float* out) {
    constexpr int V = elem<T>::kVec;
    constexpr int VPR = D / V;                               // 16-byte vectors per row
    constexpr int NRS = 64 / VPR;                            // row slots per wave
    constexpr int UNROLL = 64 / NRS < kUnroll ? 64 / NRS : kUnroll;  // NRS * UNROLL divides 64
    static_assert((NRS * UNROLL) <= 64 && 64 % (NRS * UNROLL) == 0, "q_bar row tiling");
    const int lane = threadIdx.x & 63;
    const int cv = lane % VPR, rs = lane / VPR;
    float acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = 0.f;
    for (int row0 = rs; row0 < rows; row0 += NRS * UNROLL) {
        vec16 x[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) x[u] = row_vec(row0 + u * NRS, cv);
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
        for (int e = 0; e < V; ++e) out[cv * V + e] = acc[e] * inv;
    }
}

// Address of token t of query head h of KV head j's group, query chunk i, in
// the [B, H, n_q_chunks * 64, D] rotated-query layout.
template <typename T, int D>
__device__ __forceinline__ const T* query_chunk_base(const T* q_rot, int b, int j, int i,
                                                     int n_q_heads, int r, int n_q_chunks) {
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * 64;
    return q_rot + ((static_cast<int64_t>(b) * n_q_heads + j * r) * qtok +
                    static_cast<int64_t>(i) * 64) * D;
}

// q_bar of query chunk i of (batch b, KV head j), rows read from HBM.
template <typename T, int D>
__device__ __forceinline__ void wave_query_mean(const T* __restrict__ q_rot, int b, int j, int i,
                                                int n_q_heads, int r, int n_q_chunks,
                                                float* out) {
    constexpr int V = elem<T>::kVec;
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * 64;
    const T* qbase = query_chunk_base<T, D>(q_rot, b, j, i, n_q_heads, r, n_q_chunks);
    wave_mean_rows<T, D>(
        r * 64,
        [&](int row, int cv) { return load16(qbase + ((row >> 6) * qtok + (row & 63)) * D + cv * V); },
        out);
}

}  // namespace hga
