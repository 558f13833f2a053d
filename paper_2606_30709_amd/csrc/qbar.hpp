// The routing query of a query chunk (Sec. 3.3; chunk-shared routing,
// Sec. 1): q_bar = the mean of the r*64 rotated query rows of KV head j over
// the chunk's 64 tokens and the r query heads that share the head.
#pragma once

#include "hga_device.hpp"

namespace hga {

// One wavefront reduces one query chunk in a fixed order: lane (rs, cv)
// adds the 16-byte column block cv of rows rs, rs + NRS, ... (up to 16 loads
// in flight), then a butterfly over the row slots adds the partial sums; the
// lanes with rs == 0 write out[0 .. D) (any address space).  The order
// depends only on the shapes, so q_bar is bit-identical wherever this runs.
template <typename T, int D>
__device__ __forceinline__ void wave_query_mean(const T* __restrict__ q_rot, int b, int j, int i,
                                                int n_q_heads, int r, int n_q_chunks,
                                                float* out) {
    constexpr int chunk = 64;
    constexpr int V = elem<T>::kVec;
    constexpr int VPR = D / V;                               // 16-byte vectors per row
    constexpr int NRS = 64 / VPR;                            // row slots per wave
    constexpr int UNROLL = 64 / NRS < 16 ? 64 / NRS : 16;    // NRS * UNROLL divides 64 rows
    static_assert((NRS * UNROLL) <= 64 && 64 % (NRS * UNROLL) == 0, "q_bar row tiling");
    const int lane = threadIdx.x & 63;
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
            x[u] = load16(qbase + (hh * qtok + tt) * D);
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
        for (int e = 0; e < V; ++e) out[cv * V + e] = acc[e] * inv;
    }
}

}  // namespace hga
