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

}  // namespace

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
