// Mixed-RoPE chunk and group key summaries (Sec. 3.2).
//
// One thread owns one (chunk, group, pair-block): a pair-block is the
// 16 bytes of dimensions [pb*V, pb*V + V) together with their rotate-half
// partners [D/2 + pb*V, ...), V = 16 / sizeof(element).  It walks the
// group's tokens in order, accumulating in fp32 both the group summary and
// its share of the chunk summary:
//   first half  += cos(phi) a - sin(phi) b
//   second half += sin(phi) a + cos(phi) b
// with the span's phase phi_p(o) read from LDS copies of the plan's tables.
// The group share is final; the chunk shares of the chunk's groups are added
// in group order through LDS.  The kernel is bound by the single read of K.
#include "hga_device.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

constexpr int kThreads = 256;

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void build_summaries_kernel(
    const T* __restrict__ k_rot, int64_t k_tokens, int k_chunk0, int chunk_begin, int n_chunks,
    float* __restrict__ chunk_sum, float* __restrict__ group_sum, int table_chunks, int n_kv,
    const float* __restrict__ phase_chunk, const float* __restrict__ phase_group, int chunk,
    int group) {
    constexpr int V = elem<T>::kVec;
    constexpr int HALF = D / 2;
    constexpr int NPB = HALF / V;  // pair-blocks per token
    extern __shared__ float smem[];
    float* s_pc = smem;                       // [2][chunk][HALF]
    float* s_pg = s_pc + 2 * chunk * HALF;    // [2][group][HALF]
    float* s_red = s_pg + 2 * group * HALF;   // [chunks_per_block][gpc][D]

    const int gpc = chunk / group;
    const int tpc = NPB * gpc;              // threads per chunk
    const int cpb = kThreads / tpc;         // chunks per block
    const int bh = blockIdx.y;              // b * n_kv + j
    const int tid = threadIdx.x;

    for (int i = tid; i < 2 * chunk * HALF; i += kThreads) s_pc[i] = phase_chunk[i];
    for (int i = tid; i < 2 * group * HALF; i += kThreads) s_pg[i] = phase_group[i];
    __syncthreads();

    const int local = tid / tpc;
    const int grp = (tid % tpc) / NPB;
    const int pb = tid % NPB;
    const int c_rel = blockIdx.x * cpb + local;   // chunk index within the range
    const bool active = local < cpb && c_rel < n_chunks;

    float ca[V], cb[V], ga[V], gb[V];
#pragma unroll
    for (int e = 0; e < V; ++e) ca[e] = cb[e] = ga[e] = gb[e] = 0.f;

    const int c = chunk_begin + c_rel;
    if (active) {
        const T* base = k_rot + (static_cast<int64_t>(bh) * k_tokens +
                                 static_cast<int64_t>(c - k_chunk0) * chunk + grp * group) * D;
        for (int o2 = 0; o2 < group; ++o2) {
            const int o = grp * group + o2;
            float a[V], b[V];
            elem<T>::unpack(load16(base + o2 * D + pb * V), a);
            elem<T>::unpack(load16(base + o2 * D + HALF + pb * V), b);
            const float* pcc = s_pc + o * HALF + pb * V;
            const float* pcs = s_pc + chunk * HALF + o * HALF + pb * V;
            const float* pgc = s_pg + o2 * HALF + pb * V;
            const float* pgs = s_pg + group * HALF + o2 * HALF + pb * V;
#pragma unroll
            for (int e = 0; e < V; ++e) {
                ca[e] += pcc[e] * a[e] - pcs[e] * b[e];
                cb[e] += pcs[e] * a[e] + pcc[e] * b[e];
                ga[e] += pgc[e] * a[e] - pgs[e] * b[e];
                gb[e] += pgs[e] * a[e] + pgc[e] * b[e];
            }
        }
        const float inv_g = 1.0f / static_cast<float>(group);
        float* gout = group_sum + (static_cast<int64_t>(bh) * table_chunks * gpc +
                                   static_cast<int64_t>(c) * gpc + grp) * D;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            gout[pb * V + e] = ga[e] * inv_g;
            gout[HALF + pb * V + e] = gb[e] * inv_g;
        }
        float* red = s_red + (local * gpc + grp) * D;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            red[pb * V + e] = ca[e];
            red[HALF + pb * V + e] = cb[e];
        }
    }
    __syncthreads();
    // chunk summary: add the groups' shares in group order, one thread per
    // (chunk, dimension).
    const float inv_c = 1.0f / static_cast<float>(chunk);
    for (int i = tid; i < cpb * D; i += kThreads) {
        const int l = i / D, dim = i % D;
        const int cr = blockIdx.x * cpb + l;
        if (cr >= n_chunks) continue;
        const float* red = s_red + l * gpc * D + dim;
        float s = 0.f;
        for (int g = 0; g < gpc; ++g) s += red[g * D];
        chunk_sum[(static_cast<int64_t>(bh) * table_chunks + chunk_begin + cr) * D + dim] =
            s * inv_c;
    }
}

template <typename T, int D>
hipError_t launch_t(const hga_plan& plan, const void* k_rot, int64_t k_tokens, int k_chunk0,
                    int chunk_begin, int chunk_end, float* chunk_sum, float* group_sum,
                    int table_chunks, hipStream_t stream) {
    const hga_params& p = plan.p;
    constexpr int V = elem<T>::kVec;
    constexpr int NPB = (D / 2) / V;
    const int gpc = p.chunk / p.group;
    const int tpc = NPB * gpc;
    const int cpb = kThreads / tpc;
    const int n_chunks = chunk_end - chunk_begin;
    dim3 grid((n_chunks + cpb - 1) / cpb, p.batch * p.n_kv_heads);
    const size_t lds = sizeof(float) * (2 * p.chunk * (D / 2) + 2 * p.group * (D / 2) +
                                        cpb * gpc * D);
    hipLaunchKernelGGL((build_summaries_kernel<T, D>), grid, dim3(kThreads), lds, stream,
                       static_cast<const T*>(k_rot), k_tokens, k_chunk0, chunk_begin, n_chunks,
                       chunk_sum, group_sum, table_chunks, p.n_kv_heads, plan.phase_chunk,
                       plan.phase_group, p.chunk, p.group);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_build_summaries(const hga_plan& plan, const void* k_rot, int64_t k_tokens,
                                  int k_chunk0, int chunk_begin, int chunk_end, float* chunk_sum,
                                  float* group_sum, int table_chunks, hipStream_t stream) {
    const hga_params& p = plan.p;
    if (p.dtype == HGA_F32) {
        if (p.head_dim == 64)
            return launch_t<float, 64>(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end,
                                       chunk_sum, group_sum, table_chunks, stream);
        return launch_t<float, 128>(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end,
                                    chunk_sum, group_sum, table_chunks, stream);
    }
    if (p.head_dim == 64)
        return launch_t<bf16_t, 64>(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end,
                                    chunk_sum, group_sum, table_chunks, stream);
    return launch_t<bf16_t, 128>(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end,
                                 chunk_sum, group_sum, table_chunks, stream);
}

}  // namespace hga
