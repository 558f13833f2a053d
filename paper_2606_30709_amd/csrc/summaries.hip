// Mixed-RoPE chunk and group key summaries (Sec. 3.2).
//
// For a pair p of a span starting at token s, the summary adds
// R(phi_p(o)) k_rot[s + o] over the span (then divides by its length), with
// phi_p(o) = 0 for high-frequency pairs and ((span-1)/2 - o) theta_p for the
// others.  With C = chunk and G = group, a chunk is gpc = C/G groups, and for
// a low-frequency pair the chunk phase of token o = g*G + o' splits as
//   ((C-1)/2 - o) theta_p = psi_g theta_p + ((G-1)/2 - o') theta_p,
//   psi_g = (C - G)/2 - g*G,
// so the chunk sum is the sum over its groups of R(psi_g theta_p) times the
// group sum (an identity of rotations).  High-frequency chunk pairs are plain
// sums of the rotated keys.  This needs every high-frequency group pair to be
// a high-frequency chunk pair, which the wavelength rule guarantees (the plan
// rejects other settings).
//
// Layout of the work: one wavefront per chunk.  Lane (pb, ts) owns the
// pair-block pb (eight dimensions [8 pb, 8 pb + 8) and their rotate-half
// partners) of the consecutive tokens of slice ts.  Every lane issues all
// its loads at once, accumulates its slice, pre-rotates the chunk share by its
// group's psi_g, and the slices are added in a fixed order through LDS.  The
// group phase table and the psi table live in LDS.
#include "hga_device.hpp"
#include "hga_internal.hpp"
#include "qbar.hpp"

namespace hga {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

template <typename T, int D>
struct SumGeom {
    static constexpr int V = 8;                     // pairs per lane (a pair-block)
    static constexpr int LV = elem<T>::kVec;        // elements per 16-byte load
    static constexpr int VPH = V / LV;              // loads per half pair-block
    static constexpr int HALF = D / 2;
    static constexpr int NPB = HALF / V;            // pair-blocks per token
    static constexpr int TPL = NPB;                 // tokens per lane (64 lanes per chunk)
    static constexpr int SLICES = 64 / NPB;         // token slices per chunk
    static constexpr int RD = D + 1;                // reduction row stride (floats)
};

// The summary work of workgroup `block` of `n_blocks` (a grid-stride loop
// over the (batch, KV head, chunk) items).
template <typename T, int D>
__device__ __forceinline__ void summaries_body(
    int block, int n_blocks, const T* __restrict__ k_rot, int64_t k_tokens, int k_chunk0,
    int chunk_begin, int n_chunks, float* __restrict__ chunk_sum, float* __restrict__ group_sum,
    int table_chunks, int n_bh, const float* __restrict__ phase_group,
    const float* __restrict__ phase_psi, int group, int hf_chunk) {
    using Gm = SumGeom<T, D>;
    constexpr int V = Gm::V, LV = Gm::LV, VPH = Gm::VPH, HALF = Gm::HALF, NPB = Gm::NPB,
                  TPL = Gm::TPL, SLICES = Gm::SLICES;
    constexpr int C = 64;
    // LDS rows padded so lanes reading or writing the same column of
    // different rows hit different banks (the reduction rows by one word:
    // they are only accessed a word at a time).
    constexpr int PH = HALF + 4;                   // phase-table row stride
    constexpr int RD = Gm::RD;                     // reduction row stride
    extern __shared__ __align__(16) float smem[];
    const int gpc = C / group;
    float* s_pg = smem;                            // [2][group][PH]
    float* s_psi = s_pg + 2 * group * PH;          // [2][gpc][PH]
    float* s_red = s_psi + 2 * gpc * PH;           // [kWaves][2][SLICES][RD]

    const int tid = threadIdx.x;
    {
        // the phase tables: 16-byte pieces, every load issued before any store
        constexpr int H4 = HALF / 4;
        constexpr int MAXG = (2 * 32 * H4 + kThreads - 1) / kThreads;  // group <= 32
        constexpr int MAXP = (2 * 8 * H4 + kThreads - 1) / kThreads;   // gpc <= 8
        const int ng4 = 2 * group * H4, np4 = 2 * gpc * H4;
        float4 tg[MAXG], tp[MAXP];
#pragma unroll
        for (int u = 0; u < MAXG; ++u) {
            const int x = tid + u * kThreads;
            tg[u] = reinterpret_cast<const float4*>(phase_group)[min(x, ng4 - 1)];
        }
#pragma unroll
        for (int u = 0; u < MAXP; ++u) {
            const int x = tid + u * kThreads;
            tp[u] = reinterpret_cast<const float4*>(phase_psi)[min(x, np4 - 1)];
        }
#pragma unroll
        for (int u = 0; u < MAXG; ++u) {
            const int x = tid + u * kThreads;
            if (x < ng4) *reinterpret_cast<float4*>(s_pg + (x / H4) * PH + (x % H4) * 4) = tg[u];
        }
#pragma unroll
        for (int u = 0; u < MAXP; ++u) {
            const int x = tid + u * kThreads;
            if (x < np4) *reinterpret_cast<float4*>(s_psi + (x / H4) * PH + (x % H4) * 4) = tp[u];
        }
    }
    __syncthreads();

    const int wave = tid >> 6, lane = tid & 63;
    const int pb = lane % NPB, ts = lane / NPB;
    const int o0 = ts * TPL;                       // first token of the slice
    const int g = o0 / group;                      // its group (a slice lies in one group)
    float* red = s_red + wave * 2 * SLICES * RD;
    const int64_t total = static_cast<int64_t>(n_bh) * n_chunks;

    for (int64_t item0 = static_cast<int64_t>(block) * kWaves; item0 < total;
         item0 += static_cast<int64_t>(n_blocks) * kWaves) {
        const int64_t item = item0 + wave;
        const bool active = item < total;
        const int bh = active ? static_cast<int>(item / n_chunks) : 0;
        const int c = chunk_begin + (active ? static_cast<int>(item % n_chunks) : 0);
        const T* src = k_rot + (static_cast<int64_t>(bh) * k_tokens +
                                static_cast<int64_t>(c - k_chunk0) * C + o0) * D;
        vec16 ra[TPL][VPH], rb[TPL][VPH];
        if (active) {
#pragma unroll
            for (int u = 0; u < TPL; ++u)
#pragma unroll
                for (int h = 0; h < VPH; ++h) {
                    ra[u][h] = load16(src + u * D + pb * V + h * LV);
                    rb[u][h] = load16(src + u * D + HALF + pb * V + h * LV);
                }
        }
        float ga[V], gb[V], pa[V], pbv[V];
#pragma unroll
        for (int e = 0; e < V; ++e) ga[e] = gb[e] = pa[e] = pbv[e] = 0.f;
        if (active) {
#pragma unroll
            for (int u = 0; u < TPL; ++u) {
                float a[V], b[V];
#pragma unroll
                for (int h = 0; h < VPH; ++h) {
                    elem<T>::unpack(ra[u][h], a + h * LV);
                    elem<T>::unpack(rb[u][h], b + h * LV);
                }
                const int o2 = (o0 + u) & (group - 1);
                const float* pc = s_pg + o2 * PH + pb * V;
                const float* ps = s_pg + (group + o2) * PH + pb * V;
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    ga[e] += pc[e] * a[e] - ps[e] * b[e];
                    gb[e] += ps[e] * a[e] + pc[e] * b[e];
                    pa[e] += a[e];
                    pbv[e] += b[e];
                }
            }
        }
        // slice shares: [0] group sum, [1] chunk sum (rotated by psi_g, or plain
        // for high-frequency chunk pairs)
        const float* qc = s_psi + g * PH + pb * V;
        const float* qs = s_psi + (gpc + g) * PH + pb * V;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const int p = pb * V + e;
            red[ts * RD + p] = ga[e];
            red[ts * RD + HALF + p] = gb[e];
            const bool hf = p < hf_chunk;
            red[(SLICES + ts) * RD + p] = hf ? pa[e] : qc[e] * ga[e] - qs[e] * gb[e];
            red[(SLICES + ts) * RD + HALF + p] = hf ? pbv[e] : qs[e] * ga[e] + qc[e] * gb[e];
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        if (active) {
            const int spg = group / TPL;  // slices per group
            const float inv_g = 1.0f / static_cast<float>(group);
            float* gout = group_sum + (static_cast<int64_t>(bh) * table_chunks + c) * gpc * D;
            for (int x = lane; x < gpc * D; x += 64) {
                const int gg = x / D, dim = x % D;
                float s = 0.f;
                for (int k = 0; k < spg; ++k) s += red[(gg * spg + k) * RD + dim];
                gout[x] = s * inv_g;
            }
            const float inv_c = 1.0f / static_cast<float>(C);
            float* cout_ = chunk_sum + (static_cast<int64_t>(bh) * table_chunks + c) * D;
            for (int dim = lane; dim < D; dim += 64) {
                float s = 0.f;
                for (int k = 0; k < SLICES; ++k) s += red[(SLICES + k) * RD + dim];
                cout_[dim] = s * inv_c;
            }
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void build_summaries_kernel(
    const T* __restrict__ k_rot, int64_t k_tokens, int k_chunk0, int chunk_begin, int n_chunks,
    float* __restrict__ chunk_sum, float* __restrict__ group_sum, int table_chunks, int n_bh,
    const float* __restrict__ phase_group, const float* __restrict__ phase_psi, int group,
    int hf_chunk) {
    summaries_body<T, D>(blockIdx.x, gridDim.x, k_rot, k_tokens, k_chunk0, chunk_begin, n_chunks,
                         chunk_sum, group_sum, table_chunks, n_bh, phase_group, phase_psi, group,
                         hf_chunk);
}

// Summaries (workgroups [0, n_sum_blocks)) and, in the same launch, q_bar of
// every query chunk (the other workgroups, one wavefront per (batch, KV head,
// query chunk)): the two read different tensors (K and Q) and are
// independent, so one launch streams both.
template <typename T, int D>
__global__ __launch_bounds__(kThreads) void summaries_qbar_kernel(
    const T* __restrict__ k_rot, int64_t k_tokens, int k_chunk0, int chunk_begin, int n_chunks,
    float* __restrict__ chunk_sum, float* __restrict__ group_sum, int table_chunks, int n_bh,
    const float* __restrict__ phase_group, const float* __restrict__ phase_psi, int group,
    int hf_chunk, int n_sum_blocks, const T* __restrict__ q_rot, int n_q_chunks,
    float* __restrict__ qbar, int n_q_heads, int n_kv) {
    if (static_cast<int>(blockIdx.x) < n_sum_blocks) {
        summaries_body<T, D>(blockIdx.x, n_sum_blocks, k_rot, k_tokens, k_chunk0, chunk_begin,
                             n_chunks, chunk_sum, group_sum, table_chunks, n_bh, phase_group,
                             phase_psi, group, hf_chunk);
        return;
    }
    const int unit = (static_cast<int>(blockIdx.x) - n_sum_blocks) * kWaves + (threadIdx.x >> 6);
    if (unit >= n_bh * n_q_chunks) return;
    const int i = unit % n_q_chunks, bh = unit / n_q_chunks;
    wave_query_mean<T, D>(q_rot, bh / n_kv, bh % n_kv, i, n_q_heads, n_q_heads / n_kv, n_q_chunks,
                          qbar + static_cast<int64_t>(unit) * D);
}

template <typename T, int D>
hipError_t launch_t(const hga_plan& plan, const void* k_rot, int64_t k_tokens, int k_chunk0,
                    int chunk_begin, int chunk_end, float* chunk_sum, float* group_sum,
                    int table_chunks, hipStream_t stream) {
    using Gm = SumGeom<T, D>;
    const hga_params& p = plan.p;
    const int gpc = p.chunk / p.group;
    const int n_chunks = chunk_end - chunk_begin;
    const int n_bh = p.batch * p.n_kv_heads;
    const int64_t items = static_cast<int64_t>(n_bh) * n_chunks;
    int64_t blocks = (items + kWaves - 1) / kWaves;
    if (blocks > 4096) blocks = 4096;
    const size_t lds = sizeof(float) * (2 * p.group * (Gm::HALF + 4) + 2 * gpc * (Gm::HALF + 4) +
                                        kWaves * 2 * Gm::SLICES * Gm::RD);
    hipLaunchKernelGGL((build_summaries_kernel<T, D>), dim3(static_cast<unsigned>(blocks)),
                       dim3(kThreads), lds, stream, static_cast<const T*>(k_rot), k_tokens,
                       k_chunk0, chunk_begin, n_chunks, chunk_sum, group_sum, table_chunks, n_bh,
                       plan.phase_group, plan.phase_psi, p.group, p.hf_pairs_chunk);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_sq_t(const hga_plan& plan, const void* k_rot, int64_t k_tokens, int k_chunk0,
                       int chunk_begin, int chunk_end, float* chunk_sum, float* group_sum,
                       int table_chunks, const void* q_rot, int n_q_chunks, float* qbar,
                       hipStream_t stream) {
    using Gm = SumGeom<T, D>;
    const hga_params& p = plan.p;
    const int gpc = p.chunk / p.group;
    const int n_chunks = chunk_end - chunk_begin;
    const int n_bh = p.batch * p.n_kv_heads;
    const int64_t items = static_cast<int64_t>(n_bh) * n_chunks;
    int64_t sum_blocks = (items + kWaves - 1) / kWaves;
    if (sum_blocks > 4096) sum_blocks = 4096;
    const int64_t q_blocks = (static_cast<int64_t>(n_bh) * n_q_chunks + kWaves - 1) / kWaves;
    if (sum_blocks + q_blocks > (int64_t(1) << 30)) return hipErrorInvalidConfiguration;
    const size_t lds = sizeof(float) * (2 * p.group * (Gm::HALF + 4) + 2 * gpc * (Gm::HALF + 4) +
                                        kWaves * 2 * Gm::SLICES * Gm::RD);
    hipLaunchKernelGGL((summaries_qbar_kernel<T, D>),
                       dim3(static_cast<unsigned>(sum_blocks + q_blocks)), dim3(kThreads), lds,
                       stream, static_cast<const T*>(k_rot), k_tokens, k_chunk0, chunk_begin,
                       n_chunks, chunk_sum, group_sum, table_chunks, n_bh, plan.phase_group,
                       plan.phase_psi, p.group, p.hf_pairs_chunk, static_cast<int>(sum_blocks),
                       static_cast<const T*>(q_rot), n_q_chunks, qbar, p.n_q_heads, p.n_kv_heads);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_summaries_qbar(const hga_plan& plan, const void* k_rot, int64_t k_tokens,
                                 int k_chunk0, int chunk_begin, int chunk_end, float* chunk_sum,
                                 float* group_sum, int table_chunks, const void* q_rot,
                                 int q_chunk0, int n_q_chunks, float* qbar, hipStream_t stream) {
    (void)q_chunk0;  // q_bar depends on the query rows only
    const hga_params& p = plan.p;
    if (p.dtype == HGA_F32) {
        if (p.head_dim == 64)
            return launch_sq_t<float, 64>(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end,
                                          chunk_sum, group_sum, table_chunks, q_rot, n_q_chunks,
                                          qbar, stream);
        return launch_sq_t<float, 128>(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end,
                                       chunk_sum, group_sum, table_chunks, q_rot, n_q_chunks,
                                       qbar, stream);
    }
    if (p.head_dim == 64)
        return launch_sq_t<bf16_t, 64>(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end,
                                       chunk_sum, group_sum, table_chunks, q_rot, n_q_chunks, qbar,
                                       stream);
    return launch_sq_t<bf16_t, 128>(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end,
                                    chunk_sum, group_sum, table_chunks, q_rot, n_q_chunks, qbar,
                                    stream);
}

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
