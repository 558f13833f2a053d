// Exact-token attention (Sec. 3.4, Eq. (1)) in fp32 on the vector ALUs.
//
// Used for fp32 inputs (the bf16 path runs on the matrix cores).  A
// workgroup of kSplit wavefronts per (batch, query head, query chunk): lane t
// of every wavefront owns query token t of the chunk, and wavefront w takes
// the key tiles w, w + kSplit, ... of the unit's working set with its own
// online softmax (running max / running sum, rescaled once per tile) and
// output accumulator in registers.  Key tiles of 16 rows are staged in a
// wavefront-private LDS region as fp32 (read as broadcasts).  At the end the
// partial results are combined in a fixed order through LDS, with the same
// rule as two halves of a softmax: m = max(m_a, m_b), and each side scaled by
// exp2(m_side - m).
#include <hip/hip_ext.h>
#include <math.h>

#include "attend_common.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

constexpr int kTile = 16;
constexpr int kSplit = 8;  // wavefronts per unit

template <int D>
__global__ __launch_bounds__(64 * kSplit) void attend_valu_kernel(
    const float* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const float* __restrict__ k_res,
    const float* __restrict__ v_res, int64_t res_tokens, const int32_t* __restrict__ res_slot,
    const float* __restrict__ k_routed, const float* __restrict__ v_routed,
    const int32_t* __restrict__ group_idx, float* __restrict__ out, float* __restrict__ lse,
    int n_q_heads, int n_kv, int chunk, int group, int keep_first, int window, int topk_groups,
    const float* __restrict__ k_src, const float* __restrict__ v_src, int64_t src_tokens) {
    extern __shared__ __align__(16) float smem_f[];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    float* s_k = smem_f + wave * (2 * kTile * D + kTile);  // [kTile][D]
    float* s_v = s_k + kTile * D;                          // [kTile][D]
    int* s_valid = reinterpret_cast<int*>(s_v + kTile * D);  // [kTile]

    const int r = n_q_heads / n_kv;
    const int i = blockIdx.x / r, hh = blockIdx.x % r;
    const int bh = blockIdx.y;
    const int b = bh / n_kv, j = bh % n_kv;
    const int c = q_chunk0 + i;
    const int gpc = chunk / group;
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * chunk;
    const int64_t qrow = (static_cast<int64_t>(b) * n_q_heads + j * r + hh) * qtok +
                         static_cast<int64_t>(i) * chunk + lane;
    const float scale = 1.4426950408889634f / sqrtf(static_cast<float>(D));  // log2(e)/sqrt(d)
    const int64_t res_chunks = res_tokens / chunk;

    float q[D], acc[D];
#pragma unroll
    for (int e = 0; e < D; ++e) {
        q[e] = q_rot[qrow * D + e] * scale;
        acc[e] = 0.f;
    }
    float m_run = -INFINITY, l_run = 0.f;
    bool bad = false;

    const VisibleChunks vis(c, keep_first, window);
    const int64_t unit = static_cast<int64_t>(bh) * n_q_chunks + i;
    const int32_t* gi = group_idx + unit * topk_groups;
    const int routed_rows = topk_groups * group;
    const int n_vis_tiles = vis.count * (chunk / kTile);
    const int n_rt_tiles = (routed_rows + kTile - 1) / kTile;
    const int n_tiles = n_vis_tiles + n_rt_tiles + chunk / kTile;

    for (int tile = wave; tile < n_tiles; tile += kSplit) {
        // locate this tile's rows
        const float* ksrc = nullptr;
        const float* vsrc = nullptr;
        int kind, row0 = 0;
        if (tile < n_vis_tiles) {
            kind = kTileVisible;
            const int cc = vis.chunk(tile / (chunk / kTile));
            int64_t slot = res_slot ? res_slot[cc] : cc;
            if (slot < 0 || slot >= res_chunks) { bad = true; slot = 0; }
            const int64_t off = (static_cast<int64_t>(bh) * res_tokens + slot * chunk +
                                 (tile % (chunk / kTile)) * kTile) * D;
            ksrc = k_res + off;
            vsrc = v_res + off;
        } else if (tile < n_vis_tiles + n_rt_tiles) {
            kind = kTileRouted;
            row0 = (tile - n_vis_tiles) * kTile;
            if (k_routed) {
                const int64_t off = (unit * routed_rows + row0) * D;
                ksrc = k_routed + off;
                vsrc = v_routed + off;
            }
        } else {
            kind = kTileCurrent;
            row0 = (tile - n_vis_tiles - n_rt_tiles) * kTile;
            int64_t slot = res_slot ? res_slot[c] : c;
            if (slot < 0 || slot >= res_chunks) { bad = true; slot = 0; }
            const int64_t off = (static_cast<int64_t>(bh) * res_tokens + slot * chunk + row0) * D;
            ksrc = k_res + off;
            vsrc = v_res + off;
        }
        __builtin_amdgcn_wave_barrier();  // this wave is done reading its previous tile
        for (int x = lane; x < kTile * D; x += 64) {
            const int rr = x / D, e = x % D;
            bool ok = true;
            if (kind == kTileRouted) {
                const int row = row0 + rr;
                ok = row < routed_rows;
                if (ok) {
                    const int g = gi[row / group];
                    ok = g >= 0 && g < c * gpc;
                }
            }
            const float* kp = ksrc ? ksrc + rr * D + e : nullptr;
            const float* vp = vsrc ? vsrc + rr * D + e : nullptr;
            if (!ksrc && ok) {
                // no routed buffers: routed row R of group gi[R / G] is row
                // g*G + R % G of the routed-row source (the gather's rule)
                const int row = row0 + rr;
                const int64_t tok = static_cast<int64_t>(gi[row / group]) * group + row % group;
                kp = k_src + (static_cast<int64_t>(bh) * src_tokens + tok) * D + e;
                vp = v_src + (static_cast<int64_t>(bh) * src_tokens + tok) * D + e;
            }
            s_k[rr * D + e] = ok ? *kp : 0.f;
            s_v[rr * D + e] = ok ? *vp : 0.f;
            if (e == 0) s_valid[rr] = ok;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

        float sc[kTile];
        float tmax = -INFINITY;
#pragma unroll
        for (int kk = 0; kk < kTile; ++kk) {
            float dot = 0.f;
#pragma unroll
            for (int e = 0; e < D; ++e) dot = fmaf(q[e], s_k[kk * D + e], dot);
            bool ok = s_valid[kk];
            if (kind == kTileCurrent) ok = (row0 + kk) <= lane;
            sc[kk] = ok ? dot : -INFINITY;
            tmax = fmaxf(tmax, sc[kk]);
        }
        const float m_new = fmaxf(m_run, tmax);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(m_run - m_use);
        l_run *= alpha;
#pragma unroll
        for (int e = 0; e < D; ++e) acc[e] *= alpha;
#pragma unroll
        for (int kk = 0; kk < kTile; ++kk) {
            const float pk = exp2f(sc[kk] - m_use);
            l_run += pk;
#pragma unroll
            for (int e = 0; e < D; ++e) acc[e] = fmaf(pk, s_v[kk * D + e], acc[e]);
        }
        m_run = m_new;
    }

    // Combine the wavefronts' partial results into wavefront 0, one at a
    // time, through LDS (element e of lane l at [e][l]).
    float* part = smem_f;  // [D + 2][64]
    const unsigned bad_any = __syncthreads_or(bad);
    for (int w = 1; w < kSplit; ++w) {
        __syncthreads();
        if (wave == w) {
#pragma unroll
            for (int e = 0; e < D; ++e) part[e * 64 + lane] = acc[e];
            part[D * 64 + lane] = m_run;
            part[(D + 1) * 64 + lane] = l_run;
        }
        __syncthreads();
        if (wave == 0) {
            const float mb = part[D * 64 + lane], lb = part[(D + 1) * 64 + lane];
            const float m = fmaxf(m_run, mb);
            const float mu = m == -INFINITY ? 0.f : m;
            const float fa = exp2f(m_run - mu), fb = exp2f(mb - mu);
#pragma unroll
            for (int e = 0; e < D; ++e) acc[e] = acc[e] * fa + part[e * 64 + lane] * fb;
            l_run = l_run * fa + lb * fb;
            m_run = m;
        }
    }
    if (wave != 0) return;

    const float inv = 1.0f / l_run;
    float* orow = out + qrow * D;
#pragma unroll
    for (int e = 0; e < D; ++e) orow[e] = bad_any ? NAN : acc[e] * inv;
    if (lse) lse[qrow] = bad_any ? NAN : (m_run + log2f(l_run)) * 0.6931471805599453f;
}

}  // namespace

hipError_t launch_attend_valu(const hga_plan& plan, const void* q_rot, int q_chunk0,
                              int n_q_chunks, const void* k_res, const void* v_res,
                              int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                              const void* v_routed, const int32_t* group_idx, void* out,
                              float* lse, hipEvent_t ev_start, hipEvent_t ev_stop,
                              hipStream_t stream, const void* k_src, const void* v_src,
                              int64_t src_tokens) {
    const hga_params& p = plan.p;
    const int r = p.n_q_heads / p.n_kv_heads;
    dim3 grid(n_q_chunks * r, p.batch * p.n_kv_heads);
    const size_t tiles = static_cast<size_t>(kSplit) * (2 * kTile * p.head_dim + kTile) * 4;
    const size_t merge = static_cast<size_t>(p.head_dim + 2) * 64 * 4;
    const size_t lds = tiles > merge ? tiles : merge;
#define HGA_VALU(DD)                                                                            \
    do {                                                                                        \
        static std::atomic<uint64_t> configured{0}; /* per kernel and device */                \
        const hipError_t ce = once_per_device(configured, plan.device, [&] {                   \
            return hipFuncSetAttribute(reinterpret_cast<const void*>(&attend_valu_kernel<DD>),  \
                                       hipFuncAttributeMaxDynamicSharedMemorySize,              \
                                       static_cast<int>(lds));                                  \
        });                                                                                     \
        if (ce != hipSuccess) return ce;                                                        \
        hipExtLaunchKernelGGL((attend_valu_kernel<DD>), grid, dim3(64 * kSplit), lds, stream,   \
                              ev_start, ev_stop, 0, static_cast<const float*>(q_rot), q_chunk0, \
                              n_q_chunks, static_cast<const float*>(k_res),                     \
                              static_cast<const float*>(v_res), res_tokens, res_slot,           \
                              static_cast<const float*>(k_routed),                              \
                              static_cast<const float*>(v_routed), group_idx,                   \
                              static_cast<float*>(out), lse, p.n_q_heads, p.n_kv_heads,         \
                              p.chunk, p.group, p.keep_first, recent_window(p), p.topk_groups,  \
                              static_cast<const float*>(k_src), static_cast<const float*>(v_src), \
                              src_tokens);                                                      \
    } while (0)
    if (p.head_dim == 64)
        HGA_VALU(64);
    else
        HGA_VALU(128);
#undef HGA_VALU
    return hipGetLastError();
}

}  // namespace hga
