// Exact-token attention (Sec. 3.4, Eq. (1)) for bf16 inputs on the gfx950
// matrix cores (v_mfma_f32_32x32x16_bf16), flash style.
//
// Work unit: one (batch, KV head, query chunk).  All r = Hq/Hkv query heads
// of the KV head share the unit's working set (GQA, Sec. 2), so their
// r*64 query rows are packed as 32-row query tiles; a workgroup of four
// wavefronts takes four query tiles (or, with only two tiles, two
// wavefronts per tile split each key tile between them and merge at the end).
//
// Keys stream through LDS in 64-key tiles: the visible closed chunks, the
// routed rows, then the current chunk under the causal mask.  Per tile and
// wavefront:
//   S^T[key][query] = K_tile . Q^T        (A = K rows from LDS, B = Q in VGPRs)
// so every lane owns one query column: the running max, running sum and the
// rescaling of the output are per-lane scalars, and a row maximum needs only
// one exchange with the lane holding the other half of the tile's keys.
//   O^T[d][query] += V^T . P^T            (A = V^T from LDS, B = P in VGPRs)
// P is rounded to bf16 for the product; statistics and accumulators are fp32.
// V is written to LDS transposed so that the A operand's eight keys at a fixed
// dimension are two 8-byte LDS reads.  The next tile's K/V are fetched into
// registers while the current one is being consumed.
#include <math.h>

#include "attend_common.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int KT = 64;  // keys per LDS tile (= chunk)

template <int D>
struct Smem {
    static constexpr int KSTR = D + 8;   // K row stride in LDS (bf16): +16 B against bank conflicts
    static constexpr int VSTR = KT + 8;  // V^T row stride (bf16)
    static constexpr int kTileBytes = (KT * KSTR + D * VSTR) * 2;
    static constexpr int NDT = D / 32;
    // merge area: per query-tile slot and lane, the output accumulators, m and l
    static constexpr int kMergeBytes = 2 * 64 * (NDT * 16 + 2) * 4;
    static constexpr int kBytes = kTileBytes > kMergeBytes ? kTileBytes : kMergeBytes;
};

__device__ __forceinline__ bf16x8_t as_bf16x8(const vec16& v) {
    return __builtin_bit_cast(bf16x8_t, v);
}

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attend_mfma_kernel(
    const bf16_t* __restrict__ q_rot, int q_chunk0, int n_q_chunks,
    const bf16_t* __restrict__ k_res, const bf16_t* __restrict__ v_res, int64_t res_tokens,
    const int32_t* __restrict__ res_slot, const bf16_t* __restrict__ k_routed,
    const bf16_t* __restrict__ v_routed, const int32_t* __restrict__ group_idx,
    bf16_t* __restrict__ out, float* __restrict__ lse, int n_q_heads, int n_kv, int group,
    int keep_first, int window, int topk_groups, int wg_per_unit) {
    using S = Smem<D>;
    constexpr int KSTR = S::KSTR, VSTR = S::VSTR, NDT = S::NDT;
    constexpr int NKS = D / 16;                     // k-steps of Q.K^T
    constexpr int VPR = D / 8;                      // 16-byte vectors per row
    constexpr int KVEC = KT * VPR / kThreads;       // K vectors per thread per tile
    constexpr int VPAIR = (KT / 2) * VPR / kThreads;  // V row-pair vectors per thread

    __shared__ __align__(16) unsigned char smem[S::kBytes];
    __shared__ int s_gvalid[512];
    __shared__ int s_last;
    __shared__ int s_valid[KT];
    bf16_t* sK = reinterpret_cast<bf16_t*>(smem);
    bf16_t* sVt = sK + KT * KSTR;

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int half = lane >> 5, col = lane & 31;
    const int r = n_q_heads / n_kv;
    const int nqt = 2 * r;
    const int qt_per_wg = nqt < 4 ? nqt : 4;
    const int ksplit_n = 4 / qt_per_wg;
    const int part = blockIdx.x % wg_per_unit;
    const int i = blockIdx.x / wg_per_unit;
    const int bh = blockIdx.y;
    const int b = bh / n_kv, j = bh % n_kv;
    const int c = q_chunk0 + i;
    const int gpc = KT / group;
    const int qtile = part * 4 + wave % qt_per_wg;
    const int ksplit = wave / qt_per_wg;
    const bool qactive = qtile < nqt;
    const int64_t unit = static_cast<int64_t>(bh) * n_q_chunks + i;
    const int routed_rows = topk_groups * group;
    const int64_t res_chunks = res_tokens / KT;

    // routed slot validity and the last valid slot
    if (tid == 0) s_last = -1;
    __syncthreads();
    {
        const int32_t* gi = group_idx + unit * topk_groups;
        int last = -1;
        for (int s = tid; s < topk_groups; s += kThreads) {
            const int g = gi[s];
            const int ok = g >= 0 && g < c * gpc;
            s_gvalid[s] = ok;
            if (ok) last = s;
        }
        if (last >= 0) atomicMax(&s_last, last);
    }

    // this lane's query row and its Q fragments (B operand of S^T = K.Q^T)
    const int qrow_in_unit = qtile * 32 + col;
    const int hh = qrow_in_unit / KT, t = qrow_in_unit % KT;
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * KT;
    const int64_t qrow = (static_cast<int64_t>(b) * n_q_heads + j * r + (qactive ? hh : 0)) * qtok +
                         static_cast<int64_t>(i) * KT + t;
    bf16x8_t qf[NKS];
    if (qactive) {
#pragma unroll
        for (int kk = 0; kk < NKS; ++kk) qf[kk] = as_bf16x8(load16(q_rot + qrow * D + kk * 16 + half * 8));
    }
    __syncthreads();

    const VisibleChunks vis(c, keep_first, window);
    const int n_vis = vis.count;
    const int n_rt = s_last < 0 ? 0 : ((s_last + 1) * group + KT - 1) / KT;
    const int n_tiles = n_vis + n_rt + 1;

    const float scale = 1.4426950408889634f / sqrtf(static_cast<float>(D));  // log2(e)/sqrt(d)
    f32x16_t oacc[NDT];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[dt][e] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;
    bool bad = false;

    vec16 kreg[KVEC], vreg[2 * VPAIR];
    int row_limit = KT;

    // fetch tile `tile` into registers
    auto fetch = [&](int tile) {
        const bf16_t* kb;
        const bf16_t* vb;
        row_limit = KT;
        if (tile < n_vis || tile == n_tiles - 1) {
            const int cc = tile < n_vis ? vis.chunk(tile) : c;
            int64_t slot = res_slot ? res_slot[cc] : cc;
            if (slot < 0 || slot >= res_chunks) { bad = true; slot = 0; }
            const int64_t off = (static_cast<int64_t>(bh) * res_tokens + slot * KT) * D;
            kb = k_res + off;
            vb = v_res + off;
        } else {
            const int rt = tile - n_vis;
            const int64_t off = (unit * routed_rows + rt * KT) * D;
            kb = k_routed + off;
            vb = v_routed + off;
            row_limit = routed_rows - rt * KT < KT ? routed_rows - rt * KT : KT;
        }
#pragma unroll
        for (int u = 0; u < KVEC; ++u) {
            const int v = tid + kThreads * u;
            const int row = v / VPR, cv = v % VPR;
            kreg[u] = row < row_limit ? load16(kb + row * D + cv * 8) : vec16{{0u, 0u, 0u, 0u}};
        }
#pragma unroll
        for (int u = 0; u < VPAIR; ++u) {
            const int w = tid + kThreads * u;
            const int pr = w / VPR, cv = w % VPR;
            const int r0 = 2 * pr;
            vreg[2 * u] = r0 < row_limit ? load16(vb + r0 * D + cv * 8) : vec16{{0u, 0u, 0u, 0u}};
            vreg[2 * u + 1] =
                r0 + 1 < row_limit ? load16(vb + (r0 + 1) * D + cv * 8) : vec16{{0u, 0u, 0u, 0u}};
        }
    };

    fetch(0);
    for (int tile = 0; tile < n_tiles; ++tile) {
        const int kind = tile < n_vis ? kTileVisible : (tile == n_tiles - 1 ? kTileCurrent : kTileRouted);
        const int rt_row0 = (tile - n_vis) * KT;
        const int cur_limit = row_limit;
        __syncthreads();
#pragma unroll
        for (int u = 0; u < KVEC; ++u) {
            const int v = tid + kThreads * u;
            const int row = v / VPR, cv = v % VPR;
            *reinterpret_cast<vec16*>(sK + row * KSTR + cv * 8) = kreg[u];
        }
#pragma unroll
        for (int u = 0; u < VPAIR; ++u) {
            const int w = tid + kThreads * u;
            const int pr = w / VPR, cv = w % VPR;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t lo = (vreg[2 * u].w[e >> 1] >> ((e & 1) * 16)) & 0xffffu;
                const uint32_t hi = (vreg[2 * u + 1].w[e >> 1] >> ((e & 1) * 16)) & 0xffffu;
                *reinterpret_cast<uint32_t*>(sVt + (cv * 8 + e) * VSTR + 2 * pr) = lo | (hi << 16);
            }
        }
        if (tid < KT) {
            int ok = 1;
            if (kind == kTileRouted) {
                const int row = rt_row0 + tid;
                ok = tid < cur_limit && s_gvalid[row / group];
            }
            s_valid[tid] = ok;
        }
        __syncthreads();
        if (tile + 1 < n_tiles) fetch(tile + 1);

        if (qactive) {
            f32x16_t sacc[2];
            float tmax = -INFINITY;
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                if (ksplit_n == 2 && st != ksplit) continue;
#pragma unroll
                for (int e = 0; e < 16; ++e) sacc[st][e] = 0.f;
#pragma unroll
                for (int kk = 0; kk < NKS; ++kk) {
                    const bf16x8_t a = as_bf16x8(
                        *reinterpret_cast<const vec16*>(sK + (st * 32 + col) * KSTR + kk * 16 + half * 8));
                    sacc[st] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc[st], 0, 0, 0);
                }
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int key = st * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
                    const bool ok = kind == kTileCurrent ? key <= t : s_valid[key] != 0;
                    const float x = ok ? sacc[st][e] * scale : -INFINITY;
                    sacc[st][e] = x;
                    tmax = fmaxf(tmax, x);
                }
            }
            tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
            const float m_new = fmaxf(m_run, tmax);
            const float m_use = m_new == -INFINITY ? 0.f : m_new;
            const float alpha = exp2f(m_run - m_use);
            l_run *= alpha;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int e = 0; e < 16; ++e) oacc[dt][e] *= alpha;
            m_run = m_new;
#pragma unroll
            for (int st = 0; st < 2; ++st) {
                if (ksplit_n == 2 && st != ksplit) continue;
#pragma unroll
                for (int kap = 0; kap < 2; ++kap) {
                    bf16x8_t pf;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float pv = exp2f(sacc[st][kap * 8 + e] - m_use);
                        l_run += pv;
                        pf[e] = static_cast<__bf16>(pv);
                    }
                    const int kb = st * 32 + kap * 16 + half * 4;
#pragma unroll
                    for (int dt = 0; dt < NDT; ++dt) {
                        const bf16_t* vp = sVt + (dt * 32 + col) * VSTR + kb;
                        const bf16x4_t lo = *reinterpret_cast<const bf16x4_t*>(vp);
                        const bf16x4_t hi = *reinterpret_cast<const bf16x4_t*>(vp + 8);
                        const bf16x8_t a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf, oacc[dt], 0, 0, 0);
                    }
                }
            }
        }
    }

    float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    __syncthreads();  // LDS tiles are dead from here on
    if (ksplit_n == 2) {
        float* mg = reinterpret_cast<float*>(smem) + (wave % qt_per_wg) * 64 * (NDT * 16 + 2);
        float* mine = mg + lane * (NDT * 16 + 2);
        if (ksplit == 1) {
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int e = 0; e < 16; ++e) mine[dt * 16 + e] = oacc[dt][e];
            mine[NDT * 16] = m_run;
            mine[NDT * 16 + 1] = l_tot;
        }
        __syncthreads();
        if (ksplit == 0) {
            const float mb = mine[NDT * 16], lb = mine[NDT * 16 + 1];
            const float m = fmaxf(m_run, mb);
            const float mu = m == -INFINITY ? 0.f : m;
            const float fa = exp2f(m_run - mu), fb = exp2f(mb - mu);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int e = 0; e < 16; ++e) oacc[dt][e] = oacc[dt][e] * fa + mine[dt * 16 + e] * fb;
            l_tot = l_tot * fa + lb * fb;
            m_run = m;
        }
    }
    if (!qactive || ksplit != 0) return;

    const float inv = 1.0f / l_tot;
    bf16_t* orow = out + qrow * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = dt * 32 + g4 * 8 + half * 4;
            uint32_t w0, w1;
            if (bad) {
                w0 = w1 = 0x7fc07fc0u;
            } else {
                w0 = f32_to_bf16(oacc[dt][g4 * 4 + 0] * inv) |
                     (static_cast<uint32_t>(f32_to_bf16(oacc[dt][g4 * 4 + 1] * inv)) << 16);
                w1 = f32_to_bf16(oacc[dt][g4 * 4 + 2] * inv) |
                     (static_cast<uint32_t>(f32_to_bf16(oacc[dt][g4 * 4 + 3] * inv)) << 16);
            }
            *reinterpret_cast<uint2*>(orow + d0) = make_uint2(w0, w1);
        }
    if (lse && half == 0) lse[qrow] = bad ? NAN : (m_run + log2f(l_tot)) * 0.6931471805599453f;
}

}  // namespace

hipError_t launch_attend_mfma(const hga_plan& plan, const void* q_rot, int q_chunk0,
                              int n_q_chunks, const void* k_res, const void* v_res,
                              int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                              const void* v_routed, const int32_t* group_idx, void* out,
                              float* lse, hipStream_t stream) {
    const hga_params& p = plan.p;
    const int r = p.n_q_heads / p.n_kv_heads;
    const int nqt = 2 * r;
    const int wg_per_unit = nqt <= 2 ? 1 : (nqt + 3) / 4;
    dim3 grid(n_q_chunks * wg_per_unit, p.batch * p.n_kv_heads);
#define HGA_MFMA(DD)                                                                             \
    hipLaunchKernelGGL((attend_mfma_kernel<DD>), grid, dim3(kThreads), 0, stream,                \
                       static_cast<const bf16_t*>(q_rot), q_chunk0, n_q_chunks,                  \
                       static_cast<const bf16_t*>(k_res), static_cast<const bf16_t*>(v_res),     \
                       res_tokens, res_slot, static_cast<const bf16_t*>(k_routed),               \
                       static_cast<const bf16_t*>(v_routed), group_idx,                          \
                       static_cast<bf16_t*>(out), lse, p.n_q_heads, p.n_kv_heads, p.group,       \
                       p.keep_first, recent_window(p), p.topk_groups, wg_per_unit)
    if (p.head_dim == 64) HGA_MFMA(64); else HGA_MFMA(128);
#undef HGA_MFMA
    return hipGetLastError();
}

hipError_t launch_attend_valu(const hga_plan& plan, const void* q_rot, int q_chunk0,
                              int n_q_chunks, const void* k_res, const void* v_res,
                              int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                              const void* v_routed, const int32_t* group_idx, void* out,
                              float* lse, hipStream_t stream);

hipError_t launch_attend(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                         const void* k_res, const void* v_res, int64_t res_tokens,
                         const int32_t* res_slot, const void* k_routed, const void* v_routed,
                         const int32_t* group_idx, void* out, float* lse, hipStream_t stream) {
    if (plan.p.dtype == HGA_F32)
        return launch_attend_valu(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                  res_slot, k_routed, v_routed, group_idx, out, lse, stream);
    return launch_attend_mfma(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                              res_slot, k_routed, v_routed, group_idx, out, lse, stream);
}

}  // namespace hga
