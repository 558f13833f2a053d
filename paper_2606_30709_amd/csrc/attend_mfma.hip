// Exact-token attention (Sec. 3.4, Eq. (1)) for bf16 inputs on the gfx950
// matrix cores (v_mfma_f32_32x32x16_bf16), flash style.
//
// Work unit: one (batch, KV head, query chunk).  All r = Hq/Hkv query heads
// of the KV head share the unit's working set (GQA, Sec. 2), so their
// r*64 query rows are packed as 32-row query tiles; a workgroup of four
// wavefronts takes four query tiles (or, with only two tiles, two
// wavefronts per tile split each key tile between them and merge at the end).
//
// Keys stream through LDS in 64-key tiles: first the current chunk (under
// the causal mask), then the visible closed chunks, then the routed rows --
// an order whose first fetches depend on no index load.  Per tile and
// wavefront:
//   S^T[key][query] = K_tile . Q^T        (A = K rows from LDS, B = Q in VGPRs)
// so every lane owns one query column: the running max, running sum and the
// rescaling of the output are per-lane scalars, and a row maximum needs only
// one exchange with the lane holding the other half of the tile's keys.
//   O^T[d][query] += V^T . P^T            (A = V^T, B = P in VGPRs)
// P is rounded to bf16 for the product; statistics and accumulators are fp32.
// K and V are staged row-major; the V^T operand (eight keys at one head
// dimension per lane) comes from gfx950's LDS transpose read
// (ds_read_b64_tr_b16): within each 16-lane group, lane i receives element
// i%4 of the 64-bit reads issued by lanes 4j + i/4, j = 0..3, so 16 lanes
// pointing at 4 keys x 16 dimensions hand each lane 4 keys of one dimension.
// The next key tile is fetched into registers while the current one is in
// use (the template allows a deeper ring).  All global reads go through
// buffer descriptors: rows past a buffer's end read
// as zero without a branch, which keeps the wait counts exact.
#include <math.h>

#include "attend_common.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int KT = 64;  // keys per LDS tile (= chunk)
constexpr int kXcds = 8;

template <int D>
struct Smem {
    // K rows 16 B apart modulo 128 B: the 8 rows of one A-operand read phase
    // fall in distinct banks.  V rows 32 B apart modulo 128 B: the 4 rows of
    // one transpose-read group fall in distinct banks.
    static constexpr int KSTR = D + 8;
    static constexpr int VSTR = D + 16;
    static constexpr int kTileBytes = KT * (KSTR + VSTR) * 2;
    static constexpr int NDT = D / 32;
    // merge area: per query-tile slot and lane, the output accumulators, m and l
    static constexpr int kMergeBytes = 2 * 64 * (NDT * 16 + 2) * 4;
    static constexpr int kBytes = kTileBytes > kMergeBytes ? kTileBytes : kMergeBytes;
};

__device__ __forceinline__ bf16x8_t as_bf16x8(const vec16& v) {
    return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ i16x4_t lds_read_tr16(const bf16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4_t*)(reinterpret_cast<uintptr_t>(p)));
}

// D: head dim; KS: wavefronts sharing one query tile (each takes one 32-key
// half of every key tile); P: key tiles kept in flight in registers; NW:
// wavefronts per workgroup (NW / KS query tiles per workgroup).
template <int D, int KS, int P, int NW>
__global__ __launch_bounds__(NW * 64, 2) void attend_mfma_kernel(
    const bf16_t* __restrict__ q_rot, int q_chunk0, int n_q_chunks,
    const bf16_t* __restrict__ k_res, const bf16_t* __restrict__ v_res, int64_t res_tokens,
    const int32_t* __restrict__ res_slot, const bf16_t* __restrict__ k_routed,
    const bf16_t* __restrict__ v_routed, const int32_t* __restrict__ group_idx,
    bf16_t* __restrict__ out, float* __restrict__ lse, int n_q_heads, int n_kv, int group_shift,
    int keep_first, int window, int topk_groups, int wg_per_unit, int n_blocks) {
    using S = Smem<D>;
    constexpr int KSTR = S::KSTR, VSTR = S::VSTR, NDT = S::NDT;
    constexpr int NKS = D / 16;                  // k-steps of Q.K^T
    constexpr int VPR = D / 8;                   // 16-byte vectors per row
    constexpr int kThreads = NW * 64;
    constexpr int NVEC = KT * VPR / kThreads;    // K (and V) vectors per thread per tile
    constexpr int QT = NW / KS;                  // query tiles per workgroup
    constexpr int NST = 2 / KS;                  // 32-key sub-tiles per wave per tile
    constexpr uint32_t kRowBytes = D * 2;

    __shared__ __align__(16) unsigned char smem[S::kBytes];
    __shared__ int s_gvalid[512];
    bf16_t* sK = reinterpret_cast<bf16_t*>(smem);
    bf16_t* sV = sK + KT * KSTR;

    // XCD-aware order: consecutive workgroups of one XCD take consecutive
    // (head, chunk) units, so a unit's previous chunk and the head's sink
    // chunks are still in that XCD's L2.
    const int per_xcd = (n_blocks + kXcds - 1) / kXcds;
    const int logical = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (logical >= n_blocks) return;
    const int part = logical % wg_per_unit;
    const int i = (logical / wg_per_unit) % n_q_chunks;
    const int bh = logical / wg_per_unit / n_q_chunks;

    const int tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int half = lane >> 5, col = lane & 31;
    const int r = n_q_heads / n_kv;
    const int nqt = 2 * r;
    const int b = bh / n_kv, j = bh % n_kv;
    const int c = q_chunk0 + i;
    const int group = 1 << group_shift;
    const int gpc = KT >> group_shift;
    const int qtile = part * QT + wave % QT;
    const int ksplit = wave / QT;
    const bool qactive = qtile < nqt;
    const int64_t unit = static_cast<int64_t>(bh) * n_q_chunks + i;
    const int routed_rows = topk_groups * group;
    const int64_t res_chunks = res_tokens / KT;

    // One descriptor per source: this head's resident K/V and this unit's
    // routed K/V.  Offsets are 32-bit within each.
    const buf_rsrc rk_res = make_rsrc(k_res + static_cast<int64_t>(bh) * res_tokens * D,
                                      static_cast<uint32_t>(res_chunks * KT * kRowBytes));
    const buf_rsrc rv_res = make_rsrc(v_res + static_cast<int64_t>(bh) * res_tokens * D,
                                      static_cast<uint32_t>(res_chunks * KT * kRowBytes));
    const buf_rsrc rk_rt = make_rsrc(k_routed + unit * routed_rows * D, routed_rows * kRowBytes);
    const buf_rsrc rv_rt = make_rsrc(v_routed + unit * routed_rows * D, routed_rows * kRowBytes);

    // group ids first: their validity is needed only when routed tiles are staged
    const buf_rsrc g_rsrc = make_rsrc(group_idx + unit * topk_groups, topk_groups * 4);
    constexpr int NG = 512 / kThreads;           // group-id slots per thread
    int gval[NG];
#pragma unroll
    for (int u = 0; u < NG; ++u) gval[u] = buf_load_i32(g_rsrc, (tid + kThreads * u) * 4);

    // this lane's query row and its Q fragments (B operand of S^T = K.Q^T)
    const int qrow_in_unit = qtile * 32 + col;
    const int hh = qrow_in_unit / KT, t = qrow_in_unit % KT;
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * KT;
    const int64_t qrow = (static_cast<int64_t>(b) * n_q_heads + j * r + (qactive ? hh : 0)) * qtok +
                         static_cast<int64_t>(i) * KT + t;
    // uniform descriptor over the r heads of this KV head; inactive lanes read zeros
    const int64_t q_head0 = (static_cast<int64_t>(b) * n_q_heads + j * r) * qtok;
    const buf_rsrc q_rsrc = make_rsrc(q_rot + q_head0 * D, static_cast<uint32_t>(r * qtok * kRowBytes));
    const uint32_t q_off = qactive ? static_cast<uint32_t>((qrow - q_head0) * kRowBytes)
                                   : 0xffffffffu - 0xffffu;
    bf16x8_t qf[NKS];
#pragma unroll
    for (int kk = 0; kk < NKS; ++kk)
        qf[kk] = as_bf16x8(buf_load16(q_rsrc, q_off + (kk * 16 + half * 8) * 2));

    // tile order: the current chunk, the visible closed chunks, the routed rows
    const VisibleChunks vis(c, keep_first, window);
    const int n_vis = vis.count;
    const int n_rt = (routed_rows + KT - 1) / KT;
    const int n_tiles = 1 + n_vis + n_rt;
    bool bad = false;

    // per-thread byte offset of its vectors inside a 64-row tile
    uint32_t voff[NVEC];
#pragma unroll
    for (int u = 0; u < NVEC; ++u) {
        const int v = tid + kThreads * u;
        voff[u] = (v / VPR) * kRowBytes + (v % VPR) * 16;
    }

    vec16 kreg[P][NVEC], vreg[P][NVEC];
    // Stage tile `tile` in registers; a tile past the end reads as zeros.
    auto fetch = [&](int tile, vec16 (&kr)[NVEC], vec16 (&vr)[NVEC]) {
        bool routed = false;
        uint32_t base = 0xffffffffu - 0xffffu;  // past every buffer: zeros
        if (tile < n_tiles) {
            if (tile <= n_vis) {
                const int cc = tile == 0 ? c : vis.chunk(tile - 1);
                int64_t slot = res_slot ? res_slot[cc] : cc;
                if (slot < 0 || slot >= res_chunks) { bad = true; slot = 0; }
                base = static_cast<uint32_t>(slot * KT * kRowBytes);
            } else {
                routed = true;
                base = static_cast<uint32_t>((tile - 1 - n_vis) * KT * kRowBytes);
            }
        }
        const buf_rsrc rk = routed ? rk_rt : rk_res;
        const buf_rsrc rv = routed ? rv_rt : rv_res;
#pragma unroll
        for (int u = 0; u < NVEC; ++u) {
            kr[u] = buf_load16(rk, base + voff[u]);
            vr[u] = buf_load16(rv, base + voff[u]);
        }
    };

#pragma unroll
    for (int s = 0; s < P; ++s) fetch(s, kreg[s], vreg[s]);

#pragma unroll
    for (int u = 0; u < NG; ++u) {
        const int slot = tid + kThreads * u;
        if (slot < topk_groups) s_gvalid[slot] = gval[u] >= 0 && gval[u] < c * gpc;
    }


    const float scale = 1.4426950408889634f / sqrtf(static_cast<float>(D));  // log2(e)/sqrt(d)
    f32x16_t oacc[NDT];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[dt][e] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;  // m_run in scaled (log2) units

    for (int base = 0; base < n_tiles; base += P) {
#pragma unroll
        for (int s = 0; s < P; ++s) {
            const int tile = base + s;
            if (tile >= n_tiles) break;
            const int kind = tile == 0 ? kTileCurrent : (tile <= n_vis ? kTileVisible : kTileRouted);
            const int rt_row0 = (tile - 1 - n_vis) * KT;
            __syncthreads();
#pragma unroll
            for (int u = 0; u < NVEC; ++u) {
                const int v = tid + kThreads * u;
                const int row = v / VPR, cv = v % VPR;
                *reinterpret_cast<vec16*>(sK + row * KSTR + cv * 8) = kreg[s][u];
                *reinterpret_cast<vec16*>(sV + row * VSTR + cv * 8) = vreg[s][u];
            }
            __syncthreads();
            fetch(tile + P, kreg[s], vreg[s]);

            // rows that must be masked in a routed tile: past the buffer or of an invalid slot
            bool partial = false;
            if (kind == kTileRouted) {
                partial = rt_row0 + KT > routed_rows;
                for (int g = rt_row0 >> group_shift; g < (rt_row0 + KT) >> group_shift && g < topk_groups; ++g)
                    partial |= s_gvalid[g] == 0;
            }

            if (qactive) {
                f32x16_t sacc[NST];
                float tmax = -INFINITY;
#pragma unroll
                for (int n = 0; n < NST; ++n) {
                    const int st = KS == 2 ? ksplit : n;
#pragma unroll
                    for (int e = 0; e < 16; ++e) sacc[n][e] = 0.f;
#pragma unroll
                    for (int kk = 0; kk < NKS; ++kk) {
                        const bf16x8_t a = as_bf16x8(*reinterpret_cast<const vec16*>(
                            sK + (st * 32 + col) * KSTR + kk * 16 + half * 8));
                        sacc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], sacc[n], 0, 0, 0);
                    }
                    if (kind == kTileCurrent) {
#pragma unroll
                        for (int e = 0; e < 16; ++e) {
                            const int key = st * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
                            sacc[n][e] = key > t ? -INFINITY : sacc[n][e];
                        }
                    } else if (partial) {
#pragma unroll
                        for (int e = 0; e < 16; ++e) {
                            const int row = rt_row0 + st * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
                            const int slot = min(row >> group_shift, topk_groups - 1);
                            const bool ok = row < routed_rows && s_gvalid[slot] != 0;
                            sacc[n][e] = ok ? sacc[n][e] : -INFINITY;
                        }
                    }
#pragma unroll
                    for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, sacc[n][e]);
                }
                tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64)) * scale;
                const float m_new = fmaxf(m_run, tmax);
                const float m_use = m_new == -INFINITY ? 0.f : m_new;
                const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
                l_run *= alpha;
#pragma unroll
                for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                    for (int e = 0; e < 16; ++e) oacc[dt][e] *= alpha;
                m_run = m_new;
#pragma unroll
                for (int n = 0; n < NST; ++n) {
                    const int st = KS == 2 ? ksplit : n;
#pragma unroll
                    for (int kap = 0; kap < 2; ++kap) {
                        bf16x8_t pf;
#pragma unroll
                        for (int e = 0; e < 8; ++e) {
                            const float pv =
                                __builtin_amdgcn_exp2f(fmaf(sacc[n][kap * 8 + e], scale, -m_use));
                            l_run += pv;
                            pf[e] = static_cast<__bf16>(pv);
                        }
                        // V^T operand: keys st*32 + kap*16 + {half*4 + 0..3, 8 + half*4 + 0..3}
                        // at dimension dt*32 + col; each 16-lane group points at
                        // 4 keys x 16 dimensions.
                        const int key0 = st * 32 + kap * 16 + half * 4 + ((lane & 15) >> 2);
                        const int dcol = ((lane >> 4) & 1) * 16 + (lane & 3) * 4;
#pragma unroll
                        for (int dt = 0; dt < NDT; ++dt) {
                            const bf16_t* vp = sV + key0 * VSTR + dt * 32 + dcol;
                            const i16x4_t lo = lds_read_tr16(vp);
                            const i16x4_t hi = lds_read_tr16(vp + 8 * VSTR);
                            const bf16x8_t a = __builtin_bit_cast(
                                bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                            oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf, oacc[dt], 0, 0, 0);
                        }
                    }
                }
            }
        }
    }

    float l_tot = l_run + __shfl_xor(l_run, 32, 64);
    __syncthreads();  // LDS tiles are dead from here on
    if (KS == 2) {
        float* mine = reinterpret_cast<float*>(smem) + ((wave % QT) * 64 + lane) * (NDT * 16 + 2);
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
            const float fa = __builtin_amdgcn_exp2f(m_run - mu), fb = __builtin_amdgcn_exp2f(mb - mu);
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int e = 0; e < 16; ++e) oacc[dt][e] = oacc[dt][e] * fa + mine[dt * 16 + e] * fb;
            l_tot = l_tot * fa + lb * fb;
            m_run = m;
        }
    }
    if (!qactive || ksplit != 0) return;

    const float inv = bad ? NAN : 1.0f / l_tot;
    bf16_t* orow = out + qrow * D;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = dt * 32 + g4 * 8 + half * 4;
            typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
            bf16x4_t o;
#pragma unroll
            for (int e = 0; e < 4; ++e) o[e] = static_cast<__bf16>(oacc[dt][g4 * 4 + e] * inv);
            *reinterpret_cast<bf16x4_t*>(orow + d0) = o;
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
    // One head per KV head (two query tiles): a workgroup of two wavefronts,
    // each with every key of its tile; otherwise four query tiles per group.
    const bool one_head = nqt <= 2;
    const int wg_per_unit = one_head ? 1 : (nqt + 3) / 4;
    const int64_t n_blocks64 =
        static_cast<int64_t>(p.batch) * p.n_kv_heads * n_q_chunks * wg_per_unit;
    if (n_blocks64 > (int64_t(1) << 30)) return hipErrorInvalidConfiguration;
    const int n_blocks = static_cast<int>(n_blocks64);
    const int grid = (n_blocks + kXcds - 1) / kXcds * kXcds;
    const int group_shift = p.group == 8 ? 3 : (p.group == 16 ? 4 : 5);
#define HGA_MFMA(DD, KSV, PV, NWV)                                                               \
    hipLaunchKernelGGL((attend_mfma_kernel<DD, KSV, PV, NWV>), dim3(grid), dim3(NWV * 64), 0,    \
                       stream, static_cast<const bf16_t*>(q_rot), q_chunk0, n_q_chunks,          \
                       static_cast<const bf16_t*>(k_res), static_cast<const bf16_t*>(v_res),     \
                       res_tokens, res_slot, static_cast<const bf16_t*>(k_routed),               \
                       static_cast<const bf16_t*>(v_routed), group_idx,                          \
                       static_cast<bf16_t*>(out), lse, p.n_q_heads, p.n_kv_heads, group_shift,   \
                       p.keep_first, recent_window(p), p.topk_groups, wg_per_unit, n_blocks)
    // One tile in flight per workgroup: measured faster than deeper register
    // rings, whose extra VGPRs cost more occupancy than they hide latency.
    if (p.head_dim == 64) {
        if (one_head) HGA_MFMA(64, 2, 1, 4); else HGA_MFMA(64, 1, 1, 4);
    } else {
        if (one_head) HGA_MFMA(128, 2, 1, 4); else HGA_MFMA(128, 1, 1, 4);
    }
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
