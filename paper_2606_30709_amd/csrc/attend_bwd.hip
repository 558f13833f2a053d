// Backward of the exact-token attention (Sec. 3.4, Eq. (1)) for bf16 inputs
// on the gfx950 matrix cores (v_mfma_f32_32x32x16_bf16).  Routing is not
// differentiated: the unit's working set (current chunk under the causal
// mask, visible chunks, routed groups) is the forward's.  For query row i and
// working-set key x, with s = q.k/sqrt(d), p = exp(s - lse_i) (the forward's
// log-sum-exp), D_i = dout_i . out_i:
//   dp = dout_i . v_x,  ds = p (dp - D_i),
//   dq_i = sum_x ds k_x / sqrt(d),  dk_x += sum_i ds q_i / sqrt(d),
//   dv_x += sum_i p dout_i.
// Routed rows are resident rows (group g, row o -> token g*G + o), so their
// key/value gradients land on those rows.
//
// Work item: (unit, part): a workgroup of NW wavefronts takes NW query tiles
// of 32 rows of the unit's r*64 (as the forward packs them).  Per 64-key tile
// the workgroup stages K and V row-major and K transposed in LDS; per 32-key
// sub-tile each wavefront computes, for its own 32 queries,
//   S^T = K.Q^T and dP^T = V.dO^T   (B operands: the wave's Q, dO rows in LDS),
//   P^T, dS^T elementwise           (each lane owns one query column),
//   dQ += dS.K                      (A = the lane's own dS values, in registers),
// and writes dS^T and P^T to its LDS scratch.  The key gradients of the
// sub-tile sum over every query of the workgroup, so after one barrier the
// 2*D/32 blocks (dK or dV, 32 dimensions) are split among the wavefronts:
// each contracts the scratch of all wavefronts against Q^T / dO^T fragments
// it gathered into registers once, and adds its blocks into the global fp32
// dk, dv with hardware atomics (other units share visible chunks and routed
// groups).  No two wavefronts accumulate into the same LDS words.
//
// A product's contraction index may be permuted as long as both operands use
// the same permutation: dQ's A operand is the lane's own dS^T column (keys in
// the order of the accumulator layout) and its B operand reads K^T in that
// same key order.
#include <hip/hip_runtime.h>
#include <math.h>

#include "attend_common.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int KT = 64;    // keys per tile (= chunk)
constexpr int SCR = 40;   // row stride (bf16) of the 32 x 32 scratch tiles

template <int D, int NW>
struct BwdLayout {
    static constexpr int KS = D + 8;        // row stride (bf16) of K, V, Q, dO tiles
    static constexpr int TS = KT + 4;       // row stride (bf16) of the K^T tile
    static constexpr int kK = 0;
    static constexpr int kV = kK + KT * KS * 2;
    static constexpr int kKT = kV + KT * KS * 2;
    static constexpr int kQ = kKT + D * TS * 2;                  // NW x (Q, dO) rows
    static constexpr int kScr = kQ + NW * 2 * 32 * KS * 2;       // NW x 2 buffers x (dS^T, P^T)
    static constexpr int kTok = kScr + NW * 4 * 32 * SCR * 2;    // 2 x (tile row -> token)
    static constexpr int kGid = kTok + 2 * KT * 4;
    static constexpr int kBytes = kGid + kMaxTopK * 4;
};

__device__ __forceinline__ bf16x8_t frag(const bf16_t* p) {
    return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const vec16*>(p));
}

__device__ __forceinline__ bf16x4_t frag4(const bf16_t* p) {
    return *reinterpret_cast<const bf16x4_t*>(p);
}

__device__ __forceinline__ float add_halves(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup barrier that orders LDS only: waits for this wave's LDS
// operations, not for its global atomics (which nothing here reads back).
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(1, 1))) void attend_bwd_kernel(
    const bf16_t* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const bf16_t* __restrict__ k_res,
    const bf16_t* __restrict__ v_res, int64_t res_tokens, const int32_t* __restrict__ group_idx,
    const bf16_t* __restrict__ out, const float* __restrict__ lse,
    const bf16_t* __restrict__ dout, float* __restrict__ dq, float* __restrict__ dk,
    float* __restrict__ dv, int r, int n_kv, int group_shift, int keep_first, int window,
    int topk_groups, int wg_per_unit, int n_items) {
    using Lay = BwdLayout<D, NW>;
    constexpr int NKS = D / 16;   // 16-wide k-steps over d
    constexpr int NDT = D / 32;   // 32-wide blocks of d
    constexpr int VPR = D / 8;    // 16-byte vectors per row
    constexpr int IPW = 2 * NDT / NW;  // key-gradient blocks per wave
    static_assert(IPW >= 1 && IPW * NW == 2 * NDT, "blocks must split evenly");
    extern __shared__ __align__(16) unsigned char smem[];
    bf16_t* sK = reinterpret_cast<bf16_t*>(smem + Lay::kK);
    bf16_t* sV = reinterpret_cast<bf16_t*>(smem + Lay::kV);
    bf16_t* sKT = reinterpret_cast<bf16_t*>(smem + Lay::kKT);
    bf16_t* sQall = reinterpret_cast<bf16_t*>(smem + Lay::kQ);
    bf16_t* scr_all = reinterpret_cast<bf16_t*>(smem + Lay::kScr);
    int* s_tok_all = reinterpret_cast<int*>(smem + Lay::kTok);
    int* s_gid = reinterpret_cast<int*>(smem + Lay::kGid);

    const int item = blockIdx.x;
    if (item >= n_items) return;
    const int unit = item / wg_per_unit, part = item % wg_per_unit;
    const int bh = unit / n_q_chunks, i = unit % n_q_chunks;
    const int b = bh / n_kv, j = bh % n_kv;
    const int c = q_chunk0 + i;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, col = lane & 31;
    const int group = 1 << group_shift, gpc = KT >> group_shift;
    const int nqt = 2 * r;
    const int qtile = part * NW + wave;
    const bool qactive = qtile < nqt;
    // query tiles of this workgroup that hold queries (a prefix of its waves)
    const int nqa = min(NW, nqt - part * NW);
    const int routed_rows = topk_groups * group;
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * KT;
    const int n_q_heads = r * n_kv;
    // global row of the wave's local query m (0 .. 31)
    auto qrow_of = [&](int m) {
        const int row = (qactive ? qtile : 0) * 32 + m;
        return (static_cast<int64_t>(b) * n_q_heads + j * r + row / KT) * qtok +
               static_cast<int64_t>(i) * KT + row % KT;
    };
    const int t = (qtile * 32 + col) % KT;  // this lane's query token in the chunk
    const int64_t my_row = qrow_of(col);
    const float scale2 = 1.4426950408889634f / sqrtf(static_cast<float>(D));
    const float inv_sqrt_d = 1.0f / sqrtf(static_cast<float>(D));

    for (int s = tid; s < topk_groups; s += NW * 64)
        s_gid[s] = group_idx[static_cast<int64_t>(unit) * topk_groups + s];

    // The wave's 32 rows of Q and dO stay in LDS, row-major: the B fragments
    // of S^T = K.Q^T and dP^T = V.dO^T are 16-byte row reads.
    bf16_t* sQ = sQall + wave * 2 * 32 * Lay::KS;
    bf16_t* sG = sQ + 32 * Lay::KS;
    float dsum = 0.f, lse2 = 0.f;
    if (qactive) {
        const bf16_t* qp = q_rot + my_row * D;
        const bf16_t* gp = dout + my_row * D;
        const bf16_t* op = out + my_row * D;
        float acc = 0.f;  // D_i = dout_i . out_i over this lane's half of d
#pragma unroll
        for (int kk = 0; kk < NKS; ++kk) {
            const bf16x8_t q8 = frag(qp + kk * 16 + half * 8);
            const bf16x8_t g8 = frag(gp + kk * 16 + half * 8);
            const bf16x8_t o8 = frag(op + kk * 16 + half * 8);
            *reinterpret_cast<bf16x8_t*>(sQ + col * Lay::KS + kk * 16 + half * 8) = q8;
            *reinterpret_cast<bf16x8_t*>(sG + col * Lay::KS + kk * 16 + half * 8) = g8;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                acc = fmaf(static_cast<float>(g8[e]), static_cast<float>(o8[e]), acc);
        }
        dsum = add_halves(acc);
        lse2 = lse[my_row] * 1.4426950408889634f;
    }
    lds_barrier();

    // Key-gradient block u of this wave: kind (0: dK from dS^T and Q, 1: dV
    // from P^T and dO) and 32-dimension block nb.  With NW even the kind is
    // the wave's parity.  xt[u][q][ks]: B fragment of X^T over query tile q
    // (the workgroup's q-th), k-step ks: lane holds X[ks*16 + half*8 + e][nb*32 + col].
    const int kind = wave & 1;
    bf16x8_t xt[IPW][NW][2];
#pragma unroll
    for (int u = 0; u < IPW; ++u) {
        const int nb = (wave + NW * u) >> 1;
#pragma unroll
        for (int q = 0; q < NW; ++q) {
            const bf16_t* src = sQall + (q * 2 + kind) * 32 * Lay::KS + nb * 32 + col;
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    xt[u][q][ks][e] = q < nqa ? __builtin_bit_cast(
                                                    __bf16, src[(ks * 16 + half * 8 + e) * Lay::KS])
                                              : static_cast<__bf16>(0.f);
        }
    }

    f32x16_t dqacc[NDT];
#pragma unroll
    for (int nb = 0; nb < NDT; ++nb)
#pragma unroll
        for (int e = 0; e < 16; ++e) dqacc[nb][e] = 0.f;

    const VisibleChunks vis(c, keep_first, window);
    const int n_vis = vis.count;
    const int n_rt = (routed_rows + KT - 1) / KT;
    const int n_tiles = 1 + n_vis + n_rt;
    const bf16_t* kbase = k_res + static_cast<int64_t>(bh) * res_tokens * D;
    const bf16_t* vbase = v_res + static_cast<int64_t>(bh) * res_tokens * D;
    float* gbase = (kind ? dv : dk) + static_cast<int64_t>(bh) * res_tokens * D;
    const float gscale = kind ? 1.f : inv_sqrt_d;
    const int lim = c * gpc;  // routed groups must lie in the causal past

    // scratch of wave w, buffer x: dS^T then P^T, each [key][query]
    auto scratch = [&](int w, int x) { return scr_all + (w * 2 + x) * 2 * 32 * SCR; };

    for (int tile = 0; tile < n_tiles; ++tile) {
        // Stage K, V row-major and K transposed; the token of each tile row
        // (-1: a routed row to skip, staged as zeros) goes to the token table
        // of the tile's parity.  Every wave has passed the previous tile's
        // last barrier, after which only the token table of that tile's
        // parity and the scratch are read.  Thread (row, part) issues all its
        // vectors of the row at once; consecutive threads take consecutive
        // rows, so the transposed writes are consecutive too.
        int* s_tok = s_tok_all + (tile & 1) * KT;
        {
            constexpr int TPR = NW * 64 / KT;  // threads per row
            constexpr int VPT = VPR / TPR;     // vectors per thread
            const int row = tid % KT, pv = tid / KT;
            int tok;
            if (tile <= n_vis) {
                tok = (tile == 0 ? c : vis.chunk(tile - 1)) * KT + row;
            } else {
                const int rr = (tile - 1 - n_vis) * KT + row;
                const int g = rr < routed_rows ? s_gid[rr >> group_shift] : -1;
                tok = g >= 0 && g < lim ? g * group + (rr & (group - 1)) : -1;
            }
            if (pv == 0) s_tok[row] = tok;
            vec16 kx[VPT], vx[VPT];
#pragma unroll
            for (int u = 0; u < VPT; ++u) {
                const int cv = pv * VPT + u;
                kx[u] = vec16{{0u, 0u, 0u, 0u}};
                vx[u] = kx[u];
                if (tok >= 0) {
                    kx[u] = load16(kbase + static_cast<int64_t>(tok) * D + cv * 8);
                    vx[u] = load16(vbase + static_cast<int64_t>(tok) * D + cv * 8);
                }
            }
#pragma unroll
            for (int u = 0; u < VPT; ++u) {
                const int cv = pv * VPT + u;
                *reinterpret_cast<vec16*>(sK + row * Lay::KS + cv * 8) = kx[u];
                *reinterpret_cast<vec16*>(sV + row * Lay::KS + cv * 8) = vx[u];
                const bf16_t* ke = reinterpret_cast<const bf16_t*>(&kx[u]);
#pragma unroll
                for (int e = 0; e < 8; ++e) sKT[(cv * 8 + e) * Lay::TS + row] = ke[e];
            }
        }
        lds_barrier();
        const bool current = tile == 0;
        for (int st = 0; st < 2; ++st) {
            if (qactive) {
                // S^T and dP^T of the 32-key sub-tile st
                f32x16_t sacc, pacc;
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    sacc[e] = 0.f;
                    pacc[e] = 0.f;
                }
                const int krow = st * 32 + col;
#pragma unroll
                for (int kk = 0; kk < NKS; ++kk) {
                    const int off = kk * 16 + half * 8;
                    sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        frag(sK + krow * Lay::KS + off), frag(sQ + col * Lay::KS + off), sacc, 0, 0, 0);
                    pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        frag(sV + krow * Lay::KS + off), frag(sG + col * Lay::KS + off), pacc, 0, 0, 0);
                }
                // P^T, dS^T: lane (half, col) holds keys st*32 + kl, kl below;
                // element e of fragment kap is e' = kap*8 + e of the accumulator
                bf16_t* s_dst = scratch(wave, st);
                bf16_t* s_pt = s_dst + 32 * SCR;
                bf16x8_t dsf[2];
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int kl = (e >> 2) * 8 + half * 4 + (e & 3);
                    const int key = st * 32 + kl;
                    const bool ok = s_tok[key] >= 0 && (!current || key <= t);
                    const float p = ok ? __builtin_amdgcn_exp2f(sacc[e] * scale2 - lse2) : 0.f;
                    const float ds = p * (pacc[e] - dsum);
                    const __bf16 db = static_cast<__bf16>(ds);
                    dsf[e >> 3][e & 7] = db;
                    s_dst[kl * SCR + col] = __builtin_bit_cast(bf16_t, db);
                    s_pt[kl * SCR + col] = __builtin_bit_cast(bf16_t, static_cast<__bf16>(p));
                }
                // dQ += dS.K: k-slot half*8 + e of fragment kap is key
                // st*32 + kap*16 + (e/4)*8 + half*4 + e%4, so the B operand
                // is two 4-key runs of the K^T row of dimension nb*32 + col.
#pragma unroll
                for (int kap = 0; kap < 2; ++kap)
#pragma unroll
                    for (int nb = 0; nb < NDT; ++nb) {
                        const bf16_t* kp = sKT + (nb * 32 + col) * Lay::TS + st * 32 + kap * 16 + half * 4;
                        const bf16x4_t lo = frag4(kp), hi = frag4(kp + 8);
                        const bf16x8_t bf = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                        dqacc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(dsf[kap], bf, dqacc[nb], 0, 0, 0);
                    }
            }
            lds_barrier();  // every wave's dS^T, P^T of sub-tile st are in LDS
            // This wave's key-gradient blocks over the workgroup's queries:
            // A = dS^T or P^T [key][query] of query tile q, B = xt.
#pragma unroll
            for (int u = 0; u < IPW; ++u) {
                const int nb = (wave + NW * u) >> 1;
                f32x16_t acc;
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[e] = 0.f;
#pragma unroll
                for (int q = 0; q < NW; ++q) {
                    if (q < nqa) {
                        const bf16_t* a = scratch(q, st) + kind * 32 * SCR + col * SCR + half * 8;
#pragma unroll
                        for (int ks = 0; ks < 2; ++ks)
                            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(a + ks * 16), xt[u][q][ks],
                                                                          acc, 0, 0, 0);
                    }
                }
                // acc[e]: key st*32 + (e/4)*8 + half*4 + e%4, dimension nb*32 + col
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int tok = s_tok[st * 32 + (e >> 2) * 8 + half * 4 + (e & 3)];
                    if (tok >= 0)
                        unsafeAtomicAdd(gbase + static_cast<int64_t>(tok) * D + nb * 32 + col,
                                        acc[e] * gscale);
                }
            }
        }
    }

    // dq: C layout [m = query][n = d]: lane column d = nb*32 + col, rows m
    if (qactive) {
#pragma unroll
        for (int nb = 0; nb < NDT; ++nb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int m = (e >> 2) * 8 + half * 4 + (e & 3);
                dq[qrow_of(m) * D + nb * 32 + col] = dqacc[nb][e] * inv_sqrt_d;
            }
    }
}

template <int D, int NW>
hipError_t launch_bwd_t(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                        const void* k_res, const void* v_res, int64_t res_tokens,
                        const int32_t* group_idx, const void* out, const float* lse,
                        const void* dout, float* dq, float* dk, float* dv, hipStream_t stream) {
    const hga_params& p = plan.p;
    constexpr int kLds = BwdLayout<D, NW>::kBytes;
    static bool configured = false;
    if (!configured) {
        const hipError_t e = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&attend_bwd_kernel<D, NW>),
            hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
        if (e != hipSuccess) return e;
        configured = true;
    }
    const int r = p.n_q_heads / p.n_kv_heads;
    const int wg_per_unit = (2 * r + NW - 1) / NW;
    const int64_t items = static_cast<int64_t>(p.batch) * p.n_kv_heads * n_q_chunks * wg_per_unit;
    if (items > (int64_t(1) << 30)) return hipErrorInvalidConfiguration;
    const int group_shift = p.group == 8 ? 3 : (p.group == 16 ? 4 : 5);
    hipLaunchKernelGGL((attend_bwd_kernel<D, NW>), dim3(static_cast<unsigned>(items)),
                       dim3(NW * 64), kLds, stream, static_cast<const bf16_t*>(q_rot), q_chunk0,
                       n_q_chunks, static_cast<const bf16_t*>(k_res),
                       static_cast<const bf16_t*>(v_res), res_tokens, group_idx,
                       static_cast<const bf16_t*>(out), lse, static_cast<const bf16_t*>(dout), dq,
                       dk, dv, r, p.n_kv_heads, group_shift, p.keep_first, recent_window(p),
                       p.topk_groups, wg_per_unit, static_cast<int>(items));
    return hipGetLastError();
}

}  // namespace

// Wavefronts per workgroup: four query tiles at d64 (two with one head per
// KV head, which has only two), two at d128 (the LDS budget).
size_t attend_backward_lds_bytes(const hga_plan& plan) {
    const int r = plan.p.n_q_heads / plan.p.n_kv_heads;
    if (plan.p.head_dim == 64)
        return r == 1 ? BwdLayout<64, 2>::kBytes : BwdLayout<64, 4>::kBytes;
    return BwdLayout<128, 2>::kBytes;
}

hipError_t launch_attend_backward(const hga_plan& plan, const void* q_rot, int q_chunk0,
                                  int n_q_chunks, const void* k_res, const void* v_res,
                                  int64_t res_tokens, const int32_t* group_idx, const void* out,
                                  const float* lse, const void* dout, float* dq, float* dk,
                                  float* dv, hipStream_t stream) {
    const hga_params& p = plan.p;
    const int r = p.n_q_heads / p.n_kv_heads;
#define HGA_BWD(DD, NN)                                                                         \
    return launch_bwd_t<DD, NN>(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,   \
                                group_idx, out, lse, dout, dq, dk, dv, stream)
    if (p.head_dim == 64) {
        if (r == 1) HGA_BWD(64, 2);
        HGA_BWD(64, 4);
    }
    HGA_BWD(128, 2);
#undef HGA_BWD
}

}  // namespace hga
