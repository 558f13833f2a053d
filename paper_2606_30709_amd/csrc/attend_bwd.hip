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
// Two forms.  The fused kernel serves units whose r*64 query rows fit one
// workgroup (r <= 2 at d = 64, r = 1 at d = 128); larger GQA groups take the
// split pair further below (dQ query-major, dK and dV key-major).
//
// Fused work item: (unit, part): a workgroup of NW wavefronts takes NW query
// tiles of 32 rows of the unit's r*64 (as the forward packs them).  Per 64-key tile
// the workgroup stages K and V row-major in LDS; per 32-key sub-tile each
// wavefront computes, for its own 32 queries,
//   S^T = K.Q^T and dP^T = V.dO^T   (B operands: the wave's Q, dO rows, read
//                                    from LDS into registers once),
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
// the order of the accumulator layout) and its B operand takes K^T in that
// same key order, by transpose reads of the row-major K tile (k_tr4).
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
    static constexpr int kK = 0;
    static constexpr int kV = kK + KT * KS * 2;
    static constexpr int kQ = kV + KT * KS * 2;                  // NW x (Q, dO) rows
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

typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

// Four keys of one dimension from a row-major K tile in LDS (row stride ks
// elements), by gfx950's transpose read ds_read_b64_tr_b16: within each
// 16-lane group, lane i receives element i%4 of the 8-byte reads of lanes
// 4j + i/4, j = 0..3.  Lane r of the group reads row k0 + r/4, dimensions
// d0 + 16*(group & 1) + 4*(r%4) .. +3, so lane i of group g receives keys
// k0 .. k0+3 of dimension d0 + 16*(g & 1) + i: for the 32 lanes of a half,
// dimension d0 + (lane % 32).
__device__ __forceinline__ bf16x4_t k_tr4(const bf16_t* sk, int ks, int k0, int d0) {
    const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
    const bf16_t* p = sk + (k0 + (r >> 2)) * ks + d0 + (g & 1) * 16 + (r & 3) * 4;
    return __builtin_bit_cast(bf16x4_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                            (lds_i16x4_t*)(reinterpret_cast<uintptr_t>(p))));
}

// 16-bit element e of a 16-byte vector, and its value as a float when it is
// a bf16 (taken from the 32-bit words: an element extracted from a bf16
// vector type and stored on its own was seen to be miscompiled).
__device__ __forceinline__ bf16_t elem16(const vec16& v, int e) {
    return static_cast<bf16_t>(v.w[e >> 1] >> ((e & 1) * 16));
}
__device__ __forceinline__ float bf16_value(const vec16& v, int e) {
    return __uint_as_float((e & 1) ? (v.w[e >> 1] & 0xffff0000u) : (v.w[e >> 1] << 16));
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

constexpr int kXcds = 8;  // XCDs of the chip; workgroups are dealt to them in turn

template <bool B>
struct BoolTag {
    static constexpr bool value = B;
};

// Logical work item of this workgroup: consecutive items on one XCD, so the
// workgroups of one unit (which read the same key tiles or query rows) share
// that XCD's L2.
__device__ __forceinline__ int xcd_item(int n_items) {
    const int per_xcd = (n_items + kXcds - 1) / kXcds;
    return (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
}

// Token of row `row` of tile `tile` of chunk c's working set: the current
// chunk, the visible chunks in ascending order, then the routed rows in
// group_idx order, 64 per tile; -1 for a padded, future or invalid routed row.
__device__ __forceinline__ int tile_token(int tile, int row, int c, const VisibleChunks& vis,
                                          const int* gid, int routed_rows, int group_shift, int lim) {
    if (tile <= vis.count) return (tile == 0 ? c : vis.chunk(tile - 1)) * KT + row;
    const int rr = (tile - 1 - vis.count) * KT + row;
    const int g = rr < routed_rows ? gid[rr >> group_shift] : -1;
    return g >= 0 && g < lim ? (g << group_shift) + (rr & ((1 << group_shift) - 1)) : -1;
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

    // B fragments of S^T = K.Q^T and dP^T = V.dO^T (the lane's query row,
    // dimensions kk*16 + half*8 .. +7), the same for every key tile: read
    // from LDS once
    bf16x8_t qf[NKS], gf[NKS];
#pragma unroll
    for (int kk = 0; kk < NKS; ++kk) {
        qf[kk] = frag(sQ + col * Lay::KS + kk * 16 + half * 8);
        gf[kk] = frag(sG + col * Lay::KS + kk * 16 + half * 8);
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
        // Stage K and V row-major (K^T operands are transpose reads of K); the token of each tile row
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
            const int tok = tile_token(tile, row, c, vis, s_gid, routed_rows, group_shift, lim);
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
                    sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(sK + krow * Lay::KS + off),
                                                                   qf[kk], sacc, 0, 0, 0);
                    pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(sV + krow * Lay::KS + off),
                                                                   gf[kk], pacc, 0, 0, 0);
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
                    const float p = __builtin_amdgcn_exp2f(ok ? sacc[e] * scale2 - lse2 : -INFINITY);
                    const float ds = p * (pacc[e] - dsum);
                    const __bf16 db = static_cast<__bf16>(ds);
                    dsf[e >> 3][e & 7] = db;
                    s_dst[kl * SCR + col] = __builtin_bit_cast(bf16_t, db);
                    s_pt[kl * SCR + col] = __builtin_bit_cast(bf16_t, static_cast<__bf16>(p));
                }
                // dQ += dS.K: k-slot half*8 + e of fragment kap is key
                // st*32 + kap*16 + (e/4)*8 + half*4 + e%4, so the B operand
                // is two 4-key runs of dimension nb*32 + col, transpose-read
                // from the row-major K tile.
#pragma unroll
                for (int kap = 0; kap < 2; ++kap)
#pragma unroll
                    for (int nb = 0; nb < NDT; ++nb) {
                        const int k0 = st * 32 + kap * 16 + half * 4;
                        const bf16x4_t lo = k_tr4(sK, Lay::KS, k0, nb * 32);
                        const bf16x4_t hi = k_tr4(sK, Lay::KS, k0 + 8, nb * 32);
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

// ---------------------------------------------------------------------------
// Split form for units whose query rows span several workgroups (GQA with
// r = n_q_heads/n_kv_heads > 1): there every workgroup of a unit would add
// the key gradients of the whole working set, and those fp32 atomics set the
// pace.  Instead one kernel takes dQ query-major (K/V tiles staged once per
// eight query tiles) and a second takes dK, dV key-major within the unit:
// each wavefront keeps 32 keys' K and V fragments and their dK, dV in
// registers, streams all r*64 query rows of the unit past them, and adds
// its gradients once.  S and dP are computed by both.

// dQ only: the fused kernel's query side, Q and dO fragments in registers.
template <int D>
struct DqLayout {
    static constexpr int KS = D + 8;
    static constexpr int TS = KT + 4;
    static constexpr int kK = 0;
    static constexpr int kV = kK + KT * KS * 2;
    static constexpr int kKT = kV + KT * KS * 2;
    static constexpr int kTok = kKT + D * TS * 2;
    static constexpr int kGid = kTok + KT * 4;
    static constexpr int kBytes = kGid + kMaxTopK * 4;
};

template <int D, int NW>
__global__ __launch_bounds__(NW * 64) void attend_bwd_dq_kernel(
    const bf16_t* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const bf16_t* __restrict__ k_res,
    const bf16_t* __restrict__ v_res, int64_t res_tokens, const int32_t* __restrict__ group_idx,
    const bf16_t* __restrict__ out, const float* __restrict__ lse,
    const bf16_t* __restrict__ dout, float* __restrict__ dq, int r, int n_kv, int group_shift,
    int keep_first, int window, int topk_groups, int wg_per_unit, int n_items) {
    using Lay = DqLayout<D>;
    constexpr int NKS = D / 16;
    constexpr int NDT = D / 32;
    constexpr int VPR = D / 8;
    constexpr int TPR = NW * 64 / KT;  // staging threads per tile row
    constexpr int VPT = VPR / TPR;     // 16-byte vectors per staging thread
    static_assert(VPT >= 1 && VPT * TPR == VPR, "staging split");
    extern __shared__ __align__(16) unsigned char smem[];
    bf16_t* sK = reinterpret_cast<bf16_t*>(smem + Lay::kK);
    bf16_t* sV = reinterpret_cast<bf16_t*>(smem + Lay::kV);
    bf16_t* sKT = reinterpret_cast<bf16_t*>(smem + Lay::kKT);
    int* s_tok = reinterpret_cast<int*>(smem + Lay::kTok);
    int* s_gid = reinterpret_cast<int*>(smem + Lay::kGid);

    const int item = xcd_item(n_items);
    if (item >= n_items) return;
    const int unit = item / wg_per_unit, part = item % wg_per_unit;
    const int bh = unit / n_q_chunks, i = unit % n_q_chunks;
    const int b = bh / n_kv, j = bh % n_kv;
    const int c = q_chunk0 + i;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, col = lane & 31;
    const int gpc = KT >> group_shift;
    const int qtile = part * NW + wave;
    const bool qactive = qtile < 2 * r;
    const int routed_rows = topk_groups << group_shift;
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * KT;
    const int n_q_heads = r * n_kv;
    auto qrow_of = [&](int m) {
        const int row = (qactive ? qtile : 0) * 32 + m;
        return (static_cast<int64_t>(b) * n_q_heads + j * r + row / KT) * qtok +
               static_cast<int64_t>(i) * KT + row % KT;
    };
    const int t = (qtile * 32 + col) % KT;
    const int64_t my_row = qrow_of(col);
    const float scale2 = 1.4426950408889634f / sqrtf(static_cast<float>(D));
    const float inv_sqrt_d = 1.0f / sqrtf(static_cast<float>(D));

    for (int s = tid; s < topk_groups; s += NW * 64)
        s_gid[s] = group_idx[static_cast<int64_t>(unit) * topk_groups + s];

    // B fragments of S^T = K.Q^T and dP^T = V.dO^T: the lane's query row,
    // dimensions kk*16 + half*8 .. +7
    bf16x8_t qf[NKS], gf[NKS];
    float dsum = 0.f, lse2 = 0.f;
    {
        float acc = 0.f;
#pragma unroll
        for (int kk = 0; kk < NKS; ++kk) {
            qf[kk] = bf16x8_t{};
            gf[kk] = bf16x8_t{};
            if (qactive) {
                qf[kk] = frag(q_rot + my_row * D + kk * 16 + half * 8);
                gf[kk] = frag(dout + my_row * D + kk * 16 + half * 8);
                const bf16x8_t o8 = frag(out + my_row * D + kk * 16 + half * 8);
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    acc = fmaf(static_cast<float>(gf[kk][e]), static_cast<float>(o8[e]), acc);
            }
        }
        dsum = add_halves(acc);
        if (qactive) lse2 = lse[my_row] * 1.4426950408889634f;
    }

    f32x16_t dqacc[NDT];
#pragma unroll
    for (int nb = 0; nb < NDT; ++nb)
#pragma unroll
        for (int e = 0; e < 16; ++e) dqacc[nb][e] = 0.f;

    const VisibleChunks vis(c, keep_first, window);
    const int n_tiles = 1 + vis.count + (routed_rows + KT - 1) / KT;
    const bf16_t* kbase = k_res + static_cast<int64_t>(bh) * res_tokens * D;
    const bf16_t* vbase = v_res + static_cast<int64_t>(bh) * res_tokens * D;
    const int lim = c * gpc;

    // The next tile's rows are fetched into registers while this one is
    // used.  K is also staged transposed (K^T rows, one 16-bit write per
    // element): the eight query-tile waves all read K^T for dQ, so one copy
    // per tile costs less than a transpose read per wave (measured).
    const int srow = tid % KT, pv = tid / KT;
    vec16 kx[VPT], vx[VPT];
    int stok = -1;
    auto fetch = [&](int tile) {
        stok = tile_token(tile, srow, c, vis, s_gid, routed_rows, group_shift, lim);
#pragma unroll
        for (int u = 0; u < VPT; ++u) {
            const int cv = pv * VPT + u;
            kx[u] = vec16{{0u, 0u, 0u, 0u}};
            vx[u] = kx[u];
            if (stok >= 0) {
                kx[u] = load16(kbase + static_cast<int64_t>(stok) * D + cv * 8);
                vx[u] = load16(vbase + static_cast<int64_t>(stok) * D + cv * 8);
            }
        }
    };
    fetch(0);  // the current chunk: no group id needed yet

    for (int tile = 0; tile < n_tiles; ++tile) {
        if (tile > 0) lds_barrier();  // every wave is done with the previous tile
        if (pv == 0) s_tok[srow] = stok;
#pragma unroll
        for (int u = 0; u < VPT; ++u) {
            const int cv = pv * VPT + u;
            *reinterpret_cast<vec16*>(sK + srow * Lay::KS + cv * 8) = kx[u];
            *reinterpret_cast<vec16*>(sV + srow * Lay::KS + cv * 8) = vx[u];
#pragma unroll
            for (int e = 0; e < 8; ++e) sKT[(cv * 8 + e) * Lay::TS + srow] = elem16(kx[u], e);
        }
        lds_barrier();
        if (tile + 1 < n_tiles) fetch(tile + 1);
        if (!qactive) continue;
        const bool current = tile == 0;
#pragma unroll
        for (int st = 0; st < 2; ++st) {
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
                sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(sK + krow * Lay::KS + off), qf[kk],
                                                               sacc, 0, 0, 0);
                pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(sV + krow * Lay::KS + off), gf[kk],
                                                               pacc, 0, 0, 0);
            }
            bf16x8_t dsf[2];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int key = st * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
                const bool ok = s_tok[key] >= 0 && (!current || key <= t);
                const float p = __builtin_amdgcn_exp2f(ok ? sacc[e] * scale2 - lse2 : -INFINITY);
                dsf[e >> 3][e & 7] = static_cast<__bf16>(p * (pacc[e] - dsum));
            }
#pragma unroll
            for (int kap = 0; kap < 2; ++kap)
#pragma unroll
                for (int nb = 0; nb < NDT; ++nb) {
                    const bf16_t* kp = sKT + (nb * 32 + col) * Lay::TS + st * 32 + kap * 16 + half * 4;
                    const bf16x8_t bf = __builtin_shufflevector(frag4(kp), frag4(kp + 8), 0, 1, 2, 3, 4, 5, 6, 7);
                    dqacc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(dsf[kap], bf, dqacc[nb], 0, 0, 0);
                }
        }
    }

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

// D_i = dout_i . out_i of every query row into dsum (indexed like lse):
// eight threads per row, each over every eighth 16-byte vector.
template <int D>
__global__ __launch_bounds__(256) void attend_bwd_dsum_kernel(const bf16_t* __restrict__ out,
                                                              const bf16_t* __restrict__ dout,
                                                              float* __restrict__ dsum, int64_t rows) {
    constexpr int VPR = D / 8;
    const int64_t row = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) >> 3;
    const int part = threadIdx.x & 7;
    float acc = 0.f;
    if (row < rows) {
#pragma unroll
        for (int u = 0; u < VPR / 8; ++u) {
            const vec16 g = load16(dout + row * D + (u * 8 + part) * 8);
            const vec16 o = load16(out + row * D + (u * 8 + part) * 8);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc = fmaf(bf16_value(g, e), bf16_value(o, e), acc);
        }
    }
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 4);
    if (row < rows && part == 0) dsum[row] = acc;
}

// dK, dV key-major within a unit.  Work item (unit, tile group): 2*NSUB
// wavefronts over the NSUB 32-key sub-tiles of working-set tiles
// (NSUB/2)*group .. (NSUB/2)*group + NSUB/2 - 1 (one tile for NSUB = 2).
// Wave w takes sub-tile w % NSUB in role w / NSUB: role 0 computes
// S = Q.K^T and dP = dO.V^T, then dS and dK += dS^T.Q; role 1 recomputes S
// for P and dV += P^T.dO.  The B fragments of S and dP (the lane's key row
// of K, and of V for role 0) stay in registers, so per matrix instruction
// only the query side is read from LDS.  Each wave holds one 32 x D
// accumulator block, which keeps the registers within two waves per SIMD;
// with one tile per workgroup two workgroups share a CU, and their waves,
// not held together by a common barrier, hide each other's LDS and matrix
// latencies.  The cost is S computed twice.  The unit's query rows pass in
// 32-row tiles through two LDS buffers (Q, dO row-major, -lse in log2 units
// and D_i, which a pre-pass computes once per row); the B operands of dK and
// dV (Q^T, dO^T) are transpose reads of the same rows (k_tr4).
template <int D>
struct KvLayout {
    static constexpr int KS = D + 8;       // row stride (bf16) of the Q, dO rows
    static constexpr int kQ = 0;           // per buffer: Q rows, dO rows
    static constexpr int kStat = kQ + 2 * 32 * KS * 2;  // lse2[32], dsum[32]
    static constexpr int kBuf = kStat + 64 * 4;
    static constexpr int kTok = 2 * kBuf;               // up to 4 sub-tiles x 32 key tokens
    static constexpr int kBytes = kTok + 4 * 32 * 4;
};

template <int D, int NSUB>
__global__ __launch_bounds__(NSUB * 128) __attribute__((amdgpu_waves_per_eu(2, 2))) void attend_bwd_kv_kernel(
    const bf16_t* __restrict__ q_rot, int q_chunk0, int n_q_chunks, const bf16_t* __restrict__ k_res,
    const bf16_t* __restrict__ v_res, int64_t res_tokens, const int32_t* __restrict__ group_idx,
    const float* __restrict__ dsum, const float* __restrict__ lse,
    const bf16_t* __restrict__ dout, float* __restrict__ dk, float* __restrict__ dv, int r, int n_kv,
    int group_shift, int keep_first, int window, int topk_groups, int pairs_per_unit, int n_items) {
    using Lay = KvLayout<D>;
    constexpr int NKS = D / 16;
    constexpr int NDT = D / 32;
    constexpr int VPR = D / 8;
    constexpr int TPR = NSUB * 4;                    // staging threads per query row
    constexpr int VPT = VPR >= TPR ? VPR / TPR : 1;  // vectors per staging thread
    extern __shared__ __align__(16) unsigned char smem[];
    int* s_tok = reinterpret_cast<int*>(smem + Lay::kTok);

    const int item = xcd_item(n_items);
    if (item >= n_items) return;
    const int unit = item / pairs_per_unit, pair = item % pairs_per_unit;
    const int bh = unit / n_q_chunks, i = unit % n_q_chunks;
    const int b = bh / n_kv, j = bh % n_kv;
    const int c = q_chunk0 + i;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = lane >> 5, col = lane & 31;
    const int sub = wave % NSUB, role = wave / NSUB;
    const int gpc = KT >> group_shift;
    const int routed_rows = topk_groups << group_shift;
    const VisibleChunks vis(c, keep_first, window);
    const int n_tiles = 1 + vis.count + (routed_rows + KT - 1) / KT;
    if (NSUB / 2 * pair >= n_tiles) return;  // the whole workgroup: past this unit's tiles
    const int tile = NSUB / 2 * pair + (sub >> 1);
    const int kr = (sub & 1) * 32 + col;  // the lane's key row in the tile
    const bool kactive = tile < n_tiles;
    const bool current = tile == 0;
    const int tok = kactive ? tile_token(tile, kr, c, vis,
                                         group_idx + static_cast<int64_t>(unit) * topk_groups,
                                         routed_rows, group_shift, c * gpc)
                            : -1;
    const int64_t kvoff = static_cast<int64_t>(bh) * res_tokens * D;
    const float kbias = tok >= 0 ? 0.f : -INFINITY;

    if (role == 0 && half == 0) s_tok[sub * 32 + col] = tok;
    // B fragments of S = Q.K^T and dP = dO.V^T: the lane's key row,
    // dimensions kk*16 + half*8 .. +7 (V for role 0 only)
    bf16x8_t kf[NKS], vf[NKS];
#pragma unroll
    for (int kk = 0; kk < NKS; ++kk) {
        kf[kk] = bf16x8_t{};
        vf[kk] = bf16x8_t{};
        if (tok >= 0) {
            kf[kk] = frag(k_res + kvoff + static_cast<int64_t>(tok) * D + kk * 16 + half * 8);
            if (role == 0) vf[kk] = frag(v_res + kvoff + static_cast<int64_t>(tok) * D + kk * 16 + half * 8);
        }
    }

    f32x16_t acc[NDT];  // role 0: dK, role 1: dV
#pragma unroll
    for (int nb = 0; nb < NDT; ++nb)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[nb][e] = 0.f;

    const int n_q_heads = r * n_kv;
    const int64_t qtok = static_cast<int64_t>(n_q_chunks) * KT;
    const float scale2 = 1.4426950408889634f / sqrtf(static_cast<float>(D));
    const float inv_sqrt_d = 1.0f / sqrtf(static_cast<float>(D));
    const int nq = 2 * r;  // 32-row query tiles of the unit

    // staging: thread (row sm, part sp) moves vectors sp, sp + TPR, .. of
    // the row (so the transposed writes of one instruction spread over the
    // banks); at d = 64 with 16 threads per row, parts 8 .. 15 stay idle
    const int sm = tid / TPR, sp = tid % TPR;
    const bool sput = sp < VPR;
    vec16 qx[VPT], gx[VPT];
    float lsex = 0.f, dsx = 0.f;
    auto fetch = [&](int qt) {
        const int row = qt * 32 + sm;
        const int64_t g = (static_cast<int64_t>(b) * n_q_heads + j * r + row / KT) * qtok +
                          static_cast<int64_t>(i) * KT + row % KT;
#pragma unroll
        for (int u = 0; u < VPT; ++u) {
            const int cv = u * TPR + sp;
            qx[u] = gx[u] = vec16{{0u, 0u, 0u, 0u}};
            if (sput) {
                qx[u] = load16(q_rot + g * D + cv * 8);
                gx[u] = load16(dout + g * D + cv * 8);
            }
        }
        if (sp == 0) {
            lsex = lse[g];
            dsx = dsum[g];
        }
    };
    auto put = [&](int buf) {
        unsigned char* base = smem + buf * Lay::kBuf;
        bf16_t* sQ = reinterpret_cast<bf16_t*>(base + Lay::kQ);
        bf16_t* sG = sQ + 32 * Lay::KS;
        float* s_stat = reinterpret_cast<float*>(base + Lay::kStat);
        if (sput) {
#pragma unroll
            for (int u = 0; u < VPT; ++u) {
                const int cv = u * TPR + sp;
                store16(sQ + sm * Lay::KS + cv * 8, qx[u]);
                store16(sG + sm * Lay::KS + cv * 8, gx[u]);
            }
        }
        if (sp == 0) {
            s_stat[sm] = -lsex * 1.4426950408889634f;  // -lse, log2 units
            s_stat[32 + sm] = dsx;
        }
    };

    fetch(0);
    put(0);
    lds_barrier();
    // The masks (causal on the current chunk, -inf for a skipped key row)
    // cost three vector instructions per score; most waves have neither, so
    // the query-tile loop exists in two forms and each wave takes its own
    // (the forms execute the same barriers).
    auto qtiles = [&](auto mask_tag) {
    constexpr bool kMask = decltype(mask_tag)::value;
    for (int qt = 0; qt < nq; ++qt) {
        const int buf = qt & 1;
        if (qt + 1 < nq) fetch(qt + 1);
        if (kactive) {
            const unsigned char* base = smem + buf * Lay::kBuf;
            const bf16_t* sQ = reinterpret_cast<const bf16_t*>(base + Lay::kQ);
            const bf16_t* sG = sQ + 32 * Lay::KS;
            const float* s_stat = reinterpret_cast<const float*>(base + Lay::kStat);
            // S[query][key] (and dP for role 0): lane (half, col = key) holds
            // queries 8*(e/4) + 4*half + e%4
            f32x16_t sacc, pacc;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                sacc[e] = 0.f;
                pacc[e] = 0.f;
            }
#pragma unroll
            for (int kk = 0; kk < NKS; ++kk) {
                const int off = col * Lay::KS + kk * 16 + half * 8;
                sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(sQ + off), kf[kk], sacc, 0, 0, 0);
            }
            if (role == 0) {
#pragma unroll
                for (int kk = 0; kk < NKS; ++kk) {
                    const int off = col * Lay::KS + kk * 16 + half * 8;
                    pacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(frag(sG + off), vf[kk], pacc, 0, 0, 0);
                }
            }
            // A operand (dS^T for role 0, P^T for role 1): k-slot half*8 + e
            // of fragment kap is query kap*16 + (e/4)*8 + half*4 + e%4.  A
            // skipped key row (tok < 0) has bias -inf; the current tile adds
            // the causal mask.
            bf16x8_t af[2];
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4) {
                const float4 l4 = *reinterpret_cast<const float4*>(s_stat + g4 * 8 + half * 4);
                const float nl[4] = {kMask ? l4.x + kbias : l4.x, kMask ? l4.y + kbias : l4.y,
                                     kMask ? l4.z + kbias : l4.z, kMask ? l4.w + kbias : l4.w};
                float p[4];
#pragma unroll
                for (int x = 0; x < 4; ++x) {
                    float a = fmaf(sacc[g4 * 4 + x], scale2, nl[x]);
                    if (kMask && current)
                        a = kr <= buf * 32 + g4 * 8 + half * 4 + x ? a : -INFINITY;
                    p[x] = __builtin_amdgcn_exp2f(a);
                }
                if (role == 0) {
                    const float4 d4 = *reinterpret_cast<const float4*>(s_stat + 32 + g4 * 8 + half * 4);
                    const float dv4[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
                    for (int x = 0; x < 4; ++x)
                        af[g4 >> 1][(g4 & 1) * 4 + x] = static_cast<__bf16>(p[x] * (pacc[g4 * 4 + x] - dv4[x]));
                } else {
#pragma unroll
                    for (int x = 0; x < 4; ++x) af[g4 >> 1][(g4 & 1) * 4 + x] = static_cast<__bf16>(p[x]);
                }
            }
            // role 0: dK[key][d] += dS^T.Q; role 1: dV[key][d] += P^T.dO.  The
            // B operand (query k-slots as in af, dimension nb*32 + col) is
            // two 4-query runs transpose-read from the row-major Q or dO rows.
            const bf16_t* sX = role == 0 ? sQ : sG;
#pragma unroll
            for (int kap = 0; kap < 2; ++kap)
#pragma unroll
                for (int nb = 0; nb < NDT; ++nb) {
                    const int q0 = kap * 16 + half * 4;
                    const bf16x8_t bx = __builtin_shufflevector(k_tr4(sX, Lay::KS, q0, nb * 32),
                                                                k_tr4(sX, Lay::KS, q0 + 8, nb * 32),
                                                                0, 1, 2, 3, 4, 5, 6, 7);
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[kap], bx, acc[nb], 0, 0, 0);
                }
        }
        if (qt + 1 < nq) put(buf ^ 1);
        lds_barrier();
    }
    };
    if (current || __builtin_amdgcn_ballot_w64(tok < 0) != 0)
        qtiles(BoolTag<true>{});
    else
        qtiles(BoolTag<false>{});

    // acc[nb][e]: key 8*(e/4) + 4*half + e%4 of the sub-tile, dimension nb*32 + col
    if (kactive) {
        float* dst = role == 0 ? dk : dv;
        const float scale = role == 0 ? inv_sqrt_d : 1.f;
#pragma unroll
        for (int nb = 0; nb < NDT; ++nb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int kt = s_tok[sub * 32 + (e >> 2) * 8 + half * 4 + (e & 3)];
                if (kt >= 0)
                    unsafeAtomicAdd(dst + kvoff + static_cast<int64_t>(kt) * D + nb * 32 + col,
                                    acc[nb][e] * scale);
            }
    }
}

template <int D, int kNwDq>
hipError_t launch_bwd_split_t(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                              const void* k_res, const void* v_res, int64_t res_tokens,
                              const int32_t* group_idx, const void* out, const float* lse,
                              const void* dout, float* dq, float* dk, float* dv, hipStream_t stream) {
    const hga_params& p = plan.p;
    constexpr int kSub = 2;  // 32-key sub-tiles per key-side workgroup (one tile)
    static std::atomic<uint64_t> configured{0};  // per instantiation and device
    const hipError_t ce = once_per_device(configured, plan.device, [] {
        const hipError_t e = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&attend_bwd_dq_kernel<D, kNwDq>),
            hipFuncAttributeMaxDynamicSharedMemorySize, DqLayout<D>::kBytes);
        if (e != hipSuccess) return e;
        return hipFuncSetAttribute(reinterpret_cast<const void*>(&attend_bwd_kv_kernel<D, kSub>),
                                   hipFuncAttributeMaxDynamicSharedMemorySize, KvLayout<D>::kBytes);
    });
    if (ce != hipSuccess) return ce;
    const int r = p.n_q_heads / p.n_kv_heads;
    const int group_shift = p.group == 8 ? 3 : (p.group == 16 ? 4 : 5);
    const int window = recent_window(p);
    const int64_t units = static_cast<int64_t>(p.batch) * p.n_kv_heads * n_q_chunks;
    const int wg_per_unit = (2 * r + kNwDq - 1) / kNwDq;
    // tiles of the largest working set: the last chunk's visible chunks
    const int c_max = q_chunk0 + n_q_chunks - 1;
    const int n_rt = (p.topk_groups * p.group + KT - 1) / KT;
    const int max_tiles = 1 + VisibleChunks(c_max, p.keep_first, window).count + n_rt;
    const int pairs = (max_tiles + kSub / 2 - 1) / (kSub / 2);
    const int64_t items_dq = units * wg_per_unit, items_kv = units * pairs;
    if (items_dq > (int64_t(1) << 30) || items_kv > (int64_t(1) << 30)) return hipErrorInvalidConfiguration;
    auto grid = [](int64_t n) { return dim3(static_cast<unsigned>((n + kXcds - 1) / kXcds * kXcds)); };
    // D_i goes to the first rows floats of dq, which the dq kernel (last)
    // overwrites: no workspace of its own.
    const int64_t rows = static_cast<int64_t>(p.batch) * p.n_q_heads * n_q_chunks * KT;
    float* dsum = dq;
    hipLaunchKernelGGL((attend_bwd_dsum_kernel<D>), dim3(static_cast<unsigned>((rows * 8 + 255) / 256)),
                       dim3(256), 0, stream, static_cast<const bf16_t*>(out),
                       static_cast<const bf16_t*>(dout), dsum, rows);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attend_bwd_kv_kernel<D, kSub>), grid(items_kv), dim3(kSub * 128), KvLayout<D>::kBytes, stream,
                       static_cast<const bf16_t*>(q_rot), q_chunk0, n_q_chunks,
                       static_cast<const bf16_t*>(k_res), static_cast<const bf16_t*>(v_res), res_tokens,
                       group_idx, dsum, lse, static_cast<const bf16_t*>(dout),
                       dk, dv, r, p.n_kv_heads, group_shift, p.keep_first, window, p.topk_groups, pairs,
                       static_cast<int>(items_kv));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attend_bwd_dq_kernel<D, kNwDq>), grid(items_dq), dim3(kNwDq * 64),
                       DqLayout<D>::kBytes, stream, static_cast<const bf16_t*>(q_rot), q_chunk0,
                       n_q_chunks, static_cast<const bf16_t*>(k_res), static_cast<const bf16_t*>(v_res),
                       res_tokens, group_idx, static_cast<const bf16_t*>(out), lse,
                       static_cast<const bf16_t*>(dout), dq, r, p.n_kv_heads, group_shift, p.keep_first,
                       window, p.topk_groups, wg_per_unit, static_cast<int>(items_dq));
    return hipGetLastError();
}

template <int D, int NW>
hipError_t launch_bwd_t(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                        const void* k_res, const void* v_res, int64_t res_tokens,
                        const int32_t* group_idx, const void* out, const float* lse,
                        const void* dout, float* dq, float* dk, float* dv, hipStream_t stream) {
    const hga_params& p = plan.p;
    constexpr int kLds = BwdLayout<D, NW>::kBytes;
    static std::atomic<uint64_t> configured{0};  // per instantiation and device
    const hipError_t ce = once_per_device(configured, plan.device, [] {
        return hipFuncSetAttribute(reinterpret_cast<const void*>(&attend_bwd_kernel<D, NW>),
                                   hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
    });
    if (ce != hipSuccess) return ce;
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

// One fused kernel when a workgroup holds all of a unit's query tiles (four
// at d64, two at d128); otherwise the split pair of kernels.
namespace {
bool bwd_fused(const hga_params& p) {
    const int r = p.n_q_heads / p.n_kv_heads;
    return p.head_dim == 64 ? r <= 2 : r == 1;
}
}  // namespace

size_t attend_backward_lds_bytes(const hga_plan& plan) {
    const hga_params& p = plan.p;
    const int r = p.n_q_heads / p.n_kv_heads;
    if (bwd_fused(p)) {
        if (p.head_dim == 64) return r == 1 ? BwdLayout<64, 2>::kBytes : BwdLayout<64, 4>::kBytes;
        return BwdLayout<128, 2>::kBytes;
    }
    if (p.head_dim == 64)
        return DqLayout<64>::kBytes > KvLayout<64>::kBytes ? DqLayout<64>::kBytes : KvLayout<64>::kBytes;
    return DqLayout<128>::kBytes > KvLayout<128>::kBytes ? DqLayout<128>::kBytes : KvLayout<128>::kBytes;
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
#define HGA_BWD_SPLIT(DD, NN)                                                                    \
    return launch_bwd_split_t<DD, NN>(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res,         \
                                      res_tokens, group_idx, out, lse, dout, dq, dk, dv, stream)
    if (!bwd_fused(p)) {
        // the dq kernel's wavefronts: one per 32-row query tile, up to eight
        // (the split form starts at r = 3 for d = 64, r = 2 for d = 128)
        if (p.head_dim == 64) HGA_BWD_SPLIT(64, 8);
        if (r == 2) HGA_BWD_SPLIT(128, 4);
        HGA_BWD_SPLIT(128, 8);
    }
    if (p.head_dim == 64) {
        if (r == 1) HGA_BWD(64, 2);
        HGA_BWD(64, 4);
    }
    HGA_BWD(128, 2);
#undef HGA_BWD
#undef HGA_BWD_SPLIT
}

}  // namespace hga
