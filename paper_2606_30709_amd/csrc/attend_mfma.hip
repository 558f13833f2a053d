// Exact-token attention (Sec. 3.4, Eq. (1)) for bf16 inputs on the gfx950
// matrix cores (v_mfma_f32_32x32x16_bf16), flash style.
//
// Work unit: one (batch, KV head, query chunk).  All r = Hq/Hkv query heads
// of the KV head share the unit's working set (GQA, Sec. 2), so their
// r*64 query rows are packed as 32-row query tiles; a workgroup of four
// wavefronts (eight at d128) takes as many query tiles (or, with only two
// tiles, two wavefronts per tile split each key tile between them and merge
// at the end).
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
//
// Data movement: global memory is copied straight into LDS by buffer loads
// with the LDS-destination form (64 lanes x 16 bytes land at M0 + 16*lane),
// so no VGPRs stage the tiles.  The key tiles cycle through NS LDS stages:
// when tile t is consumed, tiles t+1 .. t+NS-2 are already in flight and the
// copy of tile t+NS-1 is issued into the stage tile t-1 has freed, with one
// workgroup barrier per tile; the first NS tiles are requested together at
// the start.  The unit's group ids arrive the same way; each wavefront
// loads its query fragments straight into registers.  Each copy lane
// picks its source 16 bytes so that K lands row-major with an XOR swizzle
// and V in the order its transpose reads consume it (see swz_k and
// v_slot_source): LDS reads are free of bank conflicts, and the V reads are
// addressed by immediate offsets from one base register.  The copies are written as inline assembly and waited for with explicit
// vmcnt counts (loads complete in issue order), because the compiler's own
// tracking of LDS-destination loads would wait for every copy in flight
// before any LDS read.  V^T operands come from gfx950's LDS transpose read
// (ds_read_b64_tr_b16): within each 16-lane group, lane i receives element
// i%4 of the 64-bit reads issued by lanes 4j + i/4, j = 0..3, so 16 lanes
// pointing at 4 keys x 16 dimensions hand each lane 4 keys of one dimension.
// All global reads go through buffer descriptors: offsets past a buffer's
// end read as zero.
#include <hip/hip_ext.h>
#include <math.h>

#include "attend_common.hpp"
#include "hga_internal.hpp"

namespace hga {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int KT = 64;  // keys per LDS tile (= chunk)
constexpr int kXcds = 8;
constexpr uint32_t kAbsent = 0xffff0000u;  // an offset past every buffer: reads zeros
constexpr int kMaxGroupSlots = 512;

// Descriptor words of a raw buffer [base, base + bytes) for the copies below
// (base address, no stride, num_records = bytes); the operands are uniform.
__device__ __forceinline__ u32x4 rsrc_words(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    u32x4 r;
    r.x = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
    r.y = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32) & 0xffffu);
    r.z = __builtin_amdgcn_readfirstlane(bytes);
    r.w = 0x00020000u;
    return r;
}

// Copy 16 bytes per lane from buffer offset voff to LDS byte lds + 16*lane.
__device__ __forceinline__ void copy16_to_lds(const u32x4& rs, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(voff), "s"(rs), "s"(lds)
                 : "memory");
}

// Copy 4 bytes per lane from buffer offset voff to LDS byte lds + 4*lane.
__device__ __forceinline__ void copy4_to_lds(const u32x4& rs, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\tbuffer_load_dword %0, %1, 0 offen lds"
                 :
                 : "v"(voff), "s"(rs), "s"(lds)
                 : "memory");
}

// Wait until at most N vector-memory loads of this wavefront are in flight.
template <int N>
__device__ __forceinline__ void wait_loads() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// LDS layout of a staged tile.
// * K is row-major, unpadded, with the 16-byte chunk j of
//   row r stored at j ^ swz_k(r): the 16-byte A/B fragments read by 32 lanes
//   on 32 consecutive rows then fall in distinct banks, and each copy reads
//   whole rows.  (For D = 128, 16 chunks per row, the map uses four bits.)
// * V is stored in the order its transpose reads consume it: block
//   (st, kap, hi, dt) -- keys st*32 + kap*16 + 8*hi + 0..7, dimensions
//   dt*32 .. dt*32+31 -- is 512 B at (((st*2 + kap)*2 + hi)*NDT + dt) * 512,
//   lane l holding the 8 bytes its ds_read_b64_tr_b16 asks for: key
//   (l>>5)*4 + ((l&15)>>2), dimensions ((l>>4)&1)*16 + (l&3)*4 .. +4 (two
//   lanes share each 16-byte slot).  Every V read is one contiguous block
//   (no bank conflicts) at an immediate offset from one base register, and
//   a copy still reads 8 rows x 128 contiguous bytes.
template <int D>
__device__ __forceinline__ int swz_k(int r) {
    if constexpr (D == 64)
        return ((r ^ (r >> 3)) & 1) | (((r >> 2) & 1) << 1) | (((r >> 1) & 1) << 2);
    else
        return ((r ^ (r >> 3)) & 1) | (((r ^ (r >> 2)) & 1) << 1) | (((r >> 1) & 1) << 2) |
               ((r & 1) << 3);
}
// Source (row, 16-byte chunk) of 16-byte slot P of the V region.
template <int D>
__device__ __forceinline__ void v_slot_source(int P, int& row, int& chunk) {
    constexpr int NDT = D / 32;
    const int blk = P >> 5, q = P & 31;  // 32 slots per 512-byte block
    const int dt = blk % NDT, h = blk / NDT;  // h = (st*2 + kap)*2 + hi
    row = (h >> 2) * 32 + ((h >> 1) & 1) * 16 + (h & 1) * 8 + (q >> 4) * 4 + ((q & 7) >> 1);
    chunk = dt * 4 + ((q >> 3) & 1) * 2 + (q & 1);
}

// x and the value of lane l ^ 32 combined, without an LDS round trip:
// v_permlane32_swap hands each lane of one half the other half's value (the
// two results hold (partner, own) in lanes 0..31 and (own, partner) above).
__device__ __forceinline__ float max_xor32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float add_xor32(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                    false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ bf16x8_t lds_frag(const bf16_t* p) {
    return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const vec16*>(p));
}

__device__ __forceinline__ i16x4_t lds_read_tr16(const bf16_t* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4_t*)(reinterpret_cast<uintptr_t>(p)));
}

template <bool B>
struct BoolTag {
    static constexpr bool value = B;
};

template <int D, int NS>
struct Layout {
    static constexpr uint32_t kRowBytes = D * 2;
    static constexpr uint32_t kTileBytes = KT * kRowBytes;  // one of K or V
    static constexpr uint32_t kStageBytes = 2 * kTileBytes;
    static constexpr uint32_t kGidOffset = NS * kStageBytes;
    static constexpr uint32_t kBytes = kGidOffset + kMaxGroupSlots * 4;
};

// Per-key-tile arithmetic for one wavefront:
//   S^T = K.Q^T over its 32-key sub-tile(s), the causal mask (current chunk)
//   or the routed-row mask (partial routed tile), the online-softmax update
//   of (m_run, l_run, oacc), and O^T += V^T.P^T.
// sK/sV: the staged tile; ksplit: this wave's key half when KS == 2;
// t: this lane's query token; rt_row0: first routed row of the tile.
// With both sub-tiles in one wavefront (KS == 1) the softmax is updated per
// 32-key sub-tile, so the matrix products of one sub-tile are independent of
// the exponentials of the other and the two overlap in the wavefront.
template <int D, int KS, bool kCurrent>
__device__ __forceinline__ void tile_math(const bf16_t* sK, const bf16_t* sV,
                                          const bf16x8_t (&qf)[D / 16], f32x16_t (&oacc)[D / 32],
                                          float& m_run, float& l_run, int ksplit, int t,
                                          bool partial, int rt_row0, const int* s_gid,
                                          int routed_rows, int topk_groups, int group_shift,
                                          int id_limit) {
    constexpr int NDT = D / 32, NKS = D / 16, NST = 2 / KS;
    const int lane = threadIdx.x & 63;
    const int half = lane >> 5, col = lane & 31;
    const float scale = 1.4426950408889634f / sqrtf(static_cast<float>(D));  // log2(e)/sqrt(d)

    // S^T of 32-key sub-tile st, masked (`diag`: the current chunk's
    // sub-tile holding this wave's own tokens, under the causal mask)
    auto qk = [&](int st, f32x16_t& sacc, bool diag) {
        const int krow = st * 32 + col;
        bf16x8_t kf[NKS];
#pragma unroll
        for (int kk = 0; kk < NKS; ++kk)
            kf[kk] = lds_frag(sK + krow * D + ((2 * kk + half) ^ swz_k<D>(col)) * 8);
#pragma unroll
        for (int e = 0; e < 16; ++e) sacc[e] = 0.f;
#pragma unroll
        for (int kk = 0; kk < NKS; ++kk)
            sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], sacc, 0, 0, 0);
        if (kCurrent) {
            if (diag) {
#pragma unroll
                for (int e = 0; e < 16; ++e) {
                    const int key = st * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
                    sacc[e] = key > t ? -INFINITY : sacc[e];
                }
            }
        } else if (partial) {
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int row = rt_row0 + st * 32 + (e >> 2) * 8 + half * 4 + (e & 3);
                const int slot = min(row >> group_shift, topk_groups - 1);
                const int id = s_gid[slot];
                const bool ok = row < routed_rows && id >= 0 && id < id_limit;
                sacc[e] = ok ? sacc[e] : -INFINITY;
            }
        }
    };
    // The online softmax in three pieces.  The reference point m_run of the
    // exponentials moves only when a sub-tile's maximum exceeds it by more
    // than kSlack (log2 units): the weights exp2(s - m_run) then stay below
    // 2^kSlack, exact in fp32 and in bf16's range, and the rescale of the
    // output is rarely needed.  The normalisation and the log-sum-exp use
    // the same m_run, so the result is the softmax for any reference point.
    constexpr float kSlack = 8.0f;
    // row maximum of one sub-tile's scores (scaled: log2 units), uniform over
    // the two lanes of a query column
    auto row_max = [&](const f32x16_t& sacc) {
        float tmax = -INFINITY;
#pragma unroll
        for (int e = 0; e < 16; ++e) tmax = fmaxf(tmax, sacc[e]);
        return max_xor32(tmax) * scale;
    };
    // move the reference point to tmax where it exceeds it by more than
    // kSlack (never while the row is fully masked), rescaling O and l
    auto rebase = [&](float tmax) {
        const bool grow = tmax > m_run + kSlack;
        if (__builtin_amdgcn_ballot_w64(grow)) {
            const float alpha = grow ? __builtin_amdgcn_exp2f(m_run - tmax) : 1.0f;
            l_run *= alpha;
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int e = 0; e < 16; ++e) oacc[dt][e] *= alpha;
            m_run = grow ? tmax : m_run;
        }
    };
    // weights of one sub-tile against reference m_use, added to l; P as bf16
    auto exps = [&](const f32x16_t& sacc, float m_use, bf16x8_t* pf) {
#pragma unroll
        for (int kap = 0; kap < 2; ++kap)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float pv = __builtin_amdgcn_exp2f(fmaf(sacc[kap * 8 + e], scale, -m_use));
                l_run += pv;
                pf[kap][e] = static_cast<__bf16>(pv);
            }
    };
    auto m_use = [&]() { return m_run == -INFINITY ? 0.f : m_run; };
    // kFirst: the wave's first scores (O and l still zero, and every lane
    // has a visible key among them), so the reference point is simply set.
    auto update = [&](const f32x16_t& sacc, bf16x8_t* pf, auto first_tag) {
        constexpr bool kFirst = decltype(first_tag)::value;
        const float tmax = row_max(sacc);
        if (kFirst)
            m_run = tmax;
        else
            rebase(tmax);
        exps(sacc, m_use(), pf);
    };
    // O^T += V^T.P^T for 32-key sub-tile st
    auto pv = [&](int st, const bf16x8_t* pf) {
#pragma unroll
        for (int kap = 0; kap < 2; ++kap) {
            // V^T operand: keys st*32 + kap*16 + {half*4 + 0..3, 8 + half*4 + 0..3}
            // at dimension dt*32 + col, from the two transpose-read blocks
            // (st, kap, 0, dt) and (st, kap, 1, dt).
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt) {
                const bf16_t* vp0 = sV + ((((st * 2 + kap) * 2 + 0) * NDT + dt) * 64 + lane) * 4;
                const bf16_t* vp1 = sV + ((((st * 2 + kap) * 2 + 1) * NDT + dt) * 64 + lane) * 4;
                const i16x4_t lo = lds_read_tr16(vp0);
                const i16x4_t hi = lds_read_tr16(vp1);
                const bf16x8_t a = __builtin_bit_cast(
                    bf16x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
                oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pf[kap], oacc[dt], 0, 0, 0);
            }
        }
    };

    using First = BoolTag<true>;
    using Later = BoolTag<false>;
    if constexpr (kCurrent) {
        // The current chunk: this wave's tokens t lie in 32-key sub-tile tq
        // (the same for every lane).  Sub-tiles before tq are fully visible,
        // tq is the diagonal, later ones are fully masked and skipped.
        const int tq = __builtin_amdgcn_readfirstlane(t) >> 5;
        if constexpr (NST == 1) {
            if (ksplit > tq) return;
            f32x16_t sacc[1];
            bf16x8_t pf[2];
            qk(ksplit, sacc[0], ksplit == tq);
            update(sacc[0], pf, First{});
            pv(ksplit, pf);
        } else if (tq == 0) {
            f32x16_t s0[1];
            bf16x8_t p0[2];
            qk(0, s0[0], true);
            update(s0[0], p0, First{});
            pv(0, p0);
        } else {
            f32x16_t s0[1], s1[1];
            bf16x8_t p0[2], p1[2];
            qk(0, s0[0], false);
            qk(1, s1[0], true);
            update(s0[0], p0, First{});
            pv(0, p0);
            update(s1[0], p1, Later{});
            pv(1, p1);
        }
    } else if constexpr (NST == 1) {
        f32x16_t sacc[1];
        bf16x8_t pf[2];
        qk(ksplit, sacc[0], false);
        update(sacc[0], pf, Later{});
        pv(ksplit, pf);
    } else {
        // The steps of update-then-product per sub-tile, ordered so that
        // each sub-tile's exponentials sit beside the other sub-tile's
        // matrix products (qk(1) beside the weights of sub-tile 0, pv(0)
        // beside the maximum of sub-tile 1); every value is the one the
        // plain order gives.  Masked scores (partial routed tiles) are -inf
        // and weigh zero.
        f32x16_t s0, s1;
        bf16x8_t p0[2], p1[2];
        qk(0, s0, false);
        rebase(row_max(s0));
        const float mu0 = m_use();
        qk(1, s1, false);
        exps(s0, mu0, p0);
        const float t1 = row_max(s1);
        pv(0, p0);
        rebase(t1);
        exps(s1, m_use(), p1);
        pv(1, p1);
    }
}

// Whether routed tile rows [rt_row0, rt_row0 + 64) include any row to mask:
// lane j checks the tile's j-th group (one LDS read each), a ballot joins them.
__device__ __forceinline__ bool routed_tile_partial(int rt_row0, const int* s_gid, int routed_rows,
                                                    int topk_groups, int group_shift,
                                                    int id_limit) {
    const int lane = threadIdx.x & 63;
    const int g = (rt_row0 >> group_shift) + lane;
    bool bad = false;
    if (lane < (KT >> group_shift)) {
        const int id = g < topk_groups ? s_gid[g] : -1;
        bad = !(id >= 0 && id < id_limit);
    }
    return rt_row0 + KT > routed_rows || __builtin_amdgcn_ballot_w64(bad) != 0;
}

// Combine the two key halves of a query tile (KS == 2) through LDS (`area`:
// QT * 64 * NDT*16 floats, `ml`: QT * 128 floats, both free), then store the
// normalised output and the log-sum-exp.  Every wave of the workgroup calls.
// The normalisation 1/l is folded into the two merge factors, so each output
// element costs one multiply and one fma.
// The output tile of a query tile (32 consecutive rows of one head,
// contiguous in `out`) is staged row-major in LDS (`stage`: QT tiles of 32
// rows of kOutStride bytes, the rows padded by 8 bytes against bank
// conflicts) and written back as contiguous 16-byte non-temporal stores
// (full lines; the output is not read again by the step).
template <int D>
constexpr int kOutStride = 2 * D + 8;
template <int D, int KS, int QT>
constexpr size_t out_stage_offset() {
    return KS == 2 ? (static_cast<size_t>(QT) * 64 * (D / 32) * 16 + QT * 128) * sizeof(float) : 0;
}
template <int D, int KS, int QT>
constexpr size_t out_stage_end() {
    return out_stage_offset<D, KS, QT>() + static_cast<size_t>(QT) * 32 * kOutStride<D>;
}

template <int D, int KS, int QT>
__device__ __forceinline__ void finish_rows(f32x16_t (&oacc)[D / 32], float m_run, float l_run,
                                            float* area, float* ml_area, int qt_local, int ksplit,
                                            bool qactive, bool bad, bf16_t* orow, float* lse_at) {
    constexpr int NDT = D / 32;
    const int lane = threadIdx.x & 63, half = lane >> 5;
    float l_tot = add_xor32(l_run);
    // element k of the partner's accumulator at [qt_local][k][lane]: lanes contiguous
    float* mine = area + qt_local * (NDT * 16 * 64) + lane;
    float f_own = 1.f, f_other = 0.f;
    if (KS == 2) {
        float* ml = ml_area + qt_local * 128 + lane;
        if (ksplit == 1) {
#pragma unroll
            for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
                for (int e = 0; e < 16; ++e) mine[(dt * 16 + e) * 64] = oacc[dt][e];
            ml[0] = m_run;
            ml[64] = l_tot;
        }
        __syncthreads();
        if (ksplit == 0) {
            const float mb = ml[0], lb = ml[64];
            const float m = fmaxf(m_run, mb);
            const float mu = m == -INFINITY ? 0.f : m;
            f_own = __builtin_amdgcn_exp2f(m_run - mu);
            f_other = __builtin_amdgcn_exp2f(mb - mu);
            l_tot = l_tot * f_own + lb * f_other;
            m_run = m;
        }
    }
    if (!qactive || ksplit != 0) return;
    // l_tot >= 1 (the key that set the reference point contributes exp2(0)),
    // so the hardware reciprocal is within one ulp.
    const float inv = bad ? NAN : __builtin_amdgcn_rcpf(l_tot);
    f_own *= inv;
    f_other *= inv;
    const int col = lane & 31;
    unsigned char* stage = reinterpret_cast<unsigned char*>(area) + out_stage_offset<D, KS, QT>() +
                           static_cast<size_t>(qt_local) * 32 * kOutStride<D>;
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
            const int d0 = dt * 32 + g4 * 8 + half * 4;
            typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
            bf16x4_t o;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int k = g4 * 4 + e;
                const float x = KS == 2 ? fmaf(mine[(dt * 16 + k) * 64], f_other,
                                               oacc[dt][k] * f_own)
                                        : oacc[dt][k] * f_own;
                o[e] = static_cast<__bf16>(x);
            }
            *reinterpret_cast<bf16x4_t*>(stage + col * kOutStride<D> + d0 * 2) = o;
        }
    if (lse_at && half == 0) *lse_at = bad ? NAN : (m_run + log2f(l_tot)) * 0.6931471805599453f;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    // row r of the tile is output row (this lane's row) - col + r
    unsigned char* obase = reinterpret_cast<unsigned char*>(orow - static_cast<int64_t>(col) * D);
    constexpr int kChunks = 2 * D / 16;  // 16-byte chunks per row
#pragma unroll
    for (int it = 0; it < 32 * kChunks / 64; ++it) {
        const int idx = it * 64 + lane;
        const int r = idx / kChunks, cc = idx % kChunks;
        const vec16 v = *reinterpret_cast<const vec16*>(stage + r * kOutStride<D> + cc * 16);
        __builtin_nontemporal_store(__builtin_bit_cast(u32x4, v),
                                    reinterpret_cast<u32x4*>(obase + (r * D + cc * 8) * 2));
    }
}

// D: head dim; KS: wavefronts sharing one query tile (each
// takes one 32-key half of every key tile); NS: LDS stages of the key-tile
// ring; NW: wavefronts per workgroup (NW / KS query tiles per workgroup).
// One workgroup per (unit, part); its query rows and group ids are copied
// with the first tiles, then the key tiles stream through the ring.
// kGather: the routed rows are copied straight from the resident K/V (rows
// g*G .. g*G+G-1 of each routed group g, zeros for a padded or future group,
// as the gather step defines them), and when k_routed / v_routed are given
// the unit's first workgroup writes every routed tile it staged to them
// (with two or more workgroups per unit the first writes K and the second
// V), so the call also produces the gather step's output; when they are
// null the gathered rows live in LDS only.  Otherwise the routed rows are
// read from k_routed / v_routed.
// With kGather the routed rows come from k_src / v_src (src_tokens rows per
// head: the resident K/V itself for the prefill layout, or the history in
// pinned host memory, read through its device mapping, for a decode block).
// kSplit: the unit's key tiles are divided among split_div.d workgroups
// (split s takes tiles [ceil(s T / S), ceil((s+1) T / S)) of the T tiles, so
// split 0 holds the current chunk); each writes its unnormalised partial
// result to `partial_ws` instead of the output, and
// attend_combine_kernel merges them.
template <int D, int KS, int NS, int NW, bool kGather, bool kSplit = false>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(D == 64 && !kSplit ? 4 : 2))) void attend_mfma_kernel(
    const bf16_t* __restrict__ q_rot, int q_chunk0, int n_q_chunks,
    const bf16_t* __restrict__ k_res, const bf16_t* __restrict__ v_res, int64_t res_tokens,
    const int32_t* __restrict__ res_slot, bf16_t* __restrict__ k_routed,
    bf16_t* __restrict__ v_routed, const int32_t* __restrict__ group_idx,
    bf16_t* __restrict__ out, float* __restrict__ lse, int r, FastDiv kv_div, int group_shift,
    int keep_first, int window, int topk_groups, FastDiv wg_div, FastDiv chunk_div,
    int n_blocks, float* __restrict__ partial_ws, FastDiv split_div,
    const bf16_t* __restrict__ k_src, const bf16_t* __restrict__ v_src, int64_t src_tokens) {
    static_assert(!kSplit || KS == 1, "split form: one wavefront per query tile");
    using Lay = Layout<D, NS>;
    constexpr uint32_t kRowBytes = Lay::kRowBytes, kTileBytes = Lay::kTileBytes,
                       kStageBytes = Lay::kStageBytes;
    constexpr int kRowShift = D == 64 ? 7 : 8;    // log2(kRowBytes)
    static_assert((1u << kRowShift) == kRowBytes, "row bytes");
    constexpr int NDT = D / 32;                  // 32-wide output blocks
    constexpr int NKS = D / 16;                  // k-steps of Q.K^T
    constexpr int QT = NW / KS;                  // query tiles per workgroup
    constexpr int KI = kTileBytes / 1024 / NW;   // copies per wave per tile, for K (and V)
    constexpr int LPT = 2 * KI;                  // loads per wave per tile
    constexpr int GI = kMaxGroupSlots * 4 / 256 / NW;    // copies per wave for the group ids
    static_assert(KI >= 1 && GI >= 1, "copy split");
    static_assert(NS >= 2 && NS <= 4, "stages");
    static_assert(KS == 1 || QT * 64 * NDT * 16 * 4 <= NS * kStageBytes, "merge area");
    static_assert(out_stage_end<D, KS, QT>() <= Lay::kBytes, "output staging area");

    extern __shared__ __align__(16) unsigned char smem[];
    const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(smem));
    const int* s_gid = reinterpret_cast<const int*>(smem + Lay::kGidOffset);

    // XCD-aware order: consecutive workgroups of one XCD take consecutive
    // (head, chunk) units, so a unit's previous chunk and the head's sink
    // chunks are still in that XCD's L2.
    const int per_xcd = (n_blocks + kXcds - 1) / kXcds;
    const int logical = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (logical >= n_blocks) return;
    int item = logical, split = 0;
    if constexpr (kSplit) {
        item = split_div.div(logical);
        split = logical - item * split_div.d;
    }
    const int unit_id = wg_div.div(item);
    const int part = item - unit_id * wg_div.d;
    const int bh = chunk_div.div(unit_id);
    const int i = unit_id - bh * n_q_chunks;

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const int half = lane >> 5, col = lane & 31;
    const int nqt = 2 * r;
    const int n_kv = kv_div.d, n_q_heads = r * n_kv;
    const int b = kv_div.div(bh), j = bh - b * n_kv;
    const int c = q_chunk0 + i;
    const int group = 1 << group_shift;
    const int gpc = KT >> group_shift;
    const int qt_local = wave % QT;
    const int qtile = part * QT + qt_local;
    const int ksplit = wave / QT;
    const bool qactive = qtile < nqt;
    const int64_t unit = unit_id;
    const int routed_rows = topk_groups * group;
    const int64_t res_chunks = res_tokens / KT;

    const u32x4 rk_res = rsrc_words(k_res + static_cast<int64_t>(bh) * res_tokens * D,
                                    static_cast<uint32_t>(res_chunks * kTileBytes));
    const u32x4 rv_res = rsrc_words(v_res + static_cast<int64_t>(bh) * res_tokens * D,
                                    static_cast<uint32_t>(res_chunks * kTileBytes));
    const u32x4 rk_src = rsrc_words(k_src + static_cast<int64_t>(bh) * src_tokens * D,
                                    static_cast<uint32_t>(src_tokens * kRowBytes));
    const u32x4 rv_src = rsrc_words(v_src + static_cast<int64_t>(bh) * src_tokens * D,
                                    static_cast<uint32_t>(src_tokens * kRowBytes));
    // The routed buffers may be null (the gather form keeping the rows on
    // chip): their unit offsets are taken as integers, and the buffers are
    // only accessed when given.
    const int64_t rt_off = unit * routed_rows * static_cast<int64_t>(kRowBytes);
    const u32x4 rk_rt = rsrc_words(reinterpret_cast<const void*>(
                                       reinterpret_cast<uintptr_t>(k_routed) + rt_off),
                                   routed_rows * kRowBytes);
    const u32x4 rv_rt = rsrc_words(reinterpret_cast<const void*>(
                                       reinterpret_cast<uintptr_t>(v_routed) + rt_off),
                                   routed_rows * kRowBytes);

    // The unit's group ids into LDS.
    {
        const u32x4 rg = rsrc_words(group_idx + unit * topk_groups, topk_groups * 4);
#pragma unroll
        for (int u = 0; u < GI; ++u) {
            const int blk = u * NW + wave;
            copy4_to_lds(rg, (blk * 64 + lane) * 4, lds0 + Lay::kGidOffset + blk * 256);
        }
    }

    // this lane's query row (token t of head hh)
    const int qrow_in_unit = qtile * 32 + col;
    const int hh = qrow_in_unit / KT, t = qrow_in_unit % KT;
    const int64_t qrow = (static_cast<int64_t>(b) * n_q_heads + j * r + (qactive ? hh : 0)) *
                             (static_cast<int64_t>(n_q_chunks) * KT) +
                         static_cast<int64_t>(i) * KT + t;
    // Query fragments (B operand of S^T = K.Q^T), straight from global
    // memory into registers: row qrow, dimensions kk*16 + half*8 .. +8.
    // They are requested before any key tile, so they have arrived once the
    // first tile has.
    bf16x8_t qf[NKS];
    {
        const bf16_t* qp = q_rot + qrow * D + half * 8;
#pragma unroll
        for (int kk = 0; kk < NKS; ++kk) qf[kk] = __builtin_bit_cast(bf16x8_t, load16(qp + kk * 16));
    }

    // tile order: the current chunk, the visible closed chunks, the routed rows
    const VisibleChunks vis(c, keep_first, window);
    const int n_vis = vis.count;
    const int n_rt = (routed_rows + KT - 1) / KT;
    const int n_tiles = 1 + n_vis + n_rt;
    int t0 = 0, t1 = n_tiles;  // this workgroup's tiles
    if constexpr (kSplit) {
        const int ns = split_div.d;
        t0 = (split * n_tiles + ns - 1) / ns;
        t1 = ((split + 1) * n_tiles + ns - 1) / ns;
    }
    bool bad = false;

    // per-lane source offsets of this wave's copies inside a tile
    uint32_t koff[KI], voff[KI];
#pragma unroll
    for (int u = 0; u < KI; ++u) {
        const int pch = (u * NW + wave) * 64 + lane;
        const int row = pch / (D / 8), pc = pch % (D / 8);
        koff[u] = row * kRowBytes + (pc ^ swz_k<D>(row)) * 16;
        int vrow, vch;
        v_slot_source<D>(pch, vrow, vch);
        voff[u] = vrow * kRowBytes + vch * 16;
    }
    // Issue the copies of tile `tile` (< n_tiles) into stage `stage`.
    auto issue = [&](int tile, int stage) {
        const bool routed = tile > n_vis;
        uint32_t base;
        if (!routed) {
            const int cc = tile == 0 ? c : vis.chunk(tile - 1);
            const int64_t slot = res_slot ? res_slot[cc] : cc;
            if (slot < 0 || slot >= res_chunks) {
                bad = true;
                base = kAbsent;
            } else {
                base = static_cast<uint32_t>(slot * kTileBytes);
            }
        } else {
            base = static_cast<uint32_t>((tile - 1 - n_vis) * kTileBytes);
        }
        const uint32_t sk = lds0 + stage * kStageBytes;
        if (kGather && routed) {
            // Copied row `row` of the tile is routed row R = rt0 + row of the
            // unit, slot R / G, row R % G of the slot's group g; its source is
            // row g*G + R % G of the resident slab.  A tile starts on a group
            // boundary, so the source offset is g*G*rowbytes plus the copy
            // offset modulo G*rowbytes.  The ids are read before any is used
            // (the copies below are barriers to reordering).
            const int slot0 = ((tile - 1 - n_vis) * KT) >> group_shift;
            const uint32_t lim = static_cast<uint32_t>(c * gpc);
            const int gbytes_shift = group_shift + kRowShift;
            int gk[KI], gv[KI];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                gk[u] = s_gid[min(slot0 + static_cast<int>(koff[u] >> gbytes_shift), topk_groups - 1)];
                gv[u] = s_gid[min(slot0 + static_cast<int>(voff[u] >> gbytes_shift), topk_groups - 1)];
            }
            auto src = [&](uint32_t off, int g) {
                const int slot = slot0 + static_cast<int>(off >> gbytes_shift);
                const bool ok = slot < topk_groups && static_cast<uint32_t>(g) < lim;
                const uint32_t x = (static_cast<uint32_t>(g) << gbytes_shift) +
                                   (off & ((1u << gbytes_shift) - 1));
                return ok ? x : kAbsent;
            };
            uint32_t sk_off[KI], sv_off[KI];
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                sk_off[u] = src(koff[u], gk[u]);
                sv_off[u] = src(voff[u], gv[u]);
            }
#pragma unroll
            for (int u = 0; u < KI; ++u)
                copy16_to_lds(rk_src, sk_off[u], sk + (u * NW + wave) * 1024);
#pragma unroll
            for (int u = 0; u < KI; ++u)
                copy16_to_lds(rv_src, sv_off[u], sk + kTileBytes + (u * NW + wave) * 1024);
            return;
        }
        const u32x4 rk = routed ? rk_rt : rk_res;
        const u32x4 rv = routed ? rv_rt : rv_res;
#pragma unroll
        for (int u = 0; u < KI; ++u)
            copy16_to_lds(rk, base + koff[u], sk + (u * NW + wave) * 1024);
#pragma unroll
        for (int u = 0; u < KI; ++u)
            copy16_to_lds(rv, base + voff[u], sk + kTileBytes + (u * NW + wave) * 1024);
    };
    // kGather: write the routed tile in `stage` (this lane's own copies, so
    // its own wait suffices) to the routed buffers at the offsets it was
    // copied from, rows past the unit's routed rows left out.  With several
    // workgroups per unit, part 0 writes K and part 1 writes V.  The stores
    // are non-temporal: the routed buffers are an output of the step, not
    // read again by it, and cached copies would be written back during the
    // next kernel (measured: the next step's summaries launch 87 -> 70 us on
    // the 32K-token GQA layer, the attention unchanged).
    auto store16_nt = [](unsigned char* p, const vec16& x) {
        __builtin_nontemporal_store(__builtin_bit_cast(u32x4, x), reinterpret_cast<u32x4*>(p));
    };
    // (no routed buffers given: the routed rows are gathered into LDS only)
    const bool write_k = kGather && k_routed != nullptr && part == 0;
    const bool write_v = kGather && v_routed != nullptr && part == (wg_div.d == 1 ? 0 : 1);
    auto write_routed = [&](int tile, int stage) {
        const int rt0 = (tile - 1 - n_vis) * KT;
        const unsigned char* sk = smem + stage * kStageBytes;
        if (write_k) {
            bf16_t* kdst = k_routed + (unit * routed_rows + rt0) * D;
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const vec16 x =
                    *reinterpret_cast<const vec16*>(sk + (u * NW + wave) * 1024 + lane * 16);
                if (rt0 + static_cast<int>(koff[u] / kRowBytes) < routed_rows)
                    store16_nt(reinterpret_cast<unsigned char*>(kdst) + koff[u], x);
            }
        }
        if (write_v) {
            bf16_t* vdst = v_routed + (unit * routed_rows + rt0) * D;
#pragma unroll
            for (int u = 0; u < KI; ++u) {
                const vec16 x = *reinterpret_cast<const vec16*>(sk + kTileBytes +
                                                                (u * NW + wave) * 1024 + lane * 16);
                if (rt0 + static_cast<int>(voff[u] / kRowBytes) < routed_rows)
                    store16_nt(reinterpret_cast<unsigned char*>(vdst) + voff[u], x);
            }
        }
    };
    // Tiles requested up front; with kGather a routed tile needs the group
    // ids in LDS, so those among them wait for the first barrier (all of
    // them when a split starts among the routed tiles).
    const int n_up = min(NS, t1 - t0);
    const int n_pre = kGather ? max(0, min(n_up, n_vis + 1 - t0)) : n_up;
#pragma unroll
    for (int s = 0; s < NS; ++s)
        if (s < n_pre) issue(t0 + s, s);

    f32x16_t oacc[NDT];
#pragma unroll
    for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
        for (int e = 0; e < 16; ++e) oacc[dt][e] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;  // m_run in scaled (log2) units

    // One key tile: wait for its copies, issue a later tile's, then the
    // tile's arithmetic.  Tiles 0 .. NS-1 were issued up front; from tile 1
    // on, tile + NS - 1 goes into the stage tile - 1 has freed.  The current
    // chunk (tile 0, under the causal mask) is a separate instantiation so
    // the other tiles carry no mask work.
    auto step = [&](int tile, auto current_tag) {
        constexpr bool kCurrent = decltype(current_tag)::value;
        const int lt = tile - t0;  // position in this workgroup's tiles
        // this wave's copies of `tile` are done once at most `ahead` later
        // tiles' copies remain in flight (loads complete in issue order)
        auto wait_ahead = [&](int ahead) {
            if (NS >= 4 && ahead >= 3)
                wait_loads<(NS >= 4 ? 3 : 0) * LPT>();
            else if (NS >= 3 && ahead >= 2)
                wait_loads<(NS >= 3 ? 2 : 0) * LPT>();
            else if (ahead >= 1)
                wait_loads<LPT>();
            else
                wait_loads<0>();
        };
        wait_ahead(lt == 0 ? n_pre - 1 : min(NS - 2, t1 - 1 - tile));
        __syncthreads();
        const bool write = kGather && tile > n_vis && (write_k || write_v);
        if (lt == 0) {
            for (int s = n_pre; s < n_up; ++s) issue(t0 + s, s);
            if (kGather && n_pre == 0) {  // nothing was in flight: wait for this tile now
                wait_ahead(n_up - 1);
                __syncthreads();
            }
            if (write) write_routed(tile, lt % NS);
        } else {
            if (write) write_routed(tile, lt % NS);
            if (tile + NS - 1 < t1) issue(tile + NS - 1, (lt + NS - 1) % NS);
        }

        const int stage = lt % NS;
        const bf16_t* sK = reinterpret_cast<const bf16_t*>(smem + stage * kStageBytes);
        const bf16_t* sV = reinterpret_cast<const bf16_t*>(smem + stage * kStageBytes + kTileBytes);
        const int rt_row0 = (tile - 1 - n_vis) * KT;
        const bool partial =
            !kCurrent && tile > n_vis &&
            routed_tile_partial(rt_row0, s_gid, routed_rows, topk_groups, group_shift, c * gpc);
        if (qactive)
            tile_math<D, KS, kCurrent>(sK, sV, qf, oacc, m_run, l_run, ksplit, t, partial, rt_row0,
                                       s_gid, routed_rows, topk_groups, group_shift, c * gpc);
    };
    if (t0 == 0) step(0, BoolTag<true>{});
    for (int tile = t0 > 1 ? t0 : 1; tile < t1; ++tile) step(tile, BoolTag<false>{});

    if constexpr (kSplit) {
        // Partial result of query row qrow_in_unit over this split's keys:
        // block (unit, split) of partial_ws holds rows x D unnormalised output
        // sums, then rows x (m, l) (m in log2 units, l the sum of the
        // weights exp2(s - m); m = -inf, l = 0 when the split saw no key).
        // A split with no tile never waited for its group-id copies: every
        // LDS copy is complete before the workgroup ends.
        wait_loads<0>();
        if (!qactive) return;
        const int rows = nqt * 32;
        float* blk = partial_ws + (unit * split_div.d + split) * static_cast<int64_t>(rows) * (D + 2);
        float* po = blk + static_cast<int64_t>(qrow_in_unit) * D;
#pragma unroll
        for (int dt = 0; dt < NDT; ++dt)
#pragma unroll
            for (int g4 = 0; g4 < 4; ++g4)
                *reinterpret_cast<float4*>(po + dt * 32 + g4 * 8 + half * 4) =
                    make_float4(oacc[dt][g4 * 4], oacc[dt][g4 * 4 + 1], oacc[dt][g4 * 4 + 2],
                                oacc[dt][g4 * 4 + 3]);
        const float l_tot = add_xor32(l_run);
        if (half == 0)
            *reinterpret_cast<float2*>(blk + static_cast<int64_t>(rows) * D + 2 * qrow_in_unit) =
                make_float2(m_run, bad ? NAN : l_tot);
        return;
    }
    __syncthreads();  // LDS stages are dead from here on (every copy was waited for)
    finish_rows<D, KS, QT>(oacc, m_run, l_run, reinterpret_cast<float*>(smem),
                           reinterpret_cast<float*>(smem) + QT * 64 * NDT * 16, qt_local, ksplit,
                           qactive, bad, out + qrow * D, lse ? lse + qrow : nullptr);
}

// Merge of the split partial results: thread (row, 4 dimensions) of one
// unit weighs split s by w_s = exp2(m_s - M), M = max_s m_s, and writes
// out = (sum_s w_s O_s) / L and lse = (M + log2 L) ln 2, L = sum_s w_s l_s
// (the same normalisation the single-workgroup kernel applies, with the
// partial sums added in split order).  All of a thread's reads are issued
// before any is used (kMaxSplit slots, the unused ones skipped).

template <int D>
__global__ __launch_bounds__(256) void attend_combine_kernel(
    const float* __restrict__ part, int n_split, int rows, int n_units, int n_q_chunks, int n_kv,
    int r, bf16_t* __restrict__ out, float* __restrict__ lse) {
    constexpr int TPR = D / 4;  // threads per row
    const int64_t gt = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    const int64_t row_g = gt / TPR;
    if (row_g >= static_cast<int64_t>(n_units) * rows) return;
    const int d0 = static_cast<int>(gt % TPR) * 4;
    const int unit = static_cast<int>(row_g / rows), qr = static_cast<int>(row_g % rows);
    const int64_t blk_floats = static_cast<int64_t>(rows) * (D + 2);
    const float* base = part + static_cast<int64_t>(unit) * n_split * blk_floats;
    float2 ml[kMaxSplit];
    float4 x[kMaxSplit];
#pragma unroll
    for (int s = 0; s < kMaxSplit; ++s) {
        if (s < n_split) {
            const float* blk = base + s * blk_floats;
            ml[s] = *reinterpret_cast<const float2*>(blk + static_cast<int64_t>(rows) * D + 2 * qr);
            x[s] = *reinterpret_cast<const float4*>(blk + static_cast<int64_t>(qr) * D + d0);
        }
    }
    float m_max = -INFINITY;
#pragma unroll
    for (int s = 0; s < kMaxSplit; ++s)
        if (s < n_split) m_max = fmaxf(m_max, ml[s].x);
    // a split that saw no key (m = -inf, l = 0) weighs exp2(-inf) = 0; M is
    // finite (split 0 holds each row's own token)
    float l_sum = 0.f;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int s = 0; s < kMaxSplit; ++s) {
        if (s < n_split) {
            const float w = __builtin_amdgcn_exp2f(ml[s].x - m_max);
            l_sum = fmaf(ml[s].y, w, l_sum);
            o.x = fmaf(x[s].x, w, o.x);
            o.y = fmaf(x[s].y, w, o.y);
            o.z = fmaf(x[s].z, w, o.z);
            o.w = fmaf(x[s].w, w, o.w);
        }
    }
    const float inv = __builtin_amdgcn_rcpf(l_sum);
    // output row: query head j*r + qr/64, token i*64 + qr%64 of the unit's chunk
    const int bh = unit / n_q_chunks, i = unit % n_q_chunks;
    const int b = bh / n_kv, j = bh % n_kv;
    const int64_t qrow = (static_cast<int64_t>(b) * n_kv * r + j * r + qr / KT) *
                             (static_cast<int64_t>(n_q_chunks) * KT) +
                         static_cast<int64_t>(i) * KT + qr % KT;
    typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
    bf16x4_t v;
    v[0] = static_cast<__bf16>(o.x * inv);
    v[1] = static_cast<__bf16>(o.y * inv);
    v[2] = static_cast<__bf16>(o.z * inv);
    v[3] = static_cast<__bf16>(o.w * inv);
    *reinterpret_cast<bf16x4_t*>(out + qrow * D + d0) = v;
    if (lse && d0 == 0) lse[qrow] = (m_max + log2f(l_sum)) * 0.6931471805599453f;
}

template <int D, int KS, int NS, int NW, bool kGather, bool kSplit = false>
hipError_t launch_mfma_t(const hga_plan& plan, hipStream_t stream, hipEvent_t ev_start,
                         hipEvent_t ev_stop, const bf16_t* q_rot, int q_chunk0, int n_q_chunks,
                         const bf16_t* k_res, const bf16_t* v_res, int64_t res_tokens,
                         const int32_t* res_slot, bf16_t* k_routed, bf16_t* v_routed,
                         const int32_t* group_idx, bf16_t* out, float* lse, int group_shift,
                         int wg_per_unit, int n_items, float* part = nullptr, int n_split = 1,
                         const bf16_t* k_src = nullptr, const bf16_t* v_src = nullptr,
                         int64_t src_tokens = 0) {
    const hga_params& p = plan.p;
    if (!k_src) {  // routed rows (kGather) from the resident K/V
        k_src = k_res;
        v_src = v_res;
        src_tokens = res_tokens;
    }
    constexpr uint32_t kLds = Layout<D, NS>::kBytes;
    static std::atomic<uint64_t> configured{0};  // per instantiation and device
    const hipError_t ce = once_per_device(configured, plan.device, [] {
        return hipFuncSetAttribute(
            reinterpret_cast<const void*>(&attend_mfma_kernel<D, KS, NS, NW, kGather, kSplit>),
            hipFuncAttributeMaxDynamicSharedMemorySize, static_cast<int>(kLds));
    });
    if (ce != hipSuccess) return ce;
    const int grid = (n_items + kXcds - 1) / kXcds * kXcds;
    hipExtLaunchKernelGGL((attend_mfma_kernel<D, KS, NS, NW, kGather, kSplit>), dim3(grid),
                          dim3(NW * 64), kLds, stream, ev_start, ev_stop, 0, q_rot, q_chunk0,
                          n_q_chunks, k_res, v_res, res_tokens, res_slot, k_routed, v_routed,
                          group_idx, out, lse, p.n_q_heads / p.n_kv_heads, FastDiv(p.n_kv_heads),
                          group_shift, p.keep_first, recent_window(p), p.topk_groups,
                          FastDiv(wg_per_unit), FastDiv(n_q_chunks), n_items, part,
                          FastDiv(n_split), k_src, v_src, src_tokens);
    return hipGetLastError();
}

// Launch shape of the grouped-query d128 kernel: eight wavefronts (eight
// query tiles) per workgroup, so each staged key tile serves twice the query
// rows of a four-wavefront workgroup (the VGPR budget allows one such
// workgroup per CU either way); two LDS stages (measured: 3.4% faster steps
// on `qwen32k` than four wavefronts; three or four stages no better).
constexpr int kD128Waves = 8;
constexpr int kD128Stages = 2;

template <bool kGather>
hipError_t launch_mfma_any(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                           const void* k_res, const void* v_res, int64_t res_tokens,
                           const int32_t* res_slot, void* k_routed, void* v_routed,
                           const int32_t* group_idx, void* out, float* lse, hipEvent_t ev_start,
                           hipEvent_t ev_stop, hipStream_t stream, const void* k_src = nullptr,
                           const void* v_src = nullptr, int64_t src_tokens = 0) {
    const hga_params& p = plan.p;
    const int r = p.n_q_heads / p.n_kv_heads;
    const int nqt = 2 * r;
    // One head per KV head (two query tiles): two wavefronts per query tile,
    // each with half of every key tile; otherwise one query tile per
    // wavefront.
    const bool one_head = nqt <= 2;
    const int qt_per_wg = p.head_dim == 128 ? kD128Waves : 4;
    const int wg_per_unit = one_head ? 1 : (nqt + qt_per_wg - 1) / qt_per_wg;
    const int64_t n_items64 =
        static_cast<int64_t>(p.batch) * p.n_kv_heads * n_q_chunks * wg_per_unit;
    if (n_items64 > (int64_t(1) << 30)) return hipErrorInvalidConfiguration;
    const int n_items = static_cast<int>(n_items64);
    const int group_shift = p.group == 8 ? 3 : (p.group == 16 ? 4 : 5);
    const bf16_t* q = static_cast<const bf16_t*>(q_rot);
    const bf16_t* kr = static_cast<const bf16_t*>(k_res);
    const bf16_t* vr = static_cast<const bf16_t*>(v_res);
    bf16_t* kt = static_cast<bf16_t*>(k_routed);
    bf16_t* vt = static_cast<bf16_t*>(v_routed);
    bf16_t* o = static_cast<bf16_t*>(out);
    const bf16_t* ks = static_cast<const bf16_t*>(k_src);
    const bf16_t* vs = static_cast<const bf16_t*>(v_src);
#define HGA_ARGS                                                                                 \
    plan, stream, ev_start, ev_stop, q, q_chunk0, n_q_chunks, kr, vr, res_tokens, res_slot, kt, \
        vt, group_idx, o, lse, group_shift, wg_per_unit, n_items, nullptr, 1, ks, vs, src_tokens
    if (p.head_dim == 64) {
        if (one_head) return launch_mfma_t<64, 2, 2, 4, kGather>(HGA_ARGS);
        return launch_mfma_t<64, 1, 2, 4, kGather>(HGA_ARGS);
    }
    if (one_head) return launch_mfma_t<128, 2, 2, 4, kGather>(HGA_ARGS);
    return launch_mfma_t<128, 1, kD128Stages, kD128Waves, kGather>(HGA_ARGS);
#undef HGA_ARGS
}

// Split form (GQA configurations, r >= 2): the launch shape of
// launch_mfma_any, each workgroup repeated for n_split key ranges, then the
// merge.  `part` holds units x n_split x rows x (D + 2) floats.  kGather:
// routed rows from k_src / v_src, written to k_routed / v_routed.
template <bool kGather>
hipError_t launch_split_any(const hga_plan& plan, const void* q_rot, int q_chunk0,
                            int n_q_chunks, const void* k_res, const void* v_res,
                            int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                            const void* v_routed, const int32_t* group_idx, void* out, float* lse,
                            float* part, int n_split, hipStream_t stream,
                            const void* k_src = nullptr, const void* v_src = nullptr,
                            int64_t src_tokens = 0) {
    const hga_params& p = plan.p;
    const int r = p.n_q_heads / p.n_kv_heads;
    const int qt_per_wg = p.head_dim == 128 ? kD128Waves : 4;
    const int wg_per_unit = (2 * r + qt_per_wg - 1) / qt_per_wg;
    const int n_units = p.batch * p.n_kv_heads * n_q_chunks;
    const int n_items = n_units * wg_per_unit * n_split;
    const int group_shift = p.group == 8 ? 3 : (p.group == 16 ? 4 : 5);
    const bf16_t* q = static_cast<const bf16_t*>(q_rot);
    const bf16_t* kr = static_cast<const bf16_t*>(k_res);
    const bf16_t* vr = static_cast<const bf16_t*>(v_res);
    bf16_t* kt = const_cast<bf16_t*>(static_cast<const bf16_t*>(k_routed));
    bf16_t* vt = const_cast<bf16_t*>(static_cast<const bf16_t*>(v_routed));
    bf16_t* o = static_cast<bf16_t*>(out);
    const bf16_t* ks = static_cast<const bf16_t*>(k_src);
    const bf16_t* vs = static_cast<const bf16_t*>(v_src);
    hipError_t e;
    if (p.head_dim == 64)
        e = launch_mfma_t<64, 1, 2, 4, kGather, true>(
            plan, stream, nullptr, nullptr, q, q_chunk0, n_q_chunks, kr, vr, res_tokens, res_slot,
            kt, vt, group_idx, o, lse, group_shift, wg_per_unit, n_items, part, n_split, ks, vs,
            src_tokens);
    else
        e = launch_mfma_t<128, 1, kD128Stages, kD128Waves, kGather, true>(
            plan, stream, nullptr, nullptr, q, q_chunk0, n_q_chunks, kr, vr, res_tokens, res_slot,
            kt, vt, group_idx, o, lse, group_shift, wg_per_unit, n_items, part, n_split, ks, vs,
            src_tokens);
    if (e != hipSuccess) return e;
    const int rows = 64 * r;
    const int64_t threads = static_cast<int64_t>(n_units) * rows * (p.head_dim / 4);
    const int blocks = static_cast<int>((threads + 255) / 256);
    if (p.head_dim == 64)
        hipLaunchKernelGGL((attend_combine_kernel<64>), dim3(blocks), dim3(256), 0, stream, part,
                           n_split, rows, n_units, n_q_chunks, p.n_kv_heads, r, o, lse);
    else
        hipLaunchKernelGGL((attend_combine_kernel<128>), dim3(blocks), dim3(256), 0, stream, part,
                           n_split, rows, n_units, n_q_chunks, p.n_kv_heads, r, o, lse);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attend_valu(const hga_plan& plan, const void* q_rot, int q_chunk0,
                              int n_q_chunks, const void* k_res, const void* v_res,
                              int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                              const void* v_routed, const int32_t* group_idx, void* out,
                              float* lse, hipEvent_t ev_start, hipEvent_t ev_stop,
                              hipStream_t stream, const void* k_src = nullptr,
                              const void* v_src = nullptr, int64_t src_tokens = 0);

int64_t attend_split_bytes_per_split(const hga_plan& plan, int n_q_chunks) {
    const hga_params& p = plan.p;
    const int64_t rows = 64 * (p.n_q_heads / p.n_kv_heads);
    return static_cast<int64_t>(p.batch) * p.n_kv_heads * n_q_chunks * rows * (p.head_dim + 2) *
           static_cast<int64_t>(sizeof(float));
}

bool attend_split_applies(const hga_plan& plan) {
    return plan.p.dtype == HGA_BF16 && plan.p.n_q_heads / plan.p.n_kv_heads >= 2;
}

// Splits for a launch of n_q_chunks query chunks from q_chunk0: enough
// workgroups to give every compute unit one, at least two key tiles per
// split, at most what the workspace holds; 1 where the split form does not
// apply (fp32, one query head per KV head).
static int choose_splits(const hga_plan& plan, int q_chunk0, int n_q_chunks,
                         int64_t workspace_bytes) {
    const hga_params& p = plan.p;
    const int r = p.n_q_heads / p.n_kv_heads;
    int n_split = 1;
    if (attend_split_applies(plan)) {
        // enough workgroups to give every compute unit one, at least two key
        // tiles per split, at most what the workspace holds
        const int qt_per_wg = p.head_dim == 128 ? kD128Waves : 4;
        const int wg_per_unit = (2 * r + qt_per_wg - 1) / qt_per_wg;
        const int64_t items = static_cast<int64_t>(p.batch) * p.n_kv_heads * n_q_chunks * wg_per_unit;
        const int c_last = q_chunk0 + n_q_chunks - 1;
        const int n_rt = (p.topk_groups * p.group + KT - 1) / KT;
        const int n_tiles = 1 + VisibleChunks(c_last, p.keep_first, recent_window(p)).count + n_rt;
        int64_t want = (plan.n_cu + items - 1) / items;
        want = want < (n_tiles + 1) / 2 ? want : (n_tiles + 1) / 2;
        want = want < kMaxSplit ? want : kMaxSplit;
        const int64_t per = attend_split_bytes_per_split(plan, n_q_chunks);
        const int64_t fit = per > 0 ? workspace_bytes / per : 0;
        n_split = static_cast<int>(want < fit ? want : fit);
    }
    return n_split;
}

hipError_t launch_attend_split(const hga_plan& plan, const void* q_rot, int q_chunk0,
                               int n_q_chunks, const void* k_res, const void* v_res,
                               int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                               const void* v_routed, const int32_t* group_idx, void* out,
                               float* lse, void* workspace, int64_t workspace_bytes,
                               hipStream_t stream) {
    const int n_split = choose_splits(plan, q_chunk0, n_q_chunks, workspace_bytes);
    if (n_split <= 1)
        return launch_attend(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                             res_slot, k_routed, v_routed, group_idx, out, lse, nullptr, nullptr,
                             stream);
    return launch_split_any<false>(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                   res_slot, k_routed, v_routed, group_idx, out, lse,
                                   static_cast<float*>(workspace), n_split, stream);
}

hipError_t launch_gather_attend_split(const hga_plan& plan, const void* q_rot, int q_chunk0,
                                      int n_q_chunks, const void* k_res, const void* v_res,
                                      int64_t res_tokens, const int32_t* res_slot,
                                      const void* k_src, const void* v_src, int64_t src_tokens,
                                      const int32_t* group_idx, void* k_routed, void* v_routed,
                                      void* out, float* lse, void* workspace,
                                      int64_t workspace_bytes, hipStream_t stream) {
    const hga_params& p = plan.p;
    if (p.dtype == HGA_F32) {
        // the gather kernel, then the attention reading its output; without
        // routed buffers the attention reads the routed rows from k_src/v_src
        if (k_routed) {
            const hipError_t e = launch_gather_kv(plan, group_idx, q_chunk0, n_q_chunks, k_src,
                                                  v_src, src_tokens, k_routed, v_routed, stream);
            if (e != hipSuccess) return e;
        }
        return launch_attend_valu(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                  res_slot, k_routed, v_routed, group_idx, out, lse, nullptr,
                                  nullptr, stream, k_src, v_src, src_tokens);
    }
    const int n_split = choose_splits(plan, q_chunk0, n_q_chunks, workspace_bytes);
    if (n_split <= 1)
        return launch_mfma_any<true>(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                     res_slot, k_routed, v_routed, group_idx, out, lse, nullptr,
                                     nullptr, stream, k_src, v_src, src_tokens);
    return launch_split_any<true>(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                  res_slot, k_routed, v_routed, group_idx, out, lse,
                                  static_cast<float*>(workspace), n_split, stream, k_src, v_src,
                                  src_tokens);
}


hipError_t launch_attend(const hga_plan& plan, const void* q_rot, int q_chunk0, int n_q_chunks,
                         const void* k_res, const void* v_res, int64_t res_tokens,
                         const int32_t* res_slot, const void* k_routed, const void* v_routed,
                         const int32_t* group_idx, void* out, float* lse, hipEvent_t ev_start,
                         hipEvent_t ev_stop, hipStream_t stream) {
    if (plan.p.dtype == HGA_F32)
        return launch_attend_valu(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                  res_slot, k_routed, v_routed, group_idx, out, lse, ev_start,
                                  ev_stop, stream);
    // the routed buffers are only read on this path
    return launch_mfma_any<false>(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                  res_slot, const_cast<void*>(k_routed),
                                  const_cast<void*>(v_routed), group_idx, out, lse, ev_start,
                                  ev_stop, stream);
}

hipError_t launch_gather_attend(const hga_plan& plan, const void* q_rot, int q_chunk0,
                                int n_q_chunks, const void* k_res, const void* v_res,
                                int64_t res_tokens, const int32_t* group_idx, void* k_routed,
                                void* v_routed, void* out, float* lse, hipEvent_t ev_start,
                                hipEvent_t ev_stop, hipStream_t stream) {
    if (plan.p.dtype == HGA_F32) {
        // fp32: the gather kernel, then the attention kernel reading its
        // output; without routed buffers the attention kernel reads each
        // routed row from the resident K/V itself
        if (k_routed) {
            const hipError_t e = launch_gather_kv(plan, group_idx, q_chunk0, n_q_chunks, k_res,
                                                  v_res, res_tokens, k_routed, v_routed, stream);
            if (e != hipSuccess) return e;
        }
        return launch_attend_valu(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                  nullptr, k_routed, v_routed, group_idx, out, lse, ev_start,
                                  ev_stop, stream, k_res, v_res, res_tokens);
    }
    return launch_mfma_any<true>(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens,
                                 nullptr, k_routed, v_routed, group_idx, out, lse, ev_start,
                                 ev_stop, stream);
}

}  // namespace hga
