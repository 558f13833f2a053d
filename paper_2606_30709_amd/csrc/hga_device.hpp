// Device-side helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hga {

typedef uint16_t bf16_t;  // bfloat16 storage

struct alignas(16) vec16 {  // one 16-byte load/store
    uint32_t w[4];
};

__device__ __forceinline__ float bf16_to_f32(bf16_t x) {
    return __uint_as_float(static_cast<uint32_t>(x) << 16);
}

// Round-to-nearest-even; NaN stays a quiet NaN.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<bf16_t>((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return static_cast<bf16_t>(u >> 16);
}

// Element type traits: how many elements one 16-byte vector holds and how
// to widen them to fp32.
template <typename T> struct elem;

template <> struct elem<float> {
    static constexpr int kVec = 4;
    __device__ static __forceinline__ void unpack(const vec16& v, float* out) {
#pragma unroll
        for (int e = 0; e < 4; ++e) out[e] = __uint_as_float(v.w[e]);
    }
    __device__ static __forceinline__ float to_f32(float x) { return x; }
    __device__ static __forceinline__ float from_f32(float x) { return x; }
};

template <> struct elem<bf16_t> {
    static constexpr int kVec = 8;
    __device__ static __forceinline__ void unpack(const vec16& v, float* out) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            out[2 * e] = __uint_as_float(v.w[e] << 16);
            out[2 * e + 1] = __uint_as_float(v.w[e] & 0xffff0000u);
        }
    }
    __device__ static __forceinline__ float to_f32(bf16_t x) { return bf16_to_f32(x); }
    __device__ static __forceinline__ bf16_t from_f32(float x) { return f32_to_bf16(x); }
};

// Division of n in [0, 2^31) by a divisor d in [1, 2^31) fixed for a whole
// launch, by one high multiply, one add and one shift (Granlund and
// Montgomery, "Division by invariant integers using multiplication", 1994):
// with s = ceil(log2 d) and m = floor(2^32 (2^s - d) / d) + 1,
// floor(n / d) = (mulhi(n, m) + n) >> s.  (m + 2^32 = floor(2^(32+s)/d) + 1
// exceeds 2^(32+s)/d by at most 1, an error below 1/d for every n < 2^31;
// the sum stays below 2^32.)  Built on the host, passed by value.
struct FastDiv {
    uint32_t d, m, s;
    __host__ __device__ FastDiv() : d(1), m(1), s(0) {}
    __host__ explicit FastDiv(uint32_t div) : d(div), m(0), s(0) {
        while ((uint32_t(1) << s) < d) ++s;
        m = static_cast<uint32_t>(((uint64_t(1) << 32) * ((uint64_t(1) << s) - d)) / d + 1);
    }
    __device__ __forceinline__ uint32_t div(uint32_t n) const {
        return (__umulhi(n, m) + n) >> s;
    }
};

__device__ __forceinline__ vec16 load16(const void* p) {
    return *reinterpret_cast<const vec16*>(p);
}

__device__ __forceinline__ void store16(void* p, const vec16& v) {
    *reinterpret_cast<vec16*>(p) = v;
}

// Raw buffer access: a resource descriptor covers [base, base + bytes); a load
// whose offset falls outside returns zeros without touching memory.  Loads
// through it never need a branch, so their wait counts stay exact.
typedef __amdgpu_buffer_rsrc_t buf_rsrc;

__device__ __forceinline__ buf_rsrc make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, static_cast<int>(bytes),
                                             0x00020000);
}

__device__ __forceinline__ vec16 buf_load16(buf_rsrc r, uint32_t offset) {
    return __builtin_bit_cast(vec16, __builtin_amdgcn_raw_buffer_load_b128(r, offset, 0, 0));
}

__device__ __forceinline__ int buf_load_i32(buf_rsrc r, uint32_t offset) {
    return static_cast<int>(__builtin_amdgcn_raw_buffer_load_b32(r, offset, 0, 0));
}

// Total order on fp32 scores as unsigned keys; -0 is folded into +0 by the
// caller (score + 0.0f) so equal scores compare equal.
__device__ __forceinline__ uint32_t orderable(float s) {
    uint32_t u = __float_as_uint(s);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Packed selection key: larger score first, then smaller index.
__device__ __forceinline__ uint64_t select_key(float score, int idx) {
    return (static_cast<uint64_t>(orderable(score + 0.0f)) << 32) |
           static_cast<uint64_t>(0xffffffffu - static_cast<uint32_t>(idx));
}

__device__ __forceinline__ int key_index(uint64_t key) {
    return static_cast<int>(0xffffffffu - static_cast<uint32_t>(key & 0xffffffffu));
}

// x combined (max) with the value DPP control kCtrl moves into this lane;
// lanes that receive nothing (outside the row, or rows outside kRowMask) see 0,
// the smallest unsigned value.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t max_dpp(uint32_t x) {
    const uint32_t o = static_cast<uint32_t>(
        __builtin_amdgcn_update_dpp(0, static_cast<int>(x), kCtrl, kRowMask, 0xf, true));
    return o > x ? o : x;
}

// Wave-wide maximum of an unsigned value, uniform result.  Within each
// 16-lane row, shifts by 1, 2, 4, 8 leave the row maximum in the row's lane
// 15; row broadcasts 15 and 31 carry it into rows 1..3, and lane 63 ends with
// the maximum of the wave.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    x = max_dpp<0x111, 0xf>(x);  // row_shr:1
    x = max_dpp<0x112, 0xf>(x);  // row_shr:2
    x = max_dpp<0x114, 0xf>(x);  // row_shr:4
    x = max_dpp<0x118, 0xf>(x);  // row_shr:8
    x = max_dpp<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
    x = max_dpp<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
    return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(x), 63));
}

// x plus the value DPP control kCtrl moves into this lane (0 where nothing
// arrives: outside the row, or rows outside kRowMask).
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int add_dpp(int x) {
    return x + __builtin_amdgcn_update_dpp(0, x, kCtrl, kRowMask, 0xf, true);
}

// Inclusive prefix sum over the wave's lanes (lane l gets the sum of lanes
// 0..l): the steps of wave_max_u32 with addition -- shifts by 1, 2, 4, 8
// scan each 16-lane row, then row 0's total goes into rows 1 and 3 and the
// total of rows 0..1 into rows 2 and 3.
__device__ __forceinline__ int wave_incl_scan_add(int x) {
    x = add_dpp<0x111, 0xf>(x);  // row_shr:1
    x = add_dpp<0x112, 0xf>(x);  // row_shr:2
    x = add_dpp<0x114, 0xf>(x);  // row_shr:4
    x = add_dpp<0x118, 0xf>(x);  // row_shr:8
    x = add_dpp<0x142, 0xa>(x);  // row_bcast:15 into rows 1 and 3
    x = add_dpp<0x143, 0xc>(x);  // row_bcast:31 into rows 2 and 3
    return x;
}

// Wave-wide maximum of a 64-bit key: the high words first, then the low
// words of the lanes holding that high word -- read straight from that lane
// when only one holds it, the usual case.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
    const uint32_t hi = static_cast<uint32_t>(x >> 32);
    const uint32_t top_hi = wave_max_u32(hi);
    const uint64_t holders = __builtin_amdgcn_ballot_w64(hi == top_hi);
    uint32_t top_lo;
    if ((holders & (holders - 1)) == 0)
        top_lo = static_cast<uint32_t>(__builtin_amdgcn_readlane(
            static_cast<int>(static_cast<uint32_t>(x)), static_cast<int>(__builtin_ctzll(holders))));
    else
        top_lo = wave_max_u32(hi == top_hi ? static_cast<uint32_t>(x) : 0u);
    return (static_cast<uint64_t>(top_hi) << 32) | top_lo;
}

// Top-k selection by one wavefront over `n` packed keys in LDS (keys are
// never zero; zero marks a taken key).  Writes the k selected indices, in
// ascending order, to sel[0..k) (LDS).  All 64 lanes of the wave must call.
// Each round takes the wave-wide maximum of the lanes' best keys; the winning
// lane drops it and rescans its share.
__device__ inline void wave_select_topk_lds(uint64_t* keys, int n, int k, int* sel, int* scratch) {
    const int lane = threadIdx.x & 63;
    uint64_t best = 0;
    int best_pos = -1;
    for (int i = lane; i < n; i += 64) {
        uint64_t v = keys[i];
        if (v > best) { best = v; best_pos = i; }
    }
    for (int round = 0; round < k; ++round) {
        uint64_t top = wave_max_u64(best);
        if (best == top && best_pos >= 0) {
            scratch[round] = key_index(top);
            keys[best_pos] = 0;
            best = 0;
            best_pos = -1;
            for (int i = lane; i < n; i += 64) {
                uint64_t v = keys[i];
                if (v > best) { best = v; best_pos = i; }
            }
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // ascending order: rank of each winner among the k winners
    for (int i = lane; i < k; i += 64) {
        int v = scratch[i];
        int rank = 0;
        for (int j = 0; j < k; ++j) rank += scratch[j] < v;
        sel[rank] = v;
    }
}

// The same selection for n <= 64 * R keys and k <= 64, with each lane's
// share of the keys held in registers: a round is one wave maximum and a
// register rescan, and winner `round` is kept by lane `round`.
template <int R>
__device__ __forceinline__ void wave_select_topk_regs(const uint64_t* keys, int n, int k,
                                                      int* sel) {
    const int lane = threadIdx.x & 63;
    uint64_t v[R];
#pragma unroll
    for (int t = 0; t < R; ++t) v[t] = lane + 64 * t < n ? keys[lane + 64 * t] : 0;
    int mine = 0x7fffffff;
    for (int round = 0; round < k; ++round) {
        uint64_t best = v[0];
#pragma unroll
        for (int t = 1; t < R; ++t) best = v[t] > best ? v[t] : best;
        const uint64_t top = wave_max_u64(best);
#pragma unroll
        for (int t = 0; t < R; ++t) v[t] = v[t] == top ? 0 : v[t];
        if (lane == round) mine = key_index(top);
    }
    int rank = 0;
    for (int j = 0; j < k; ++j) rank += __builtin_amdgcn_readlane(mine, j) < mine;
    if (lane < k) sel[rank] = mine;
}

// The same selection by a threshold instead of k rounds, for larger k: the
// k-th largest score T (the high words) is found bit by bit from the most
// significant one -- T grows by a bit while at least k keys stay >= T, a
// ballot count per bit -- then every key above T is taken and, of the keys
// equal to T, the first k - (#above) in position order (equal scores go to
// the lower index).  Positions are then compacted in order, so the output is
// ascending by position; callers whose ids increase with the position (both
// routing stages) get ascending ids, as from the rounds.  n <= 64 * R keys,
// k <= n.
template <int R>
__device__ __forceinline__ void wave_select_topk_threshold(const uint64_t* keys, int n, int k,
                                                           int* sel) {
    const int lane = threadIdx.x & 63;
    uint32_t hi[R], id[R];
#pragma unroll
    for (int t = 0; t < R; ++t) {
        const uint64_t v = lane + 64 * t < n ? keys[lane + 64 * t] : 0;
        hi[t] = static_cast<uint32_t>(v >> 32);  // 0 marks no key; real keys are above 0
        id[t] = static_cast<uint32_t>(key_index(v));
    }
    uint32_t T = 0;
    for (int b = 31; b >= 0; --b) {
        const uint32_t cand = T | (1u << b);
        int cnt = 0;
#pragma unroll
        for (int t = 0; t < R; ++t) cnt += __popcll(__builtin_amdgcn_ballot_w64(hi[t] >= cand));
        if (cnt >= k) T = cand;
    }
    int need = k;
#pragma unroll
    for (int t = 0; t < R; ++t) need -= __popcll(__builtin_amdgcn_ballot_w64(hi[t] > T));
    int base = 0;
    const uint64_t below = (uint64_t(1) << lane) - 1;
#pragma unroll
    for (int t = 0; t < R; ++t) {
        // a tied key is taken when fewer than `need` ties precede it
        const bool eq = hi[t] == T;
        const uint64_t eqm = __builtin_amdgcn_ballot_w64(eq);
        const bool pick = hi[t] > T || (eq && __popcll(eqm & below) < need);
        const uint64_t m = __builtin_amdgcn_ballot_w64(pick);
        if (pick) sel[base + __popcll(m & below)] = static_cast<int>(id[t]);
        base += __popcll(m);
        const int ne = __popcll(eqm);
        need -= ne < need ? ne : need;
    }
}

// Dispatch on size; every form selects the same keys and writes them in
// ascending id order.  The threshold form (for k >= 8, where k rounds cost
// more than its 32 steps) needs ids that increase with the position
// (`ids_by_position`); the others sort by id themselves.
__device__ __forceinline__ void wave_select_topk(uint64_t* keys, int n, int k, int* sel,
                                                 int* scratch, bool ids_by_position = false) {
    if (ids_by_position && k >= 8 && n <= 64 * 16) {
        if (n <= 64 * 2)
            wave_select_topk_threshold<2>(keys, n, k, sel);
        else if (n <= 64 * 4)
            wave_select_topk_threshold<4>(keys, n, k, sel);
        else if (n <= 64 * 8)
            wave_select_topk_threshold<8>(keys, n, k, sel);
        else
            wave_select_topk_threshold<16>(keys, n, k, sel);
    } else if (k <= 64 && n <= 64)
        wave_select_topk_regs<1>(keys, n, k, sel);
    else if (k <= 64 && n <= 64 * 2)
        wave_select_topk_regs<2>(keys, n, k, sel);
    else if (k <= 64 && n <= 64 * 4)
        wave_select_topk_regs<4>(keys, n, k, sel);
    else if (k <= 64 && n <= 64 * 8)
        wave_select_topk_regs<8>(keys, n, k, sel);
    else if (k <= 64 && n <= 64 * 16)
        wave_select_topk_regs<16>(keys, n, k, sel);
    else
        wave_select_topk_lds(keys, n, k, sel, scratch);
}

}  // namespace hga
