// Host side of the C ABI: plan creation, argument validation before any
// launch, status codes and the per-thread error message.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <new>
#include <string>
#include <vector>

#include "hga.h"
#include "attend_common.hpp"
#include "hga_internal.hpp"

namespace {

// Largest byte extent of one head's slab the kernels address (32-bit
// offsets, with room above for the "absent" marker offset).
constexpr int64_t kMaxSlabBytes = 0xfff00000ll;


thread_local std::string g_last_error;

hga_status fail(hga_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

hga_status hip_fail(hipError_t e, const char* what) {
    return fail(HGA_EHIP, "%s: %s (%d)", what, hipGetErrorString(e), static_cast<int>(e));
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Pair p is high-frequency for a span when its wavelength 2*pi/theta_p is at
// most the span (Sec. 3.2 leaves the split open; this is the rule used).
int high_freq_pairs(int span, int head_dim, double base) {
    int n = 0;
    for (int p = 0; p < head_dim / 2; ++p) {
        const double theta = std::pow(base, -2.0 * p / head_dim);
        if (2.0 * M_PI / theta <= static_cast<double>(span)) ++n;
    }
    return n;
}

// cos and sin of phi_p(o) = ((span - 1)/2 - o) * theta_p for low-frequency
// pairs and 0 for high-frequency ones, in double, stored as fp32
// [2][span][head_dim/2].
std::vector<float> phase_table(int span, int head_dim, double base, int n_hf) {
    const int half = head_dim / 2;
    std::vector<float> t(2 * static_cast<size_t>(span) * half);
    for (int o = 0; o < span; ++o)
        for (int p = 0; p < half; ++p) {
            double phi = 0.0;
            if (p >= n_hf) phi = ((span - 1) / 2.0 - o) * std::pow(base, -2.0 * p / head_dim);
            t[static_cast<size_t>(o) * half + p] = static_cast<float>(std::cos(phi));
            t[static_cast<size_t>(span + o) * half + p] = static_cast<float>(std::sin(phi));
        }
    return t;
}

// cos and sin of psi_g theta_p, psi_g = (chunk - group)/2 - g*group: the
// rotation taking group g's middle position to the chunk's middle position
// (used for the low-frequency chunk pairs), [2][chunk/group][head_dim/2].
std::vector<float> psi_table(int chunk, int group, int head_dim, double base) {
    const int half = head_dim / 2, gpc = chunk / group;
    std::vector<float> t(2 * static_cast<size_t>(gpc) * half);
    for (int g = 0; g < gpc; ++g)
        for (int p = 0; p < half; ++p) {
            const double psi = ((chunk - group) / 2.0 - g * group) * std::pow(base, -2.0 * p / head_dim);
            t[static_cast<size_t>(g) * half + p] = static_cast<float>(std::cos(psi));
            t[static_cast<size_t>(gpc + g) * half + p] = static_cast<float>(std::sin(psi));
        }
    return t;
}

hga_status validate_params(const hga_params* p) {
    if (!p) return fail(HGA_EINVAL, "params is NULL");
    if (p->batch < 1 || p->n_q_heads < 1 || p->n_kv_heads < 1)
        return fail(HGA_EINVAL, "batch, n_q_heads and n_kv_heads must be >= 1");
    if (p->n_q_heads % p->n_kv_heads != 0)
        return fail(HGA_EINVAL, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)",
                    p->n_q_heads, p->n_kv_heads);
    if (p->n_q_heads / p->n_kv_heads > 16)
        return fail(HGA_EUNSUPPORTED, "GQA ratio %d above 16 is not supported",
                    p->n_q_heads / p->n_kv_heads);
    if (static_cast<int64_t>(p->batch) * p->n_kv_heads > 65535)
        return fail(HGA_EUNSUPPORTED, "batch * n_kv_heads above 65535 is not supported");
    if (p->head_dim != 64 && p->head_dim != 128)
        return fail(HGA_EUNSUPPORTED, "head_dim %d not supported (64 or 128)", p->head_dim);
    if (p->chunk != 64) return fail(HGA_EUNSUPPORTED, "chunk %d not supported (64)", p->chunk);
    if (p->group != 8 && p->group != 16 && p->group != 32)
        return fail(HGA_EUNSUPPORTED, "group %d not supported (8, 16 or 32)", p->group);
    if (p->keep_first < 0 || p->keep_last < 0)
        return fail(HGA_EINVAL, "keep_first and keep_last must be >= 0");
    if (p->force_prev != 0 && p->force_prev != 1)
        return fail(HGA_EINVAL, "force_prev must be 0 or 1");
    if (p->topk_chunks < 1 || p->topk_chunks > hga::kMaxTopK)
        return fail(HGA_EINVAL, "topk_chunks must be in [1, %d]", hga::kMaxTopK);
    if (p->topk_groups < 1 || p->topk_groups > hga::kMaxTopK)
        return fail(HGA_EINVAL, "topk_groups must be in [1, %d]", hga::kMaxTopK);
    if (p->hf_pairs_chunk < -1 || p->hf_pairs_chunk > p->head_dim / 2 ||
        p->hf_pairs_group < -1 || p->hf_pairs_group > p->head_dim / 2)
        return fail(HGA_EINVAL, "hf_pairs_* must be -1 or in [0, head_dim/2]");
    if (p->dtype != HGA_F32 && p->dtype != HGA_BF16)
        return fail(HGA_EINVAL, "dtype must be HGA_F32 or HGA_BF16");
    if (!(p->rope_base > 1.0) || !std::isfinite(p->rope_base))
        return fail(HGA_EINVAL, "rope_base must be finite and > 1");
    return HGA_OK;
}

hga_status check_plan(const hga_plan* plan) {
    if (!plan) return fail(HGA_EINVAL, "plan is NULL");
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != plan->device)
        return fail(HGA_EINVAL, "current device %d is not the plan's device %d", dev, plan->device);
    return HGA_OK;
}

hga_status check_tensor(const void* p, const char* name) {
    if (!p) return fail(HGA_EINVAL, "%s is NULL", name);
    if (!aligned(p, 16)) return fail(HGA_EALIGN, "%s is not 16-byte aligned", name);
    return HGA_OK;
}

// Most slots a warm-cache partition may have (its LRU keys live in LDS).
constexpr int32_t kMaxCacheSlots = 8192;

// A caller workspace: NULL with 0 bytes, or 16-byte aligned with > 0 bytes.
hga_status check_workspace(const void* workspace, int64_t workspace_bytes) {
    if (workspace_bytes < 0) return fail(HGA_EINVAL, "workspace_bytes must be >= 0");
    if (workspace_bytes > 0) {
        if (!workspace) return fail(HGA_EINVAL, "workspace is NULL with workspace_bytes > 0");
        if (!aligned(workspace, 16)) return fail(HGA_EALIGN, "workspace is not 16-byte aligned");
    }
    return HGA_OK;
}

hga_status check_index(const void* p, const char* name) {
    if (!p) return fail(HGA_EINVAL, "%s is NULL", name);
    if (!aligned(p, 4)) return fail(HGA_EALIGN, "%s is not 4-byte aligned", name);
    return HGA_OK;
}

hga_status launched(hipError_t e, const char* what) {
    if (e != hipSuccess) return hip_fail(e, what);
    return HGA_OK;
}

// A launch reports its error through hipGetLastError(), which also returns
// errors that earlier, unrelated runtime calls on this thread left behind;
// clear those first so a launch is charged only with its own failure.
void clear_stale_error() { (void)hipGetLastError(); }

#define HGA_TRY(x)                      \
    do {                                \
        hga_status st_ = (x);           \
        if (st_ != HGA_OK) return st_;  \
    } while (0)

}  // namespace

extern "C" {

int32_t hga_version(void) { return (1 << 16) | 0; }

int32_t hga_visible_chunks(const hga_params* params, int32_t c, int32_t* chunks, int32_t cap) {
    HGA_TRY(validate_params(params));
    if (c < 0 || cap < 0) return fail(HGA_EINVAL, "c and cap must be >= 0");
    if (cap > 0 && !chunks) return fail(HGA_EINVAL, "chunks is NULL");
    // the enumeration the attention kernels use
    const hga::VisibleChunks vis(c, params->keep_first, hga::recent_window(*params));
    for (int idx = 0; idx < vis.count && idx < cap; ++idx) chunks[idx] = vis.chunk(idx);
    clear_stale_error();
    return vis.count;
}

const char* hga_status_string(int32_t status) {
    switch (status) {
        case HGA_OK: return "HGA_OK: success";
        case HGA_EINVAL: return "HGA_EINVAL: invalid argument";
        case HGA_EUNSUPPORTED: return "HGA_EUNSUPPORTED: valid but not supported by the kernels";
        case HGA_EALIGN: return "HGA_EALIGN: misaligned pointer";
        case HGA_EHIP: return "HGA_EHIP: HIP runtime error";
        default: return "unknown hga_status";
    }
}

const char* hga_last_error(void) { return g_last_error.c_str(); }

hga_status hga_plan_create(const hga_params* params, hga_plan** plan) {
    if (!plan) return fail(HGA_EINVAL, "plan out-pointer is NULL");
    HGA_TRY(validate_params(params));
    hga_params p = *params;
    if (p.hf_pairs_chunk < 0) p.hf_pairs_chunk = high_freq_pairs(p.chunk, p.head_dim, p.rope_base);
    if (p.hf_pairs_group < 0) p.hf_pairs_group = high_freq_pairs(p.group, p.head_dim, p.rope_base);
    if (p.hf_pairs_chunk < p.hf_pairs_group)
        return fail(HGA_EUNSUPPORTED, "hf_pairs_chunk (%d) below hf_pairs_group (%d) is not "
                    "supported: a high-frequency group pair must be high-frequency for the chunk",
                    p.hf_pairs_chunk, p.hf_pairs_group);
    const std::vector<float> tg = phase_table(p.group, p.head_dim, p.rope_base, p.hf_pairs_group);
    const std::vector<float> tc = psi_table(p.chunk, p.group, p.head_dim, p.rope_base);

    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    int max_lds = 0;
    e = hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    int n_cu = 0;
    e = hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    // the device's copy of the library's static scratch (allocation-free split
    // attention): its address, taken once per device with the device current
    e = hga::static_scratch_init(dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (static scratch)");
    hga_plan* pl = new (std::nothrow) hga_plan();
    if (!pl) return fail(HGA_EINVAL, "out of host memory");
    pl->p = p;
    pl->device = dev;
    pl->max_lds = max_lds;
    pl->n_cu = n_cu;
    float* buf = nullptr;
    const size_t bytes = (tc.size() + tg.size()) * sizeof(float);
    e = hipMalloc(&buf, bytes);
    if (e != hipSuccess) {
        delete pl;
        return hip_fail(e, "hipMalloc (phase tables)");
    }
    e = hipMemcpy(buf, tg.data(), tg.size() * sizeof(float), hipMemcpyHostToDevice);
    if (e == hipSuccess)
        e = hipMemcpy(buf + tg.size(), tc.data(), tc.size() * sizeof(float), hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(buf);
        delete pl;
        return hip_fail(e, "hipMemcpy (phase tables)");
    }
    pl->phase_group = buf;
    pl->phase_psi = buf + tg.size();
    // the spread routing form's workspace: keys, then per-unit counters that
    // start at zero (each call leaves them at zero)
    void* ws = nullptr;
    e = hipMalloc(&ws, hga::route_workspace_bytes());
    if (e == hipSuccess) {
        pl->route_keys = static_cast<uint64_t*>(ws);
        pl->route_count = reinterpret_cast<unsigned*>(
            static_cast<unsigned char*>(ws) +
            sizeof(uint64_t) * hga::kRouteSpreadUnits * hga::kRouteSpreadCandidates);
        // a synchronous copy of zeros (no device-wide synchronisation)
        const unsigned zeros[hga::kRouteSpreadUnits] = {};
        e = hipMemcpy(pl->route_count, zeros, sizeof(zeros), hipMemcpyHostToDevice);
    }
    if (e != hipSuccess) {
        (void)hipFree(ws);
        (void)hipFree(buf);
        delete pl;
        return hip_fail(e, "hipMalloc/hipMemcpy (routing workspace)");
    }
    *plan = pl;
    return HGA_OK;
}

hga_status hga_plan_destroy(hga_plan* plan) {
    if (!plan) return HGA_OK;
    hipError_t e = hipFree(plan->phase_group);
    const hipError_t e2 = hipFree(plan->route_keys);
    if (e == hipSuccess) e = e2;
    delete plan;
    if (e != hipSuccess) return hip_fail(e, "hipFree (phase tables)");
    return HGA_OK;
}

hga_status hga_plan_params(const hga_plan* plan, hga_params* out) {
    if (!plan || !out) return fail(HGA_EINVAL, "plan or out is NULL");
    *out = plan->p;
    return HGA_OK;
}

namespace {

// Checks of a summary build; *empty is set when the chunk range is empty.
hga_status check_summaries(const hga_plan* plan, const void* k_rot, int64_t k_tokens,
                           int32_t k_chunk0, int32_t chunk_begin, int32_t chunk_end,
                           float* chunk_sum, float* group_sum, int32_t table_chunks, bool* empty) {
    HGA_TRY(check_plan(plan));
    const hga_params& p = plan->p;
    if (k_tokens < 0 || k_chunk0 < 0 || table_chunks < 0)
        return fail(HGA_EINVAL, "k_tokens, k_chunk0 and table_chunks must be >= 0");
    if (chunk_begin < k_chunk0 || chunk_end < chunk_begin || chunk_end > table_chunks)
        return fail(HGA_EINVAL, "need k_chunk0 <= chunk_begin <= chunk_end <= table_chunks "
                    "(got %d, %d, %d, %d)", k_chunk0, chunk_begin, chunk_end, table_chunks);
    if (static_cast<int64_t>(chunk_end - k_chunk0) * p.chunk > k_tokens)
        return fail(HGA_EINVAL, "chunks up to %d need %lld tokens of k_rot, have %lld", chunk_end,
                    static_cast<long long>(static_cast<int64_t>(chunk_end - k_chunk0) * p.chunk),
                    static_cast<long long>(k_tokens));
    *empty = chunk_end == chunk_begin;
    if (*empty) return HGA_OK;
    HGA_TRY(check_tensor(k_rot, "k_rot"));
    HGA_TRY(check_tensor(chunk_sum, "chunk_sum"));
    HGA_TRY(check_tensor(group_sum, "group_sum"));
    return HGA_OK;
}

}  // namespace

hga_status hga_build_summaries(const hga_plan* plan, const void* k_rot, int64_t k_tokens,
                               int32_t k_chunk0, int32_t chunk_begin, int32_t chunk_end,
                               float* chunk_sum, float* group_sum, int32_t table_chunks,
                               void* stream) {
    bool empty = false;
    HGA_TRY(check_summaries(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end, chunk_sum,
                            group_sum, table_chunks, &empty));
    if (empty) return HGA_OK;
    clear_stale_error();
    return launched(hga::launch_build_summaries(*plan, k_rot, k_tokens, k_chunk0, chunk_begin,
                                                chunk_end, chunk_sum, group_sum, table_chunks,
                                                static_cast<hipStream_t>(stream)),
                    "hga_build_summaries launch");
}

hga_status hga_build_summaries_qbar(const hga_plan* plan, const void* k_rot, int64_t k_tokens,
                                    int32_t k_chunk0, int32_t chunk_begin, int32_t chunk_end,
                                    float* chunk_sum, float* group_sum, int32_t table_chunks,
                                    const void* q_rot, int32_t q_chunk0, int32_t n_q_chunks,
                                    float* qbar, void* stream) {
    bool empty = false;
    HGA_TRY(check_summaries(plan, k_rot, k_tokens, k_chunk0, chunk_begin, chunk_end, chunk_sum,
                            group_sum, table_chunks, &empty));
    if (q_chunk0 < 0 || n_q_chunks < 0)
        return fail(HGA_EINVAL, "q_chunk0 and n_q_chunks must be >= 0");
    if (n_q_chunks > 0) {
        HGA_TRY(check_tensor(q_rot, "q_rot"));
        HGA_TRY(check_tensor(qbar, "qbar"));
    }
    if (empty && n_q_chunks == 0) return HGA_OK;
    clear_stale_error();
    return launched(hga::launch_summaries_qbar(*plan, k_rot, k_tokens, k_chunk0, chunk_begin,
                                               chunk_end, chunk_sum, group_sum, table_chunks,
                                               q_rot, q_chunk0, n_q_chunks, qbar,
                                               static_cast<hipStream_t>(stream)),
                    "hga_build_summaries_qbar launch");
}

namespace {

// Checks shared by the chunk-routing calls; *n_max gets the largest number of
// middle chunks of a query chunk.
hga_status check_route_chunks(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                              int32_t n_q_chunks, const float* chunk_sum, int32_t table_chunks,
                              float* qbar, int32_t* chunk_idx, bool groups, int* n_max,
                              const char* q_name = "q_rot") {
    HGA_TRY(check_plan(plan));
    const hga_params& p = plan->p;
    if (q_chunk0 < 0 || n_q_chunks < 0 || table_chunks < 0)
        return fail(HGA_EINVAL, "q_chunk0, n_q_chunks and table_chunks must be >= 0");
    if (n_q_chunks == 0) return HGA_OK;
    if (static_cast<int64_t>(q_chunk0) + n_q_chunks - 1 > table_chunks)
        return fail(HGA_EINVAL, "query chunk %d needs summaries of earlier chunks but "
                    "table_chunks is %d", q_chunk0 + n_q_chunks - 1, table_chunks);
    *n_max = hga::middle_count(p, q_chunk0 + n_q_chunks - 1);
    if (*n_max > hga::kMaxChunkCandidates)
        return fail(HGA_EUNSUPPORTED, "%d middle chunks exceed the %d-candidate limit", *n_max,
                    hga::kMaxChunkCandidates);
    if (hga::route_lds_bytes(*plan, *n_max, groups) > static_cast<size_t>(plan->max_lds))
        return fail(HGA_EUNSUPPORTED, "%d middle chunks do not fit the device's %d-byte LDS",
                    *n_max, plan->max_lds);
    HGA_TRY(check_tensor(q_rot, "q_rot"));
    HGA_TRY(check_tensor(qbar, "qbar"));
    HGA_TRY(check_index(chunk_idx, "chunk_idx"));
    if (*n_max > 0) HGA_TRY(check_tensor(chunk_sum, "chunk_sum"));
    return HGA_OK;
}

}  // namespace

hga_status hga_route_chunks(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                            int32_t n_q_chunks, const float* chunk_sum, int32_t table_chunks,
                            float* qbar, int32_t* chunk_idx, void* stream) {
    int n_max = 0;
    HGA_TRY(check_route_chunks(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum, table_chunks, qbar,
                               chunk_idx, false, &n_max));
    if (n_q_chunks == 0) return HGA_OK;
    clear_stale_error();
    return launched(hga::launch_route_chunks(*plan, q_rot, q_chunk0, n_q_chunks, chunk_sum,
                                             table_chunks, qbar, chunk_idx,
                                             static_cast<hipStream_t>(stream)),
                    "hga_route_chunks launch");
}

hga_status hga_route(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                     int32_t n_q_chunks, const float* chunk_sum, const float* group_sum,
                     int32_t table_chunks, float* qbar, int32_t* chunk_idx, int32_t* group_idx,
                     void* stream) {
    int n_max = 0;
    HGA_TRY(check_route_chunks(plan, q_rot, q_chunk0, n_q_chunks, chunk_sum, table_chunks, qbar,
                               chunk_idx, true, &n_max));
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_tensor(group_sum, "group_sum"));
    HGA_TRY(check_index(group_idx, "group_idx"));
    clear_stale_error();
    return launched(hga::launch_route(*plan, q_rot, q_chunk0, n_q_chunks, chunk_sum, group_sum,
                                      table_chunks, qbar, chunk_idx, group_idx,
                                      static_cast<hipStream_t>(stream)),
                    "hga_route launch");
}

hga_status hga_route_qbar(const hga_plan* plan, const float* qbar, int32_t q_chunk0,
                          int32_t n_q_chunks, const float* chunk_sum, const float* group_sum,
                          int32_t table_chunks, int32_t* chunk_idx, int32_t* group_idx,
                          void* stream) {
    int n_max = 0;
    // the checks of hga_route, with qbar in the place of the query rows
    HGA_TRY(check_route_chunks(plan, qbar, q_chunk0, n_q_chunks, chunk_sum, table_chunks,
                               const_cast<float*>(qbar), chunk_idx, true, &n_max, "qbar"));
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_tensor(group_sum, "group_sum"));
    HGA_TRY(check_index(group_idx, "group_idx"));
    clear_stale_error();
    return launched(hga::launch_route_from_qbar(*plan, qbar, q_chunk0, n_q_chunks, chunk_sum,
                                                group_sum, table_chunks, chunk_idx, group_idx,
                                                static_cast<hipStream_t>(stream)),
                    "hga_route_qbar launch");
}

hga_status hga_route_groups(const hga_plan* plan, const float* qbar, const int32_t* chunk_idx,
                            int32_t q_chunk0, int32_t n_q_chunks, const float* group_sum,
                            int32_t table_chunks, int32_t* group_idx, void* stream) {
    HGA_TRY(check_plan(plan));
    if (q_chunk0 < 0 || n_q_chunks < 0 || table_chunks < 0)
        return fail(HGA_EINVAL, "q_chunk0, n_q_chunks and table_chunks must be >= 0");
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_tensor(qbar, "qbar"));
    HGA_TRY(check_index(chunk_idx, "chunk_idx"));
    HGA_TRY(check_tensor(group_sum, "group_sum"));
    HGA_TRY(check_index(group_idx, "group_idx"));
    clear_stale_error();
    return launched(hga::launch_route_groups(*plan, qbar, chunk_idx, q_chunk0, n_q_chunks,
                                             group_sum, table_chunks, group_idx,
                                             static_cast<hipStream_t>(stream)),
                    "hga_route_groups launch");
}

// Device addresses of two pinned host allocations (their device mappings).
static hga_status map_host_sources(const void* k_src, const void* v_src, const void** ks,
                                   const void** vs) {
    void* dk = nullptr;
    void* dv = nullptr;
    hipError_t e = hipHostGetDevicePointer(&dk, const_cast<void*>(k_src), 0);
    if (e != hipSuccess) {
        (void)hipGetLastError();  // the failed lookup must not surface at a later launch
        return fail(HGA_EINVAL, "k_src is not a mapped pinned host allocation (%s)",
                    hipGetErrorString(e));
    }
    e = hipHostGetDevicePointer(&dv, const_cast<void*>(v_src), 0);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(HGA_EINVAL, "v_src is not a mapped pinned host allocation (%s)",
                    hipGetErrorString(e));
    }
    if (!aligned(dk, 16) || !aligned(dv, 16))
        return fail(HGA_EALIGN, "mapped host sources are not 16-byte aligned");
    *ks = dk;
    *vs = dv;
    return HGA_OK;
}

hga_status hga_gather_kv(const hga_plan* plan, const int32_t* group_idx, int32_t q_chunk0,
                         int32_t n_q_chunks, const void* k_src, const void* v_src,
                         int64_t src_tokens, int32_t src_on_host, void* k_routed,
                         void* v_routed, void* stream) {
    HGA_TRY(check_plan(plan));
    if (q_chunk0 < 0 || n_q_chunks < 0 || src_tokens < 0)
        return fail(HGA_EINVAL, "q_chunk0, n_q_chunks and src_tokens must be >= 0");
    if (src_on_host != 0 && src_on_host != 1) return fail(HGA_EINVAL, "src_on_host must be 0 or 1");
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_index(group_idx, "group_idx"));
    HGA_TRY(check_tensor(k_src, "k_src"));
    HGA_TRY(check_tensor(v_src, "v_src"));
    HGA_TRY(check_tensor(k_routed, "k_routed"));
    HGA_TRY(check_tensor(v_routed, "v_routed"));
    const void* ks = k_src;
    const void* vs = v_src;
    if (src_on_host) HGA_TRY(map_host_sources(k_src, v_src, &ks, &vs));
    clear_stale_error();
    return launched(hga::launch_gather_kv(*plan, group_idx, q_chunk0, n_q_chunks, ks, vs,
                                          src_tokens, k_routed, v_routed,
                                          static_cast<hipStream_t>(stream)),
                    "hga_gather_kv launch");
}

hga_status hga_gather_kv_cached(const hga_plan* plan, const int32_t* group_idx, int32_t c,
                                const void* k_src, const void* v_src, int64_t src_tokens,
                                int32_t src_on_host, void* cache_k, void* cache_v,
                                int32_t n_slots, int32_t* slot_group, int32_t* slot_used,
                                int32_t* group_slot, int64_t map_groups, int32_t* entry_slot,
                                int32_t tick, void* k_routed, void* v_routed, int32_t* n_fetched,
                                void* stream) {
    HGA_TRY(check_plan(plan));
    const hga_params& p = plan->p;
    if (c < 0 || src_tokens < 0 || tick < 0)
        return fail(HGA_EINVAL, "c, src_tokens and tick must be >= 0");
    if (src_on_host != 0 && src_on_host != 1) return fail(HGA_EINVAL, "src_on_host must be 0 or 1");
    if (n_slots < p.topk_groups || n_slots > kMaxCacheSlots)
        return fail(HGA_EINVAL, "n_slots must be in [topk_groups = %d, %d], got %d",
                    p.topk_groups, kMaxCacheSlots, n_slots);
    const int64_t need = static_cast<int64_t>(c) * p.chunk;
    if (src_tokens < need)
        return fail(HGA_EINVAL, "k_src/v_src hold %lld tokens per head; the causal past of query "
                    "chunk %d needs %lld", static_cast<long long>(src_tokens), c,
                    static_cast<long long>(need));
    if (map_groups < src_tokens / p.group)
        return fail(HGA_EINVAL, "group_slot holds %lld groups per head; a %lld-token source has "
                    "%lld", static_cast<long long>(map_groups), static_cast<long long>(src_tokens),
                    static_cast<long long>(src_tokens / p.group));
    if (hga::gather_cached_lds_bytes(*plan, n_slots) > static_cast<size_t>(plan->max_lds))
        return fail(HGA_EUNSUPPORTED, "cache bookkeeping for %d slots exceeds the LDS limit",
                    n_slots);
    HGA_TRY(check_index(group_idx, "group_idx"));
    HGA_TRY(check_tensor(k_src, "k_src"));
    HGA_TRY(check_tensor(v_src, "v_src"));
    HGA_TRY(check_tensor(cache_k, "cache_k"));
    HGA_TRY(check_tensor(cache_v, "cache_v"));
    HGA_TRY(check_index(slot_group, "slot_group"));
    HGA_TRY(check_index(slot_used, "slot_used"));
    HGA_TRY(check_index(group_slot, "group_slot"));
    HGA_TRY(check_index(entry_slot, "entry_slot"));
    HGA_TRY(check_tensor(k_routed, "k_routed"));
    HGA_TRY(check_tensor(v_routed, "v_routed"));
    if (n_fetched && !aligned(n_fetched, 4)) return fail(HGA_EALIGN, "n_fetched is not 4-byte aligned");
    const void* ks = k_src;
    const void* vs = v_src;
    if (src_on_host) HGA_TRY(map_host_sources(k_src, v_src, &ks, &vs));
    clear_stale_error();
    return launched(hga::launch_gather_kv_cached(*plan, group_idx, c, ks, vs, src_tokens, cache_k,
                                                 cache_v, n_slots, slot_group, slot_used,
                                                 group_slot, map_groups, tick,
                                                 entry_slot, k_routed, v_routed, n_fetched,
                                                 static_cast<hipStream_t>(stream)),
                    "hga_gather_kv_cached launch");
}

namespace {

// Checks shared by the attention calls (the plan is already checked and
// n_q_chunks > 0).
hga_status check_attend(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                        int32_t n_q_chunks, const void* k_res, const void* v_res,
                        int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                        const void* v_routed, const int32_t* group_idx, const void* out,
                        const float* lse, bool routed_optional = false) {
    const hga_params& p = plan->p;
    if (!res_slot && (static_cast<int64_t>(q_chunk0) + n_q_chunks) * p.chunk > res_tokens)
        return fail(HGA_EINVAL, "without res_slot the resident K/V must cover chunks up to %d "
                    "(%lld tokens), have %lld", q_chunk0 + n_q_chunks - 1,
                    static_cast<long long>((static_cast<int64_t>(q_chunk0) + n_q_chunks) * p.chunk),
                    static_cast<long long>(res_tokens));
    if (res_slot && res_tokens < p.chunk)
        return fail(HGA_EINVAL, "resident buffer holds no full chunk");
    {
        // the kernels address one head's slab with 32-bit offsets
        const int64_t row_bytes = static_cast<int64_t>(p.head_dim) * (p.dtype == HGA_BF16 ? 2 : 4);
        const int64_t r = p.n_q_heads / p.n_kv_heads;
        const int64_t q_slab = r * (static_cast<int64_t>(n_q_chunks) * p.chunk) * row_bytes;
        if (res_tokens * row_bytes >= kMaxSlabBytes || q_slab >= kMaxSlabBytes)
            return fail(HGA_EUNSUPPORTED, "one head's K/V (%lld bytes) or the query rows of one "
                        "KV head (%lld bytes) exceed the %lld-byte addressing limit",
                        static_cast<long long>(res_tokens * row_bytes),
                        static_cast<long long>(q_slab), static_cast<long long>(kMaxSlabBytes));
    }
    if (res_slot) HGA_TRY(check_index(res_slot, "res_slot"));
    HGA_TRY(check_tensor(q_rot, "q_rot"));
    HGA_TRY(check_tensor(k_res, "k_res"));
    HGA_TRY(check_tensor(v_res, "v_res"));
    if (routed_optional && !k_routed && !v_routed) {
        // the gather forms without routed buffers: the rows stay on chip
    } else {
        if (routed_optional && (!k_routed || !v_routed))
            return fail(HGA_EINVAL, "k_routed and v_routed must both be given or both be NULL");
        HGA_TRY(check_tensor(k_routed, "k_routed"));
        HGA_TRY(check_tensor(v_routed, "v_routed"));
    }
    HGA_TRY(check_index(group_idx, "group_idx"));
    HGA_TRY(check_tensor(out, "out"));
    if (lse && !aligned(lse, 4)) return fail(HGA_EALIGN, "lse is not 4-byte aligned");
    return HGA_OK;
}

}  // namespace

hga_status hga_attend_timed(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                            int32_t n_q_chunks, const void* k_res, const void* v_res,
                            int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                            const void* v_routed, const int32_t* group_idx, void* out, float* lse,
                            void* start_event, void* stop_event, void* stream) {
    HGA_TRY(check_plan(plan));
    if (q_chunk0 < 0 || n_q_chunks < 0 || res_tokens < 0)
        return fail(HGA_EINVAL, "q_chunk0, n_q_chunks and res_tokens must be >= 0");
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_attend(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens, res_slot,
                         k_routed, v_routed, group_idx, out, lse));
    clear_stale_error();
    return launched(hga::launch_attend(*plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res,
                                       res_tokens, res_slot, k_routed, v_routed, group_idx, out,
                                       lse, static_cast<hipEvent_t>(start_event),
                                       static_cast<hipEvent_t>(stop_event),
                                       static_cast<hipStream_t>(stream)),
                    "hga_attend launch");
}

int64_t hga_attend_split_workspace(const hga_plan* plan, int32_t n_q_chunks) {
    if (check_plan(plan) != HGA_OK || n_q_chunks < 0) return -1;
    return hga::kMaxSplit * hga::attend_split_bytes_per_split(*plan, n_q_chunks);
}

hga_status hga_attend_split(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                            int32_t n_q_chunks, const void* k_res, const void* v_res,
                            int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                            const void* v_routed, const int32_t* group_idx, void* out, float* lse,
                            void* workspace, int64_t workspace_bytes, void* stream) {
    HGA_TRY(check_plan(plan));
    if (q_chunk0 < 0 || n_q_chunks < 0 || res_tokens < 0 || workspace_bytes < 0)
        return fail(HGA_EINVAL,
                    "q_chunk0, n_q_chunks, res_tokens and workspace_bytes must be >= 0");
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_attend(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens, res_slot,
                         k_routed, v_routed, group_idx, out, lse));
    HGA_TRY(check_workspace(workspace, workspace_bytes));
    clear_stale_error();
    return launched(hga::launch_attend_split(*plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res,
                                             res_tokens, res_slot, k_routed, v_routed, group_idx,
                                             out, lse, workspace, workspace ? workspace_bytes : 0,
                                             static_cast<hipStream_t>(stream)),
                    "hga_attend_split launch");
}

hga_status hga_attend_split_static(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                                   int32_t n_q_chunks, const void* k_res, const void* v_res,
                                   int64_t res_tokens, const int32_t* res_slot,
                                   const void* k_routed, const void* v_routed,
                                   const int32_t* group_idx, void* out, float* lse, void* stream) {
    HGA_TRY(check_plan(plan));
    if (q_chunk0 < 0 || n_q_chunks < 0 || res_tokens < 0)
        return fail(HGA_EINVAL, "q_chunk0, n_q_chunks and res_tokens must be >= 0");
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_attend(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens, res_slot,
                         k_routed, v_routed, group_idx, out, lse));
    void* scratch = hga::static_scratch(plan->device);
    if (!scratch) return fail(HGA_EHIP, "no static scratch address for device %d", plan->device);
    if (hga::attend_split_applies(*plan)) {
        const int64_t per = hga::attend_split_bytes_per_split(*plan, n_q_chunks);
        if (2 * per > hga::kStaticScratchBytes)
            return fail(HGA_EUNSUPPORTED, "two splits of %d query chunks need %lld bytes of "
                        "scratch, above the static %lld bytes; use hga_attend_split with a "
                        "workspace", n_q_chunks, static_cast<long long>(2 * per),
                        static_cast<long long>(hga::kStaticScratchBytes));
    }
    clear_stale_error();
    return launched(hga::launch_attend_split(*plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res,
                                             res_tokens, res_slot, k_routed, v_routed, group_idx,
                                             out, lse, scratch, hga::kStaticScratchBytes,
                                             static_cast<hipStream_t>(stream)),
                    "hga_attend_split_static launch");
}

int64_t hga_static_scratch_bytes(void) { return hga::kStaticScratchBytes; }

hga_status hga_gather_attend_split(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                                   int32_t n_q_chunks, const void* k_res, const void* v_res,
                                   int64_t res_tokens, const int32_t* res_slot,
                                   const void* k_src, const void* v_src, int64_t src_tokens,
                                   int32_t src_on_host, const int32_t* group_idx, void* k_routed,
                                   void* v_routed, void* out, float* lse, void* workspace,
                                   int64_t workspace_bytes, void* stream) {
    HGA_TRY(check_plan(plan));
    if (q_chunk0 < 0 || n_q_chunks < 0 || res_tokens < 0 || src_tokens < 0 ||
        workspace_bytes < 0)
        return fail(HGA_EINVAL, "q_chunk0, n_q_chunks, res_tokens, src_tokens and "
                    "workspace_bytes must be >= 0");
    if (src_on_host != 0 && src_on_host != 1) return fail(HGA_EINVAL, "src_on_host must be 0 or 1");
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_attend(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens, res_slot,
                         k_routed, v_routed, group_idx, out, lse, true));
    const hga_params& p = plan->p;
    const int64_t need = static_cast<int64_t>(q_chunk0 + n_q_chunks - 1) * p.chunk;
    if (src_tokens < need)
        return fail(HGA_EINVAL, "k_src/v_src hold %lld tokens per head; the causal past of query "
                    "chunk %d needs %lld", static_cast<long long>(src_tokens),
                    q_chunk0 + n_q_chunks - 1, static_cast<long long>(need));
    const int64_t row_bytes = static_cast<int64_t>(p.head_dim) * (p.dtype == HGA_BF16 ? 2 : 4);
    if (src_tokens * row_bytes >= kMaxSlabBytes)
        return fail(HGA_EUNSUPPORTED, "one head's routed-row source (%lld bytes) exceeds the "
                    "%lld-byte addressing limit", static_cast<long long>(src_tokens * row_bytes),
                    static_cast<long long>(kMaxSlabBytes));
    HGA_TRY(check_tensor(k_src, "k_src"));
    HGA_TRY(check_tensor(v_src, "v_src"));
    HGA_TRY(check_workspace(workspace, workspace_bytes));
    const void* ks = k_src;
    const void* vs = v_src;
    if (src_on_host) HGA_TRY(map_host_sources(k_src, v_src, &ks, &vs));
    clear_stale_error();
    return launched(hga::launch_gather_attend_split(
                        *plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens, res_slot,
                        ks, vs, src_tokens, group_idx, k_routed, v_routed, out, lse, workspace,
                        workspace ? workspace_bytes : 0, static_cast<hipStream_t>(stream)),
                    "hga_gather_attend_split launch");
}

hga_status hga_attend_backward(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                               int32_t n_q_chunks, const void* k_res, const void* v_res,
                               int64_t res_tokens, const int32_t* group_idx, const void* out,
                               const float* lse, const void* dout, float* dq, float* dk,
                               float* dv, void* stream) {
    HGA_TRY(check_plan(plan));
    if (q_chunk0 < 0 || n_q_chunks < 0 || res_tokens < 0)
        return fail(HGA_EINVAL, "q_chunk0, n_q_chunks and res_tokens must be >= 0");
    if (plan->p.dtype != HGA_BF16)
        return fail(HGA_EUNSUPPORTED, "the attention backward is built for bf16 plans");
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_attend(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens, nullptr,
                         k_res, v_res, group_idx, out, lse));
    if (!lse) return fail(HGA_EINVAL, "lse (the forward's log-sum-exp) is required");
    HGA_TRY(check_tensor(dout, "dout"));
    HGA_TRY(check_tensor(dq, "dq"));
    HGA_TRY(check_tensor(dk, "dk"));
    HGA_TRY(check_tensor(dv, "dv"));
    if (hga::attend_backward_lds_bytes(*plan) > static_cast<size_t>(plan->max_lds))
        return fail(HGA_EUNSUPPORTED, "the backward's LDS tiles exceed the device limit");
    clear_stale_error();
    return launched(hga::launch_attend_backward(*plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res,
                                                res_tokens, group_idx, out, lse, dout, dq, dk, dv,
                                                static_cast<hipStream_t>(stream)),
                    "hga_attend_backward launch");
}

hga_status hga_gather_attend(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                             int32_t n_q_chunks, const void* k_res, const void* v_res,
                             int64_t res_tokens, const int32_t* group_idx, void* k_routed,
                             void* v_routed, void* out, float* lse, void* start_event,
                             void* stop_event, void* stream) {
    HGA_TRY(check_plan(plan));
    if (q_chunk0 < 0 || n_q_chunks < 0 || res_tokens < 0)
        return fail(HGA_EINVAL, "q_chunk0, n_q_chunks and res_tokens must be >= 0");
    if (n_q_chunks == 0) return HGA_OK;
    HGA_TRY(check_attend(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens, nullptr,
                         k_routed, v_routed, group_idx, out, lse, true));
    clear_stale_error();
    return launched(hga::launch_gather_attend(*plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res,
                                              res_tokens, group_idx, k_routed, v_routed, out, lse,
                                              static_cast<hipEvent_t>(start_event),
                                              static_cast<hipEvent_t>(stop_event),
                                              static_cast<hipStream_t>(stream)),
                    "hga_gather_attend launch");
}

namespace {

// Checks of one block step on chunk c (nothing launched).
hga_status check_block_step(const hga_plan* plan, const void* q_block, int32_t c,
                            const void* k_res, const void* v_res, int64_t res_tokens,
                            float* chunk_sum, float* group_sum, int32_t table_chunks, float* qbar,
                            int32_t* chunk_idx, int32_t* group_idx, void* k_routed,
                            void* v_routed, void* out, float* lse) {
    HGA_TRY(check_plan(plan));
    const hga_params& p = plan->p;
    if (c < 0 || res_tokens < 0 || table_chunks < 0)
        return fail(HGA_EINVAL, "c, res_tokens and table_chunks must be >= 0");
    if (table_chunks < c + 1)
        return fail(HGA_EINVAL, "the block's chunk %d needs table_chunks > %d (got %d)", c, c,
                    table_chunks);
    int n_max = 0;
    HGA_TRY(check_route_chunks(plan, q_block, c, 1, chunk_sum, table_chunks, qbar, chunk_idx,
                               true, &n_max, "q_block"));
    HGA_TRY(check_tensor(group_sum, "group_sum"));
    HGA_TRY(check_index(group_idx, "group_idx"));
    HGA_TRY(check_attend(plan, q_block, c, 1, k_res, v_res, res_tokens, nullptr, k_routed,
                         v_routed, group_idx, out, lse));
    bool empty = false;
    HGA_TRY(check_summaries(plan, k_res, res_tokens, 0, c, c + 1, chunk_sum, group_sum,
                            table_chunks, &empty));
    (void)p;
    return HGA_OK;
}

// The three launches of one block step (checks done).
hipError_t launch_block_step(const hga_plan& plan, const void* q_block, int32_t c,
                             const void* k_res, const void* v_res, int64_t res_tokens,
                             float* chunk_sum, float* group_sum, int32_t table_chunks,
                             float* qbar, int32_t* chunk_idx, int32_t* group_idx, void* k_routed,
                             void* v_routed, void* out, float* lse, void* workspace,
                             int64_t workspace_bytes, hipStream_t stream) {
    hipError_t e = hga::launch_route(plan, q_block, c, 1, chunk_sum, group_sum, table_chunks,
                                     qbar, chunk_idx, group_idx, stream);
    if (e != hipSuccess) return e;
    if (workspace)
        e = hga::launch_gather_attend_split(plan, q_block, c, 1, k_res, v_res, res_tokens, nullptr,
                                            k_res, v_res, res_tokens, group_idx, k_routed,
                                            v_routed, out, lse, workspace, workspace_bytes,
                                            stream);
    else
        e = hga::launch_gather_attend(plan, q_block, c, 1, k_res, v_res, res_tokens, group_idx,
                                      k_routed, v_routed, out, lse, nullptr, nullptr, stream);
    if (e != hipSuccess) return e;
    return hga::launch_build_summaries(plan, k_res, res_tokens, 0, c, c + 1, chunk_sum,
                                       group_sum, table_chunks, stream);
}

}  // namespace

hga_status hga_block_step(const hga_plan* plan, const void* q_block, int32_t c,
                          const void* k_res, const void* v_res, int64_t res_tokens,
                          float* chunk_sum, float* group_sum, int32_t table_chunks, float* qbar,
                          int32_t* chunk_idx, int32_t* group_idx, void* k_routed, void* v_routed,
                          void* out, float* lse, void* workspace, int64_t workspace_bytes,
                          void* stream) {
    HGA_TRY(check_block_step(plan, q_block, c, k_res, v_res, res_tokens, chunk_sum, group_sum,
                             table_chunks, qbar, chunk_idx, group_idx, k_routed, v_routed, out,
                             lse));
    HGA_TRY(check_workspace(workspace, workspace_bytes));
    clear_stale_error();
    return launched(launch_block_step(*plan, q_block, c, k_res, v_res, res_tokens, chunk_sum,
                                      group_sum, table_chunks, qbar, chunk_idx, group_idx,
                                      k_routed, v_routed, out, lse,
                                      workspace_bytes > 0 ? workspace : nullptr, workspace_bytes,
                                      static_cast<hipStream_t>(stream)),
                    "hga_block_step launch");
}

hga_status hga_prefill_blocks(const hga_plan* plan, const void* q_blocks, int32_t n_blocks,
                              const void* k_res, const void* v_res, int64_t res_tokens,
                              float* chunk_sum, float* group_sum, int32_t table_chunks,
                              float* qbar, int32_t* chunk_idx, int32_t* group_idx,
                              void* k_routed, void* v_routed, void* out, float* lse,
                              void* workspace, int64_t workspace_bytes, void* stream) {
    HGA_TRY(check_plan(plan));
    if (n_blocks < 0) return fail(HGA_EINVAL, "n_blocks must be >= 0");
    HGA_TRY(check_workspace(workspace, workspace_bytes));
    if (n_blocks == 0) return HGA_OK;
    const hga_params& p = plan->p;
    const int64_t eb = p.dtype == HGA_BF16 ? 2 : 4;
    const int64_t bq = static_cast<int64_t>(p.batch) * p.n_q_heads * p.chunk;  // rows per block
    const int64_t bkv = static_cast<int64_t>(p.batch) * p.n_kv_heads;
    const int64_t q_bytes = bq * p.head_dim * eb;
    const int64_t qbar_elems = bkv * p.head_dim;
    const int64_t ci_elems = bkv * p.topk_chunks;
    const int64_t gi_elems = bkv * p.topk_groups;
    const int64_t rt_bytes = bkv * p.topk_groups * p.group * p.head_dim * eb;
    auto at = [](const void* base, int64_t bytes) {
        return static_cast<const void*>(static_cast<const unsigned char*>(base) + bytes);
    };
    auto atw = [](void* base, int64_t bytes) {
        return static_cast<void*>(static_cast<unsigned char*>(base) + bytes);
    };
    // every block is checked before the first launch (the last block is the
    // most demanding, block 0 the one with no candidates)
    for (int32_t c : {0, n_blocks - 1}) {
        HGA_TRY(check_block_step(
            plan, at(q_blocks, c * q_bytes), c, k_res, v_res, res_tokens, chunk_sum, group_sum,
            table_chunks, qbar + c * qbar_elems, chunk_idx + c * ci_elems,
            group_idx + c * gi_elems, atw(k_routed, c * rt_bytes), atw(v_routed, c * rt_bytes),
            atw(out, c * q_bytes), lse ? lse + c * bq : nullptr));
    }
    clear_stale_error();
    for (int32_t c = 0; c < n_blocks; ++c) {
        const hipError_t e = launch_block_step(
            *plan, at(q_blocks, c * q_bytes), c, k_res, v_res, res_tokens, chunk_sum, group_sum,
            table_chunks, qbar + c * qbar_elems, chunk_idx + c * ci_elems,
            group_idx + c * gi_elems, atw(k_routed, c * rt_bytes), atw(v_routed, c * rt_bytes),
            atw(out, c * q_bytes), lse ? lse + c * bq : nullptr,
            workspace_bytes > 0 ? workspace : nullptr, workspace_bytes,
            static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return launched(e, "hga_prefill_blocks launch");
    }
    return HGA_OK;
}

hga_status hga_attend(const hga_plan* plan, const void* q_rot, int32_t q_chunk0,
                      int32_t n_q_chunks, const void* k_res, const void* v_res,
                      int64_t res_tokens, const int32_t* res_slot, const void* k_routed,
                      const void* v_routed, const int32_t* group_idx, void* out, float* lse,
                      void* stream) {
    return hga_attend_timed(plan, q_rot, q_chunk0, n_q_chunks, k_res, v_res, res_tokens, res_slot,
                            k_routed, v_routed, group_idx, out, lse, nullptr, nullptr, stream);
}

}  // extern "C"
