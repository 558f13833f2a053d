// Library-held device scratch for the allocation-free split attention
// (hga_attend_split_static): one fixed array per device, alive until the
// process ends, used in place of a caller workspace.
//
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address is taken once per device with hipGetSymbolAddress (with
// that device current, at plan creation) and only that address is handed to
// kernels.  Every call on a device shares the device's array, so calls that
// overlap in time on one device race; the split attention writes every
// partial result before its merge reads it, so nothing needs clearing.
#include <hip/hip_runtime.h>

#include <mutex>

#include "hga_internal.hpp"

static __device__ __align__(256) unsigned char scratch[hga::kStaticScratchBytes];

namespace hga {
namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

hipError_t static_scratch_init(int device) {
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[device]) return hipSuccess;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[device] = p;
    return hipSuccess;
}

void* static_scratch(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
}

}  // namespace hga
