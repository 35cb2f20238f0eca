// Library-owned split-partial storage for mla_lowbit_decode_attn_noalloc, the
// decode entry point for callers that cannot allocate device memory.
//
// `scratch` is one file-scope device array: every GPU the library runs on
// holds its own copy from module load until the process ends.  Host code
// never passes the array's name to a kernel (on the host it only stands in
// for the symbol): the first call on a device, with that device current,
// resolves the device address once with hipGetSymbolAddress and keeps it per
// device; kernels receive that address as their partial buffers.  Every call
// on one GPU shares that GPU's array, so calls that overlap on one GPU race.
#include <hip/hip_runtime.h>

#include <mutex>

#include "internal.h"

namespace mla {
namespace {

constexpr int kMaxDevices = 64;
constexpr size_t kScratchBytes = static_cast<size_t>(kNoallocSplitRows) * kNoallocRowBytes;

// Layout: part_o [rows][512] fp16, then part_m [rows] fp32, part_s [rows] fp32.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};

}  // namespace

hipError_t noalloc_partials(float** part_m, float** part_s, uint16_t** part_o) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    void* base = nullptr;
    {
        std::lock_guard<std::mutex> lock(g_mu);
        if (g_scratch[dev] == nullptr) {
            void* p = nullptr;
            e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess) return e;
            if (p == nullptr) return hipErrorInvalidSymbol;
            g_scratch[dev] = p;
        }
        base = g_scratch[dev];
    }
    uint8_t* b = static_cast<uint8_t*>(base);
    *part_o = reinterpret_cast<uint16_t*>(b);
    *part_m = reinterpret_cast<float*>(b + static_cast<size_t>(kNoallocSplitRows) * 1024);
    *part_s = reinterpret_cast<float*>(b + static_cast<size_t>(kNoallocSplitRows) * 1028);
    return hipSuccess;
}

}  // namespace mla
