// Static device scratch of rf_keyframe_attention_noalloc, the attention entry
// point for callers that cannot allocate device memory.
//
// The split-key tail of bf16 attention keeps each part's unnormalised output
// and (reference max, row sum) in fp32 until the combine kernel merges them.
// rf_keyframe_attention_ws takes that buffer from the caller; the
// allocation-free entry point takes it from the array below, which every GPU
// the library runs on holds (its own copy, at its own address) until the
// process ends. In host code `scratch` names a host-side stand-in, never the
// device memory: its device address is looked up once per device, with that
// device current, and only that address is passed to kernels.
//
// Every call on one GPU shares that GPU's array. Nothing in it has to start at
// zero (each part writes all of its rows before the combine reads them), but
// two calls that overlap in time on one GPU (different streams, or different
// threads) race on it.
#include <mutex>

#include "rf_internal.h"

static __device__ __align__(256) uint8_t scratch[rf::kAttentionScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
void *g_scratch[kMaxDevices];   // device address of `scratch`, per device (NULL until looked up)

}  // namespace

namespace rf {

hipError_t attention_scratch(void **out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mutex);
    if (!g_scratch[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p || (reinterpret_cast<uintptr_t>(p) & 255u)) return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

}  // namespace rf
