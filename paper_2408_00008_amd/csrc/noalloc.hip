// moe_forward_noalloc: the whole layer for callers that cannot allocate device
// memory (code under graph capture, tight serving loops, harnesses that
// forbid allocation).  Its scratch -- routing arrays, the SwiGLU
// intermediate h, the gate-weighted slot outputs y and their reduction-part
// slices -- lives in one file-scope device array of fixed size, so the call
// allocates nothing.  Each GPU the library runs on holds its own copy of the
// array (loaded with the code object, kept until the process ends).
//
// The array's name is a host-side stand-in in host code; its device address
// is looked up once per device with hipGetSymbolAddress (with that device
// current) and only that address is handed to the kernels.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <mutex>

#include "launch.hpp"
#include "moe.h"

namespace moe {
moe_status_t set_last_error(moe_status_t s, const char* fmt, ...);
moe_status_t forward_fixed_scratch(const moe_bf16_t* x, const moe_bf16_t* router_w,
                                   const float* router_bias, const moe_bf16_t* w1,
                                   const moe_bf16_t* w3, const moe_bf16_t* w2, int64_t T,
                                   int32_t d, int32_t ffn, int32_t E, int32_t k,
                                   const float* residual, moe_bf16_t* out, float* out_f32,
                                   hipStream_t stream, ScratchFn scratch_fn);
}  // namespace moe

namespace {
// 64 MiB: the 256-token skewed Mixtral decode step (h 14.7 MB, y with two
// reduction-part slices 16.8 MB) fits, and so does any Mixtral-shape step of
// up to 256 tokens.
constexpr size_t kScratchBytes = size_t(64) << 20;
}  // namespace

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices];  // device address of `scratch` on each device, once looked up

int fixed_scratch(size_t bytes, void** out)
{
    if (bytes > kScratchBytes)
        return moe::set_last_error(MOE_ERR_NO_MEMORY,
                                   "moe_forward_noalloc: these sizes need %zu bytes of scratch, "
                                   "more than its fixed %zu-byte array; use moe_forward_ex with a "
                                   "caller workspace",
                                   bytes, kScratchBytes);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return moe::set_last_error(MOE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return moe::set_last_error(MOE_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return moe::set_last_error(MOE_ERR_HIP, "hipGetSymbolAddress(scratch): %s",
                                       hipGetErrorString(e));
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return MOE_OK;
}

}  // namespace

extern "C" moe_status_t moe_forward_noalloc(const moe_bf16_t* x, const moe_bf16_t* router_w,
                                            const float* router_bias, const moe_bf16_t* w1,
                                            const moe_bf16_t* w3, const moe_bf16_t* w2, int64_t T,
                                            int32_t d, int32_t ffn, int32_t E, int32_t k,
                                            const float* residual, moe_bf16_t* out,
                                            float* out_f32, hipStream_t stream)
{
    return moe::forward_fixed_scratch(x, router_w, router_bias, w1, w3, w2, T, d, ffn, E, k,
                                      residual, out, out_f32, stream, &fixed_scratch);
}
