// unisvq_gemm without a caller workspace: the workspace of the prefill and
// small-batch product (the fp16 copy of bf16 activations with its per-token
// scales, and the fp32 partial sums of a K split) lives in a fixed device
// array of this library, so a call allocates nothing -- for callers that
// cannot allocate (code under HIP graph capture, tight serving loops).
#include <mutex>

#include "common.hpp"

namespace unisvq {
namespace {

// One copy per device, held until the process ends.  In host code the name
// `scratch` is only a host-side stand-in: kernels get the device address
// looked up per device below.
constexpr size_t kScratchBytes = size_t{32} << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
void* scratch_ptr[kMaxDevices];
bool scratch_ready[kMaxDevices];
std::mutex scratch_mutex;

// Device address of this device's scratch array (looked up on the first call
// on the device, with that device current); UNISVQ_EHIP if the lookup fails.
int scratch_for_current_device(void** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return UNISVQ_EHIP;
    std::lock_guard<std::mutex> lock(scratch_mutex);
    if (!scratch_ready[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return UNISVQ_EHIP;
        scratch_ptr[dev] = p;
        scratch_ready[dev] = true;
    }
    *out = scratch_ptr[dev];
    return UNISVQ_OK;
}

}  // namespace

size_t noalloc_scratch_bytes() { return kScratchBytes; }

int launch_gemm_noalloc(int64_t N, int64_t K, const uint8_t* packed, int64_t M, const void* x, int x_dtype, void* y,
                        int y_dtype, hipStream_t s) {
    if (gemm_workspace_bytes(N, K, M, x_dtype) > kScratchBytes) return UNISVQ_ESCRATCH;
    void* ws = nullptr;
    const int st = scratch_for_current_device(&ws);
    if (st != UNISVQ_OK) return st;
    return launch_gemm(N, K, packed, M, x, x_dtype, y, y_dtype, ws, s);
}

}  // namespace unisvq
