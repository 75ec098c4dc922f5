// mq_qlinear_noalloc: the qlinear with its split-K workspace in a static
// device array instead of memory the caller or the library allocates.
//
// The K split of the prefill kernel keeps per-tile arrival counters and the
// slices' int32 partial sums in a workspace.  Callers that cannot allocate
// device memory (code under HIP graph capture, serving loops that forbid
// hipMalloc) get that workspace from `scratch`, one array of
// MQ_NOALLOC_SCRATCH_BYTES per GPU, resident from the library's load until
// the process ends.
#include <atomic>

#include "mq.h"
#include "mq_internal.h"

namespace {

constexpr int64_t kScratchBytes = MQ_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "whole 256-byte blocks");

// The workspace itself.  In host code this name is a host-side stand-in:
// kernels and copies take the device address from hipGetSymbolAddress.
static __device__ __align__(256) int8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
// device address of `scratch` per device, looked up on the first call there
std::atomic<void*> g_scratch[kMaxDevices];

// Device address of this device's `scratch`, or nullptr on a HIP error.
void* scratch_ptr(int dev)
{
    void* ptr = g_scratch[dev].load(std::memory_order_acquire);
    if (ptr) return ptr;
    // the current device is `dev`: its own copy of the array
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch[dev].store(ptr, std::memory_order_release);
    return ptr;
}

// Zero the arrival counters (a fill kernel, not a memset node, so the call
// can be captured into a HIP graph).
__global__ void zero_counters(int32_t* c, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        c[i] = 0;
}

}  // namespace

extern "C" mq_status mq_qlinear_noalloc(const int8_t* a_q, int64_t M, int64_t K, int64_t N,
                                        const void* w_q, int32_t w_bits, const float* w_scale,
                                        const int32_t* w_colsum, float a_scale, int32_t a_zp,
                                        float out_scale, int32_t out_zp, int32_t out_bits,
                                        const float* bias, void* y_q, void* stream)
{
    mq::QLinearArgs p;
    int32_t path = MQ_PATH_AUTO;
    mq_status st = mq::qlinear_validate(a_q, 8, nullptr, M, K, N, w_q, w_bits, w_scale, nullptr,
                                        w_colsum, a_scale, a_zp, out_scale, out_zp, out_bits,
                                        bias, y_q, nullptr, 0, MQ_PATH_AUTO, &p, &path);
    if (st != MQ_OK || M == 0 || N == 0) return st;
    const int64_t need = mq_qlinear_workspace_bytes(M, K, N, w_bits, out_bits);
    if (need < 0) return MQ_ERR_INVALID_ARG;
    if (need > kScratchBytes) return MQ_ERR_UNSUPPORTED;  // the split would not fit
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (need > 0) {
        int dev = -1;
        if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return MQ_ERR_HIP;
        void* ws = scratch_ptr(dev);
        if (!ws) return MQ_ERR_HIP;
        p.ws = ws;
        p.ws_bytes = kScratchBytes;
        const int64_t words = mq::prefill_counter_bytes(p) / 4;
        if (words > 0) {
            zero_counters<<<(unsigned)((words + 255) / 256), 256, 0, s>>>(
                static_cast<int32_t*>(ws), words);
            if (hipGetLastError() != hipSuccess) return MQ_ERR_HIP;
        }
    }
    return mq::qlinear_dispatch(p, path, s);
}
