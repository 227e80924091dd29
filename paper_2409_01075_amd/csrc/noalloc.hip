// vx_gemm_batched_noalloc: the batched GEMM for callers that cannot
// allocate (code under HIP graph capture, serving loops that forbid device
// allocation).  Its split-K scratch -- arrival counters, then fp32 partials --
// is one array in static device storage, so no call allocates anything; each
// GPU holds its own copy of the array until the process ends.
#include <mutex>

#include <hip/hip_runtime.h>

#include "vx_internal.h"

namespace {

constexpr size_t kScratchTickets = 64 * 1024;               // 16384 arrival counters
constexpr size_t kScratchPartials = 16ull * 1024 * 1024;    // fp32 partial tiles
constexpr size_t kScratchBytes = kScratchTickets + kScratchPartials;
constexpr int kMaxDevices = 64;

// The array's name is a host-side stand-in in host code: kernels get the
// device address found by hipGetSymbolAddress below, never the name.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Zeroes the arrival counters (a kernel rather than a memset, so that a
// caller may capture it in a graph).
__global__ void vx_scratch_clear(unsigned* tickets, int n)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        tickets[i] = 0u;
}

std::mutex g_mu;
void* g_ptr[kMaxDevices];       // scratch address per device
bool g_clear[kMaxDevices];      // its counters are known to be zero

// Set-up, once per device, with that device current: the array's address,
// and its counters cleared on `stream` ahead of the call's own kernel.  A
// clear captured into a graph is not counted as done: the next call outside
// capture clears again (the counters reset themselves after every use, so
// later calls need no clear).
vx_status scratch_for(int dev, hipStream_t stream, void** out)
{
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return VX_ERR_HIP;
        }
        g_ptr[dev] = p;
    }
    if (!g_clear[dev]) {
        const int n = (int)(kScratchTickets / sizeof(unsigned));
        hipLaunchKernelGGL(vx_scratch_clear, dim3((n + 255) / 256), dim3(256), 0, stream, (unsigned*)g_ptr[dev], n);
        if (hipGetLastError() != hipSuccess)
            return VX_ERR_HIP;
        hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
            (void)hipGetLastError();
            cs = hipStreamCaptureStatusActive;
        }
        g_clear[dev] = cs == hipStreamCaptureStatusNone;
    }
    *out = g_ptr[dev];
    return VX_OK;
}

}  // namespace

extern "C" vx_status vx_gemm_batched_noalloc(int64_t batch, int64_t M, int64_t N, int64_t K, vx_dtype dtype,
                                             const void* A, int64_t strideA, const void* B, int64_t strideB,
                                             void* C, int64_t strideC, void* stream)
{
    bool noop = false;
    vx_status st = vxi_gemm_check(batch, M, N, K, dtype, A, strideA, B, strideB, C, strideC, &noop);
    if (st != VX_OK || noop)
        return st;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return VX_ERR_HIP;
    void* p = nullptr;
    st = scratch_for(dev, (hipStream_t)stream, &p);
    if (st != VX_OK)
        return st;
    return vxi_gemm_scratch(batch, M, N, K, dtype, A, strideA, B, strideB, C, strideC, stream, p, kScratchTickets,
                            kScratchPartials);
}
