// switchsd_noalloc.hip -- switchsd_step for callers that cannot allocate
// device memory (code under HIP graph capture, tight serving loops): the
// workspace and the T > 0 scratch come from a fixed array in device memory
// instead of the caller.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <atomic>

#include "switchsd.h"
#include "switchsd_internal.h"

namespace {

// Scratch of one GPU: the step's workspace, then the scratch of a draw at
// T > 0, each 256-byte aligned.  Held by every GPU the library runs on until
// the process ends.
constexpr size_t kScratchBytes = (size_t)SWITCHSD_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
// The device address of `scratch` on each GPU (the array's name in host code
// is only a host-side stand-in), set at the first call on that GPU.
std::atomic<void *> g_scratch[kMaxDevices];

__global__ __launch_bounds__(256) void k_zero(uint4 *p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
        p[i] = uint4{0u, 0u, 0u, 0u};
}

size_t round_up(size_t n) { return (n + 255) / 256 * 256; }

// The scratch of the current GPU.  At the first call on a GPU: its address
// from hipGetSymbolAddress (with that GPU current), then a clear on `stream`,
// ordered before the call's kernels (every kernel leaves the workspace zeroed
// again, so later calls need no clear).
int device_scratch(void **out, hipStream_t stream) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
        return SWITCHSD_EHIP;
    void *p = g_scratch[dev].load();
    if (!p) {
        void *q = nullptr;
        if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q)
            return SWITCHSD_EHIP;
        hipLaunchKernelGGL(k_zero, dim3(1024), dim3(256), 0, stream, (uint4 *)q,
                           kScratchBytes / sizeof(uint4));
        if (hipGetLastError() != hipSuccess)
            return SWITCHSD_EHIP;
        g_scratch[dev].store(q);
        p = q;
    }
    *out = p;
    return SWITCHSD_OK;
}

}  // namespace

extern "C" int switchsd_step_noalloc(const switchsd_step_args *args, hipStream_t stream) {
    // every argument is checked before the first call's clear is launched
    int rc = switchsd::check_step_args(args);
    if (rc || args->B == 0)
        return rc;
    const size_t ws = switchsd_workspace_bytes(args->B, args->R, args->Lmax, args->cfg.n_cand);
    const size_t sws =
        args->temperature != 0.0f ? switchsd_sample_workspace_bytes(args->B, args->R, args->V) : 0;
    if (round_up(ws) + sws > kScratchBytes)
        return SWITCHSD_ESCRATCH;
    void *base = nullptr;
    if ((rc = device_scratch(&base, stream)))
        return rc;
    switchsd_step_args a = *args;
    if (args->temperature != 0.0f) {
        a.sample_workspace = (char *)base + round_up(ws);
        a.sample_workspace_bytes = kScratchBytes - round_up(ws);
    }
    return switchsd_step(&a, base, round_up(ws), stream);
}
