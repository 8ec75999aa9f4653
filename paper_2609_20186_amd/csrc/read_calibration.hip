// read_calibration.hip -- the achievable HBM read rate of one launch of a
// given size on this GPU, with the access pattern of the verify argmax
// stream: 256-lane work-groups each reading a contiguous share in 16 KB
// chunks of 16-byte nontemporal loads, the next chunk in flight while the
// current one is reduced (an integer maximum, so that no load is dead); and a
// delay kernel that lets the benchmark queue its timed launches before they
// run.  Measurement support for the benchmark; not part of the step's
// library.
#include <hip/hip_runtime.h>

#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kThreads = 256, kUnroll = 4, kChunkVecs = kThreads * kUnroll;

__device__ __forceinline__ void load(u32x4 (&v)[kUnroll], const u32x4 *p, int64_t q0, int64_t n) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
        const int64_t q = q0 + u * kThreads + threadIdx.x;
        v[u] = __builtin_nontemporal_load(p + (q < n ? q : n - 1));
    }
}

__device__ __forceinline__ uint32_t vmax(const u32x4 (&v)[kUnroll], uint32_t m) {
#pragma unroll
    for (int u = 0; u < kUnroll; ++u)
        m = max(max(max(m, v[u][0]), max(v[u][1], v[u][2])), v[u][3]);
    return m;
}

// Work-group g reads chunks [C g / G, C (g + 1) / G) with `kDepth` chunks in
// flight: the loop is unrolled by kDepth so that every buffer is a fixed set
// of registers.
template <int kDepth>
__global__ __launch_bounds__(kThreads) void k_read(const u32x4 *src, int64_t nvec, uint32_t *out) {
    const int64_t g = blockIdx.x, G = gridDim.x;
    const int64_t C = (nvec + kChunkVecs - 1) / kChunkVecs;
    const int64_t c0 = C * g / G, c1 = C * (g + 1) / G;
    uint32_t m = 0;
    u32x4 buf[kDepth][kUnroll];
#pragma unroll
    for (int j = 0; j < kDepth - 1; ++j)
        if (c0 + j < c1)
            load(buf[j], src, (c0 + j) * kChunkVecs, nvec);
    for (int64_t c = c0; c < c1; c += kDepth) {
#pragma unroll
        for (int j = 0; j < kDepth; ++j) {
            if (c + j + kDepth - 1 < c1)
                load(buf[(j + kDepth - 1) % kDepth], src, (c + j + kDepth - 1) * kChunkVecs, nvec);
            if (c + j < c1)
                m = vmax(buf[j], m);
        }
    }
    // one word per work-group (the lanes' maximum), so the loads are live
    __shared__ uint32_t red;
    if (threadIdx.x == 0)
        red = 0;
    __syncthreads();
    atomicMax(&red, m);
    __syncthreads();
    if (threadIdx.x == 0)
        out[g] = red;
}

// Static share, then dynamic claims: chunks [0, S) are split evenly over the
// work-groups (two in flight); chunks [S, C) form 8 pools, one per XCD
// (work-groups are dispatched to the XCDs in turn, block index mod 8), from
// which wave 0 claims one chunk at a time with an atomic on the pool's
// counter, one claim ahead of the chunk being reduced, moving on to the next
// pool when one runs dry.  ctr: 8 zeroed counters per launch.
__global__ __launch_bounds__(kThreads) void k_read_dyn(const u32x4 *src, int64_t nvec,
                                                       int64_t S, uint32_t *ctr, uint32_t *out) {
    const int64_t g = blockIdx.x, G = gridDim.x;
    const int64_t C = (nvec + kChunkVecs - 1) / kChunkVecs;
    const int64_t c0 = S * g / G, c1 = S * (g + 1) / G;
    uint32_t m = 0;
    u32x4 A[kUnroll], B[kUnroll];
    __shared__ int64_t claim[2];
    const int x0 = (int)(g & 7);
    int pool = 0;  // pools tried so far (wave 0, lane 0)
    // claims chunk indices from the pools; -1 when every pool is empty
    auto next_claim = [&]() -> int64_t {
        while (pool < 8) {
            const int x = (x0 + pool) & 7;
            const int64_t p0 = S + (C - S) * x / 8, p1 = S + (C - S) * (x + 1) / 8;
            const uint32_t i = atomicAdd(&ctr[x * 16], 1u);
            if (p0 + (int64_t)i < p1)
                return p0 + i;
            ++pool;
        }
        return -1;
    };
    if (threadIdx.x == 0)
        claim[0] = next_claim();
    // the static share, two in flight
    if (c0 < c1) {
        load(A, src, c0 * kChunkVecs, nvec);
        int64_t c = c0;
        for (; c + 1 < c1; c += 2) {
            load(B, src, (c + 1) * kChunkVecs, nvec);
            m = vmax(A, m);
            load(A, src, (c + 2 < c1 ? c + 2 : c + 1) * kChunkVecs, nvec);
            m = vmax(B, m);
        }
        if (c < c1)
            m = vmax(A, m);
    }
    __syncthreads();
    int64_t cur = claim[0];
    int k = 0;
    if (cur >= 0)
        load(A, src, cur * kChunkVecs, nvec);
    while (cur >= 0) {
        if (threadIdx.x == 0)
            claim[(k + 1) & 1] = next_claim();
        __syncthreads();
        const int64_t nxt = claim[(k + 1) & 1];
        if (nxt >= 0)
            load(B, src, nxt * kChunkVecs, nvec);
        m = vmax(A, m);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            A[u] = B[u];
        cur = nxt;
        ++k;
        __syncthreads();
    }
    __shared__ uint32_t red;
    if (threadIdx.x == 0)
        red = 0;
    __syncthreads();
    atomicMax(&red, m);
    __syncthreads();
    if (threadIdx.x == 0)
        out[g] = red;
}

// Holds the stream for `ticks` of the 100 MHz real-time clock (bounded: it
// exits when the time is up).
__global__ void k_delay(uint64_t ticks) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (__builtin_amdgcn_s_memrealtime() - t0 < ticks)
        __builtin_amdgcn_s_sleep(8);
}

}  // namespace

// The static-plus-claims variant: `static_percent` of the chunks split
// evenly, the rest claimed from 8 per-XCD pools; ctr: 8 zeroed counters, each
// on its own 64-byte line (128 uint32), used by this launch only.
extern "C" int switchsd_calibrate_read_dyn(const void *src, int64_t bytes, int32_t workgroups,
                                           int32_t static_percent, uint32_t *ctr, uint32_t *out,
                                           hipStream_t stream) {
    if (!src || !out || !ctr || bytes < 16 || (bytes & 15) || ((uintptr_t)src & 15) ||
        workgroups < 1 || static_percent < 0 || static_percent > 100)
        return -1;
    const int64_t nvec = bytes / 16;
    const int64_t C = (nvec + kChunkVecs - 1) / kChunkVecs;
    hipLaunchKernelGGL(k_read_dyn, dim3((unsigned)workgroups), dim3(kThreads), 0, stream,
                       (const u32x4 *)src, nvec, C * static_percent / 100, ctr, out);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

// Measurement support: a one-lane kernel that returns after `microseconds`
// (at most one second), so that launches queued behind it start back to
// back.  Returns 0, -1 for a bad argument, -3 for a failed launch.
extern "C" int switchsd_calibrate_delay(double microseconds, hipStream_t stream) {
    if (!(microseconds >= 0.0) || microseconds > 1e6)
        return -1;
    hipLaunchKernelGGL(k_delay, dim3(1), dim3(1), 0, stream, (uint64_t)(microseconds * 100.0));
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

// Reads `bytes` (a multiple of 16, 16-byte aligned device memory) with
// `workgroups` work-groups and `depth` (1..4) 16 KB chunks in flight per
// work-group; out [workgroups] receives one word each.  Returns 0, -1 for bad
// arguments, -3 for a failed launch.
extern "C" int switchsd_calibrate_read(const void *src, int64_t bytes, int32_t workgroups,
                                       int32_t depth, uint32_t *out, hipStream_t stream) {
    if (!src || !out || bytes < 16 || (bytes & 15) || ((uintptr_t)src & 15) || workgroups < 1 ||
        depth < 1 || depth > 4)
        return -1;
    const dim3 g((unsigned)workgroups), t(kThreads);
    const u32x4 *s = (const u32x4 *)src;
    switch (depth) {
    case 1:
        hipLaunchKernelGGL(k_read<1>, g, t, 0, stream, s, bytes / 16, out);
        break;
    case 2:
        hipLaunchKernelGGL(k_read<2>, g, t, 0, stream, s, bytes / 16, out);
        break;
    case 3:
        hipLaunchKernelGGL(k_read<3>, g, t, 0, stream, s, bytes / 16, out);
        break;
    default:
        hipLaunchKernelGGL(k_read<4>, g, t, 0, stream, s, bytes / 16, out);
        break;
    }
    return hipGetLastError() == hipSuccess ? 0 : -3;
}
