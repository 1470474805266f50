// probes.hip -- measurement kernels (not part of the compute path).
//
// HBM read probe: streams `bytes` of device memory with 16-byte loads, four
// in flight per thread, and folds them into one word per workgroup so the
// loads cannot be dropped.  Timed over the byte count an HBM-bound kernel
// moves, it gives the read bandwidth this GPU sustains at that size -- the
// measured ceiling the attention and score kernels are compared with, next
// to the published 8 TB/s.
#include "pulse_internal.h"

namespace pulse {

constexpr int kProbeThreads = 256;
constexpr int kProbeGrid = 2048;

__global__ __launch_bounds__(kProbeThreads) void probe_hbm_read_kernel(const u32x4* __restrict__ src, int64_t n16,
                                                                       uint32_t* __restrict__ sink) {
    uint32_t acc = 0;
    const int64_t stride = (int64_t)gridDim.x * kProbeThreads;
    int64_t i = (int64_t)blockIdx.x * kProbeThreads + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 a = __builtin_nontemporal_load(src + i);
        const u32x4 b = __builtin_nontemporal_load(src + i + stride);
        const u32x4 c = __builtin_nontemporal_load(src + i + 2 * stride);
        const u32x4 d = __builtin_nontemporal_load(src + i + 3 * stride);
        acc ^= a[0] ^ a[1] ^ a[2] ^ a[3] ^ b[0] ^ b[1] ^ b[2] ^ b[3];
        acc ^= c[0] ^ c[1] ^ c[2] ^ c[3] ^ d[0] ^ d[1] ^ d[2] ^ d[3];
    }
    for (; i < n16; i += stride) {
        const u32x4 a = __builtin_nontemporal_load(src + i);
        acc ^= a[0] ^ a[1] ^ a[2] ^ a[3];
    }
    __shared__ uint32_t red[kProbeThreads / kWave];
    for (int off = 32; off >= 1; off >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, off);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = 0;
        for (int w = 0; w < kProbeThreads / kWave; ++w) r ^= red[w];
        sink[blockIdx.x] = r;
    }
}

int32_t probe_hbm_sink_words() { return kProbeGrid; }

hipError_t launch_probe_hbm_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t st, hipEvent_t start,
                                 hipEvent_t stop) {
    const int64_t n16 = (int64_t)(bytes / 16);
    if (n16 == 0) return hipSuccess;
    // enough workgroups for four loads in flight per thread, at most kProbeGrid
    const int64_t need = (n16 + 4 * kProbeThreads - 1) / (4 * kProbeThreads);
    const unsigned grid = (unsigned)(need < 1 ? 1 : (need < kProbeGrid ? need : kProbeGrid));
    launch_timed(probe_hbm_read_kernel, dim3(grid), dim3(kProbeThreads), 0u, st, start, stop, (const u32x4*)src, n16,
                 sink);
    return hipGetLastError();
}

}  // namespace pulse
