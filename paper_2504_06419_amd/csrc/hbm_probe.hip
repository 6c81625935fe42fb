// hbm_probe.hip -- streaming-read probe (gfx950).
//
// The rate at which a plain streaming kernel reads HBM on this device: the
// practical ceiling the attention kernels are compared against, next to the
// 8 TB/s of the specification.  Like the attention kernels, every wave streams
// its own contiguous share of the buffer, kProbeUnroll 1 KB nontemporal loads
// in flight (a grid-stride sweep of the whole buffer measured 10 % slower,
// plain loads 13 % slower); 2048 waves, two per SIMD.  The loads are folded
// with XOR so they cannot be dropped, and every wave writes its fold to one
// sink word: the XOR of all sink words equals the XOR of every 32-bit word of
// the buffer.
#include "mfma_common.h"

namespace spire {

constexpr int kProbeThreads = 256;
constexpr int kProbeUnroll = 8;
constexpr int kProbeWaves = SPIRE_HBM_PROBE_SINK_WORDS;

__global__ __launch_bounds__(kProbeThreads) void hbm_read_kernel(const u32x4 *buf, int64_t n16,
                                                                 uint32_t *sink) {
    const int lane = threadIdx.x & 63;
    const int64_t wid = (int64_t)blockIdx.x * (kProbeThreads / 64) + (threadIdx.x >> 6);
    // whole groups of 64 lanes x kProbeUnroll chunks per wave; the rest below
    const int64_t per = (n16 / kProbeWaves) & ~(int64_t)(64 * kProbeUnroll - 1);
    const u32x4 *p = buf + wid * per;
    u32x4 acc = u32x4{0u, 0u, 0u, 0u};
    for (int64_t j = 0; j < per; j += 64 * kProbeUnroll) {
        u32x4 v[kProbeUnroll];
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) v[u] = __builtin_nontemporal_load(p + j + 64 * u + lane);
#pragma unroll
        for (int u = 0; u < kProbeUnroll; ++u) acc ^= v[u];
    }
    // the last n16 - kProbeWaves * per chunks, spread over all threads
    for (int64_t i = (int64_t)kProbeWaves * per + (int64_t)blockIdx.x * kProbeThreads + threadIdx.x; i < n16;
         i += (int64_t)gridDim.x * kProbeThreads)
        acc ^= __builtin_nontemporal_load(buf + i);
    uint32_t x = acc.x ^ acc.y ^ acc.z ^ acc.w;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x ^= __shfl_xor(x, o);
    if (lane == 0) sink[wid] = x;
}

hipError_t launch_hbm_read(const void *buf, int64_t bytes, uint32_t *sink, hipStream_t st) {
    constexpr int grid = kProbeWaves / (kProbeThreads / 64);  // one sink word per wave
    hipLaunchKernelGGL(hbm_read_kernel, dim3(grid), dim3(kProbeThreads), 0, st,
                       static_cast<const u32x4 *>(buf), bytes / 16, sink);
    return hipGetLastError();
}

}  // namespace spire
