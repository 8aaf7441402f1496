// bench_kernels.hip -- device helpers of the benchmark harness (not part of
// the checkpoint path).
//
//   gockpt_bench_spin   stand-in for a training step's forward/backward: one
//                       wavefront per compute unit waits on the constant-rate
//                       wall clock for the requested time.  Every wave exits
//                       after the deadline or after a hard iteration cap.
//   gockpt_bench_copy   plain 16-byte-vector device copy of a known size, the
//                       reference for achievable HBM bandwidth and for scaling
//                       the hardware byte counters.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(64) void spin_kernel(uint64_t ticks, uint64_t max_iter, uint32_t* sink) {
    const uint64_t t0 = wall_clock64();
    uint64_t it = 0;
    while (wall_clock64() - t0 < ticks && it < max_iter) {
        __builtin_amdgcn_s_sleep(8);
        ++it;
    }
    if (threadIdx.x == 0 && blockIdx.x == 0 && sink != nullptr) sink[0] = static_cast<uint32_t>(it);
}

__global__ __launch_bounds__(256) void copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                   uint64_t n16) {
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride)
        dst[i] = src[i];
}

}  // namespace

extern "C" {

// Wall-clock counter rate in kHz (0 on error).
int gockpt_bench_wallclock_khz(void) {
    int dev = 0, khz = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    if (hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) return 0;
    return khz;
}

// Occupy the device for `ms` milliseconds on `stream` (0 < ms <= 60000).
int gockpt_bench_spin(void* stream, double ms, int n_waves) {
    if (!(ms > 0.0) || ms > 60000.0 || n_waves < 1 || n_waves > 65536) return -1;
    const int khz = gockpt_bench_wallclock_khz();
    if (khz <= 0) return -5;
    const uint64_t ticks = static_cast<uint64_t>(ms * static_cast<double>(khz));
    // One loop iteration sleeps far longer than one wall-clock tick, so the
    // cap only ends a wave whose clock would not advance.
    const uint64_t max_iter = ticks + 1000000ull;
    hipLaunchKernelGGL(spin_kernel, dim3(n_waves), dim3(64), 0, static_cast<hipStream_t>(stream), ticks, max_iter,
                       static_cast<uint32_t*>(nullptr));
    return static_cast<int>(hipGetLastError());
}

// dst <- src, `bytes` a multiple of 16, both 16-byte aligned.
int gockpt_bench_copy(void* dst, const void* src, uint64_t bytes, int grid, void* stream) {
    if (bytes % 16 != 0 || (reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src)) % 16 != 0)
        return -1;
    if (grid < 1) grid = 1;
    hipLaunchKernelGGL(copy_kernel, dim3(grid), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const u32x4*>(src), static_cast<u32x4*>(dst), bytes / 16);
    return static_cast<int>(hipGetLastError());
}

}  // extern "C"
