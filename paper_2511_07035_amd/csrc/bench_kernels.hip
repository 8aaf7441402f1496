// bench_kernels.hip -- device helpers of the benchmark harness (not part of
// the checkpoint path).
//
//   gockpt_bench_spin   stand-in for a training step's forward/backward: one
//                       wavefront per compute unit waits on the constant-rate
//                       wall clock for the requested time.  Every wave exits
//                       after the deadline or after a hard iteration cap.
//   gockpt_bench_hog    the same wait in blocks of four wavefronts, enough of
//                       them to hold every wave slot of the device: work that
//                       needs compute units cannot start beside it.
//   gockpt_bench_copy   plain 16-byte-vector device copy of a known size, the
//                       reference for achievable HBM bandwidth and for scaling
//                       the hardware byte counters.
//   gockpt_bench_convert  the 16-bit conversions of the arithmetic contract on
//                       the device, over a range of bit patterns: fp32 ->
//                       bf16 (round to nearest even), bf16 -> fp32 and fp16
//                       -> fp32, the functions the update kernel inlines.
//   gockpt_bench_divsqrt  q = a / b and r = sqrt(a) in fp32 on the device,
//                       built with the library's flags, so tests can check
//                       the device's division and square root bit for bit
//                       against the host's IEEE operations.
//   gockpt_bench_stream HBM ceilings of this device for the access patterns
//                       the hot path uses: read-only, write-only, and a
//                       memory twin of the fused update (same quads, same
//                       five input and four output streams, trivial math).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gockpt_contract.h"

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

__global__ __launch_bounds__(256) void hog_kernel(uint64_t ticks, uint64_t max_iter) {
    const uint64_t t0 = wall_clock64();
    uint64_t it = 0;
    while (wall_clock64() - t0 < ticks && it < max_iter) {
        __builtin_amdgcn_s_sleep(8);
        ++it;
    }
}

__global__ __launch_bounds__(256) void convert_kernel(int mode, uint64_t base, uint64_t count, void* out) {
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < count; i += stride) {
        const uint64_t x = base + i;
        if (mode == 0)
            static_cast<uint16_t*>(out)[i] = gockpt::f32_to_bf16_rne(gockpt::bits_to_f32(static_cast<uint32_t>(x)));
        else if (mode == 1)
            static_cast<uint32_t*>(out)[i] = gockpt::f32_to_bits(gockpt::bf16_to_f32(static_cast<uint16_t>(x)));
        else
            static_cast<uint32_t*>(out)[i] = gockpt::f32_to_bits(gockpt::fp16_to_f32(static_cast<uint16_t>(x)));
    }
}

__global__ __launch_bounds__(256) void copy_kernel(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                   uint64_t n16) {
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride)
        dst[i] = src[i];
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void read_kernel(const u32x4* __restrict__ a, uint64_t n16, uint32_t* sink) {
    uint32_t acc = 0;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16; i += stride) {
        const u32x4 v = __builtin_nontemporal_load(a + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9E3779B9u && sink != nullptr) sink[0] = acc;  // keeps the loads alive
}

__global__ __launch_bounds__(256) void write_kernel(u32x4* __restrict__ a, uint64_t n16) {
    const uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n16) a[i] = (u32x4){1u, 2u, 3u, 4u};
}

// Same memory pattern as the fused update, one quad of 4 elements per lane:
// read g (8 B), p, m, v (16 B each); write p, m, v (16 B each), w (8 B).
__global__ __launch_bounds__(256) void twin_kernel(const u32x2* __restrict__ g, f32x4* __restrict__ p,
                                                   f32x4* __restrict__ m, f32x4* __restrict__ v,
                                                   u32x2* __restrict__ w, uint64_t nquads) {
    const uint64_t q = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q >= nquads) return;
    const u32x2 gg = g[q];
    const f32x4 a = p[q], b = m[q], c = v[q];
    const float x = __uint_as_float(gg.x << 16);
    p[q] = a + x;
    m[q] = b + x;
    v[q] = c + x;
    w[q] = gg ^ (u32x2){1u, 1u};
}

__global__ __launch_bounds__(256) void divsqrt_kernel(const float* __restrict__ a, const float* __restrict__ b,
                                                      float* __restrict__ q, float* __restrict__ r, uint64_t n) {
    const uint64_t i = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    q[i] = a[i] / b[i];
    r[i] = __builtin_sqrtf(a[i]);
}

}  // namespace

extern "C" {

// mode 0: out (uint16[count]) = bf16_rne(fp32 with bits base + i), base +
// count <= 2^32; mode 1: out (uint32[count]) = bits of bf16_to_f32(base + i),
// mode 2: the same for fp16_to_f32, base + count <= 2^16 for both.
int gockpt_bench_convert(int mode, uint64_t base, uint64_t count, void* out, void* stream) {
    if (mode < 0 || mode > 2 || out == nullptr) return -1;
    if (base + count > (mode == 0 ? (1ull << 32) : (1ull << 16))) return -1;
    if (count == 0) return 0;
    uint64_t grid = (count + 255) / 256;
    if (grid > 65536) grid = 65536;
    hipLaunchKernelGGL(convert_kernel, dim3(static_cast<unsigned>(grid)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), mode, base, count, out);
    return static_cast<int>(hipGetLastError());
}

// n elements; a, b, q, r device fp32 arrays of n.
int gockpt_bench_divsqrt(const void* a, const void* b, void* q, void* r, uint64_t n, void* stream) {
    if (n == 0) return 0;
    const uint64_t grid = (n + 255) / 256;
    if (grid > 0xFFFFFFFFull) return -1;
    hipLaunchKernelGGL(divsqrt_kernel, dim3(static_cast<unsigned>(grid)), dim3(256), 0, static_cast<hipStream_t>(stream),
                       static_cast<const float*>(a), static_cast<const float*>(b), static_cast<float*>(q),
                       static_cast<float*>(r), n);
    return static_cast<int>(hipGetLastError());
}

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

// `blocks` blocks of 256 threads wait `ms` milliseconds (0 < ms <= 60000) on
// `stream`; blocks beyond what the device holds at once start when earlier
// ones end.
int gockpt_bench_hog(void* stream, double ms, int blocks) {
    if (!(ms > 0.0) || ms > 60000.0 || blocks < 1 || blocks > 65536) return -1;
    const int khz = gockpt_bench_wallclock_khz();
    if (khz <= 0) return -5;
    const uint64_t ticks = static_cast<uint64_t>(ms * static_cast<double>(khz));
    hipLaunchKernelGGL(hog_kernel, dim3(blocks), dim3(256), 0, static_cast<hipStream_t>(stream), ticks,
                       ticks + 1000000ull);
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

// mode 0: read `a` (bytes), 1: write `a` (bytes), 2: fused-update twin over
// n elements (a = bf16 gradients, b/c/d = fp32 p/m/v, e = bf16 weights).
// Buffers 16-byte aligned; sizes multiples of 16 bytes (mode 2: n multiple of 4).
int gockpt_bench_stream(int mode, void* a, void* b, void* c, void* d, void* e, uint64_t bytes_or_n, void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    if ((reinterpret_cast<uintptr_t>(a) % 16) != 0) return -1;
    if (mode == 0) {
        if (bytes_or_n % 16 != 0) return -1;
        hipLaunchKernelGGL(read_kernel, dim3(2048), dim3(256), 0, s, static_cast<const u32x4*>(a), bytes_or_n / 16,
                           static_cast<uint32_t*>(nullptr));
    } else if (mode == 1) {
        if (bytes_or_n % 16 != 0) return -1;
        const uint64_t n16 = bytes_or_n / 16;
        const uint64_t grid = (n16 + 255) / 256;
        if (grid == 0 || grid > 0xFFFFFFFFull / 256) return -1;
        hipLaunchKernelGGL(write_kernel, dim3(static_cast<unsigned>(grid)), dim3(256), 0, s, static_cast<u32x4*>(a),
                           n16);
    } else if (mode == 2) {
        if (bytes_or_n % 4 != 0 || !b || !c || !d || !e) return -1;
        const uint64_t nq = bytes_or_n / 4;
        const uint64_t grid = (nq + 255) / 256;
        if (grid == 0 || grid > 0xFFFFFFFFull / 256) return -1;
        hipLaunchKernelGGL(twin_kernel, dim3(static_cast<unsigned>(grid)), dim3(256), 0, s,
                           static_cast<const u32x2*>(a), static_cast<f32x4*>(b), static_cast<f32x4*>(c),
                           static_cast<f32x4*>(d), static_cast<u32x2*>(e), nq);
    } else {
        return -1;
    }
    return static_cast<int>(hipGetLastError());
}

}  // extern "C"
