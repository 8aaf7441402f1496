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
//   gockpt_bench_fill_grads  one step's synthetic 16-bit gradients, standing
//                       in for the backward's writes of the gradient buffer:
//                       N(0, sigma) or Laplace(0, b) from a counter-based
//                       generator, times the loss scale, rounded to bf16 or
//                       fp16 by HIP's own conversions; optionally +inf at one
//                       index.
#include <hip/hip_bf16.h>
#include <hip/hip_fp16.h>
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

// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11): ten rounds of two
// 32x32->64 multiplications with the round keys bumped by the Weyl constants.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint2 k) {
#pragma unroll
    for (int r = 0; r < 10; ++r) {
        const uint32_t lo0 = 0xD2511F53u * c.x, hi0 = __umulhi(0xD2511F53u, c.x);
        const uint32_t lo1 = 0xCD9E8D57u * c.z, hi1 = __umulhi(0xCD9E8D57u, c.z);
        c = make_uint4(hi1 ^ c.y ^ k.x, lo1, hi0 ^ c.w ^ k.y, lo0);
        k.x += 0x9E3779B9u;
        k.y += 0xBB67AE85u;
    }
    return c;
}

// Uniform in the open interval (0, 1) from the top 23 bits: (k + 1/2) 2^-23
// is exact in fp32 for every k < 2^23, so the largest value is 1 - 2^-24.
__device__ __forceinline__ float unit_open(uint32_t r) {
    return (static_cast<float>(r >> 9) + 0.5f) * 1.1920928955078125e-07f;
}

// law 0: N(0, param) by Box-Muller, 1: Laplace(0, param) by the inverse CDF.
// Each lane draws 8 values (two Philox blocks keyed by the seed, counter =
// group index) and stores them as one 16-byte vector.
__global__ __launch_bounds__(256) void fill_grads_kernel(uint16_t* __restrict__ out, uint64_t n, uint2 key, int law,
                                                         float param, float scale, int fp16, int64_t plant) {
    const uint64_t ngroups = (n + 7) / 8;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t gi = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; gi < ngroups; gi += stride) {
        const uint32_t lo = static_cast<uint32_t>(gi), hi = static_cast<uint32_t>(gi >> 32);
        const uint4 a = philox4x32_10(make_uint4(lo, hi, 0u, 0u), key);
        const uint4 b = philox4x32_10(make_uint4(lo, hi, 1u, 0u), key);
        const uint32_t r[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        float x[8];
        if (law == 0) {
#pragma unroll
            for (int j = 0; j < 8; j += 2) {
                const float rad = sqrtf(-2.0f * logf(unit_open(r[j])));
                float sn, cs;
                sincosf(6.2831853071795865f * unit_open(r[j + 1]), &sn, &cs);
                x[j] = rad * cs * param;
                x[j + 1] = rad * sn * param;
            }
        } else {
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const float u = unit_open(r[j]) - 0.5f;  // exact: |u| <= 1/2 - 2^-24, so 1 - 2|u| > 0
                const float mag = -param * logf(1.0f - 2.0f * fabsf(u));
                x[j] = u < 0.0f ? -mag : mag;
            }
        }
        uint16_t h[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const float v = x[j] * scale;
            h[j] = fp16 ? __half_as_ushort(__float2half(v)) : __bfloat16_as_ushort(__float2bfloat16(v));
        }
        const uint64_t i0 = gi * 8;
        if (plant >= 0 && static_cast<uint64_t>(plant) >= i0 && static_cast<uint64_t>(plant) < i0 + 8)
            h[plant - static_cast<int64_t>(i0)] = fp16 ? 0x7C00u : 0x7F80u;
        if (i0 + 8 <= n) {
            u32x4 v;
            v.x = h[0] | (static_cast<uint32_t>(h[1]) << 16);
            v.y = h[2] | (static_cast<uint32_t>(h[3]) << 16);
            v.z = h[4] | (static_cast<uint32_t>(h[5]) << 16);
            v.w = h[6] | (static_cast<uint32_t>(h[7]) << 16);
            __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(out + i0));
        } else {
            for (uint64_t j = 0; i0 + j < n; ++j) out[i0 + j] = h[j];
        }
    }
}

}  // namespace

extern "C" {

// One step's gradients into out (uint16[n], 16-byte aligned): law 0 N(0,
// param), 1 Laplace(0, param), each value times `scale`, rounded to bf16
// (fp16 = 0) or fp16 (fp16 = 1); plant_index >= 0 sets that element to +inf.
// The draw depends only on (seed, element index).
int gockpt_bench_fill_grads(void* out, uint64_t n, uint64_t seed, int law, float param, float scale, int fp16,
                            int64_t plant_index, void* stream) {
    if (out == nullptr || (reinterpret_cast<uintptr_t>(out) % 16) != 0 || law < 0 || law > 1) return -1;
    if (plant_index >= 0 && static_cast<uint64_t>(plant_index) >= n) return -1;
    if (n == 0) return 0;
    const uint64_t groups = (n + 7) / 8;
    uint64_t grid = (groups + 255) / 256;
    if (grid > 65536) grid = 65536;
    const uint2 key = make_uint2(static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32));
    hipLaunchKernelGGL(fill_grads_kernel, dim3(static_cast<unsigned>(grid)), dim3(256), 0,
                       static_cast<hipStream_t>(stream), static_cast<uint16_t*>(out), n, key, law, param, scale,
                       fp16, plant_index);
    return static_cast<int>(hipGetLastError());
}

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
