// gockpt_cast.hip -- bf16 weights re-derived from the fp32 master weights
// after a checkpoint is loaded (Sec. 4.3.2): w = bf16_rne(master), the same
// rounding the fused update applies, so the weights equal, bit for bit, those
// the training run held when the checkpoint was taken.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gockpt_contract.h"

namespace gockpt {

namespace {

// One quad per lane, grid-stride; the last n mod 4 elements by lane 0..3 of
// the first block.
__global__ __launch_bounds__(256) void cast_bf16_kernel(const float4* __restrict__ p, uint2* __restrict__ w,
                                                        const float* __restrict__ p_tail, uint16_t* __restrict__ w_tail,
                                                        uint64_t nquads, uint32_t tail) {
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * blockDim.x;
    for (uint64_t q = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x; q < nquads; q += stride) {
        const float4 x = p[q];
        uint2 o;
        o.x = static_cast<uint32_t>(f32_to_bf16_rne(x.x)) | (static_cast<uint32_t>(f32_to_bf16_rne(x.y)) << 16);
        o.y = static_cast<uint32_t>(f32_to_bf16_rne(x.z)) | (static_cast<uint32_t>(f32_to_bf16_rne(x.w)) << 16);
        w[q] = o;
    }
    if (blockIdx.x == 0 && threadIdx.x < tail) w_tail[threadIdx.x] = f32_to_bf16_rne(p_tail[threadIdx.x]);
}

}  // namespace

// p and w: device arrays of n elements, 16- and 8-byte aligned.
int launch_cast_bf16(const float* p, uint16_t* w, int64_t n, hipStream_t stream) {
    if (n <= 0) return hipSuccess;
    const uint64_t nquads = static_cast<uint64_t>(n) / 4;
    const uint32_t tail = static_cast<uint32_t>(n % 4);
    uint64_t blocks = (nquads + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (blocks == 0) blocks = 1;
    hipLaunchKernelGGL(cast_bf16_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream,
                       reinterpret_cast<const float4*>(p), reinterpret_cast<uint2*>(w), p + nquads * 4,
                       w + nquads * 4, nquads, tail);
    return static_cast<int>(hipGetLastError());
}

}  // namespace gockpt
