// gockpt_contract.h -- the arithmetic the device update and the host replay
// share.  Both sides include this file so that the restored checkpoint is the
// bit pattern the device would have produced (Sec. 4.3.1 requires the CPU
// reconstruction to equal a direct transfer of the last step's state).
//
// Every per-element operation is one IEEE-754 fp32 operation rounded to
// nearest even.  Translation units that include this file are built with
// -ffp-contract=off; the pragma below repeats that for this header.  fp32
// division and square root must be the correctly rounded ones (the HIP
// default; never built with fast-math or -fgpu-flush-denormals-to-zero).
#pragma once

#include <stdint.h>
#include <string.h>

#if defined(__HIPCC__)
#include <hip/hip_runtime.h>
#define GOCKPT_HD __host__ __device__ __forceinline__
#else
#define GOCKPT_HD static inline __attribute__((always_inline))
#endif

#pragma clang fp contract(off)

namespace gockpt {

// Optimizer constants of a context (fp64 as given by the caller).
struct HParams {
    double beta1, beta2, eps, weight_decay;
};

// Scalars of one step (see the contract in gockpt.h).
struct StepScalars {
    float b1, b2, omb1, omb2, eps;
    float decay, step_size, sqrt_bc2, inv_scale;
};

GOCKPT_HD float bits_to_f32(uint32_t u) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __uint_as_float(u);
#else
    float f;
    memcpy(&f, &u, 4);
    return f;
#endif
}

GOCKPT_HD uint32_t f32_to_bits(float f) {
#if defined(__HIP_DEVICE_COMPILE__)
    return __float_as_uint(f);
#else
    uint32_t u;
    memcpy(&u, &f, 4);
    return u;
#endif
}

// bf16 -> fp32 is exact.
GOCKPT_HD float bf16_to_f32(uint16_t b) { return bits_to_f32(static_cast<uint32_t>(b) << 16); }

// Gradient storage formats (the training run's 16-bit gradients are FP16 or
// BF16, Sec. 2.2).
enum GradKind : int { kGradBF16 = 0, kGradFP16 = 1 };

// fp16 -> fp32 is exact: the exponent is rebiased (15 -> 127) and the
// fraction widened; subnormal halves are normalised; infinities keep their
// sign; NaNs become quiet NaNs with the fraction in the top bits.
GOCKPT_HD float fp16_to_f32(uint16_t h) {
    const uint32_t sign = static_cast<uint32_t>(h & 0x8000u) << 16;
    const uint32_t e = (h >> 10) & 0x1Fu;
    const uint32_t f = h & 0x3FFu;
    uint32_t u;
    if (e == 0x1Fu) {
        u = sign | 0x7F800000u | (f ? (0x00400000u | (f << 13)) : 0u);
    } else if (e != 0u) {
        u = sign | ((e + 112u) << 23) | (f << 13);
    } else if (f == 0u) {
        u = sign;
    } else {
        const uint32_t k = 31u - static_cast<uint32_t>(__builtin_clz(f));  // leading bit, 0..9
        u = sign | ((k + 103u) << 23) | ((f << (23u - k)) & 0x7FFFFFu);
    }
    return bits_to_f32(u);
}

template <int kKind>
GOCKPT_HD float grad_to_f32(uint16_t b) {
    return kKind == kGradFP16 ? fp16_to_f32(b) : bf16_to_f32(b);
}

// inf or NaN: the exponent field is all ones.
template <int kKind>
GOCKPT_HD bool grad_nonfinite(uint16_t b) {
    return kKind == kGradFP16 ? (b & 0x7C00u) == 0x7C00u : (b & 0x7F80u) == 0x7F80u;
}

// fp32 -> bf16, round to nearest even; NaN -> canonical quiet 0x7FC0.
// Adding 0x7FFF plus the lowest kept bit carries into the kept half exactly
// when the dropped half is above 0x8000, or equal to it with an odd kept half.
GOCKPT_HD uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = f32_to_bits(f);
    if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u;
    u += 0x7FFFu + ((u >> 16) & 1u);
    return static_cast<uint16_t>(u >> 16);
}

// beta^t, fp64, square-and-multiply from the highest exponent bit down.  The
// loop starts at t's highest set bit: above it r stays exactly 1 (1 * 1 = 1),
// so starting there gives the same bits in fewer steps.
GOCKPT_HD double pow_int(double beta, int64_t t) {
    double r = 1.0;
    if (t <= 0) return r;
    for (int bit = 63 - __builtin_clzll(static_cast<unsigned long long>(t)); bit >= 0; --bit) {
        r = r * r;
        if ((t >> bit) & 1) r = r * beta;
    }
    return r;
}

GOCKPT_HD StepScalars step_scalars(const HParams& hp, float lr, int64_t t, float scale_used) {
    StepScalars s;
    const double bc1 = 1.0 - pow_int(hp.beta1, t);
    const double bc2 = 1.0 - pow_int(hp.beta2, t);
    const double lr_d = static_cast<double>(lr);
    s.b1 = static_cast<float>(hp.beta1);
    s.b2 = static_cast<float>(hp.beta2);
    s.omb1 = static_cast<float>(1.0 - hp.beta1);
    s.omb2 = static_cast<float>(1.0 - hp.beta2);
    s.eps = static_cast<float>(hp.eps);
    s.decay = static_cast<float>(1.0 - lr_d * hp.weight_decay);
    s.step_size = static_cast<float>(lr_d / bc1);
    const float bc2_f = static_cast<float>(bc2);
    s.sqrt_bc2 = __builtin_sqrtf(bc2_f);
    s.inv_scale = 1.0f / scale_used;
    return s;
}

// One AdamW update of one element: unscale, moments, decoupled decay, Adam
// step.  Written one rounded operation per statement.
template <int kKind = kGradBF16>
GOCKPT_HD void adamw_update(const StepScalars& s, uint16_t gbits, float& p, float& m, float& v) {
    float g = grad_to_f32<kKind>(gbits);
    g = g * s.inv_scale;
    const float m_keep = s.b1 * m;
    const float m_new = s.omb1 * g;
    m = m_keep + m_new;
    const float g2 = g * g;
    const float v_keep = s.b2 * v;
    const float v_new = s.omb2 * g2;
    v = v_keep + v_new;
    p = p * s.decay;
    const float root = __builtin_sqrtf(v);
    float denom = root / s.sqrt_bc2;
    denom = denom + s.eps;
    const float ratio = m / denom;
    const float delta = s.step_size * ratio;
    p = p - delta;
}

}  // namespace gockpt
