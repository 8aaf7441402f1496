// gockpt_kernels.hip -- device side of the GoCkpt hot path for gfx950.
//
//   prepass_kernel   one read of the 16-bit gradients (bf16 or fp16, Sec. 2.2):
//                    inf/NaN test on the raw bits (loss-scale skip) and the
//                    sum of squares of the unscaled gradient; one partial per
//                    block.
//   scan_kernel      the prepass over one bucket of gradients [begin, end),
//                    run by the caller as soon as the backward has written
//                    it: inf/NaN test and the sum of squares of the scaled
//                    gradient in fp64 (the scale is applied at the finalize,
//                    so the scan does not depend on the previous step).
//   finalize_kernel  one block: reduces the partials (of the prepass or of the
//                    bucket scans) in a fixed order, moves the loss scaler
//                    and the step count, computes the step's scalars and
//                    writes the step record (and, inside a window, the skip
//                    decision to the host).
//   gate_kernel      one wavefront on the copy stream that waits until the
//                    host has emptied a staging slot before a copy reuses it.
//   fused_kernel     the mixed-precision AdamW update of every element
//                    (Sec. 2.2, AdamW of Sec. 4.3.1) fused with the window's
//                    pack (Sec. 4.2.1): the step's part of the updated state
//                    and the gradients of the parts already sent are written
//                    into the staging ring in the same pass over HBM.
//
// Memory layout: flat structure-of-arrays -- master, exp_avg, exp_avg_sq
// (fp32), working weights (bf16) and gradients (bf16 or fp16), each
// contiguous over the flat parameter space.  The fused kernel gives each lane
// one quad of 4 consecutive elements per tile (see fused_kernel); the prepass
// reads 8 gradients per lane per iteration.  The kernels are HBM-bound (28
// bytes per element per step plus the pack), so no LDS and no matrix cores:
// the work is elementwise.

#include <hip/hip_runtime.h>

#include "gockpt_internal.h"

#pragma clang fp contract(off)

namespace gockpt {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 ld_u32x4(const void* p) {
    return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ f32x4 ld_f32x4(const float* p) {
    return *reinterpret_cast<const f32x4*>(p);
}
__device__ __forceinline__ void st_f32x4(float* p, f32x4 v) {
    *reinterpret_cast<f32x4*>(p) = v;
}
__device__ __forceinline__ void st_u32x4(void* p, u32x4 v) {
    *reinterpret_cast<u32x4*>(p) = v;
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// State streams of the fused kernel: every byte is touched once per step and
// next used a whole training step later, far beyond what the caches hold, so
// loads and stores carry the nontemporal hint (measured on the update's
// memory twin: 6.19 -> 6.49 TB/s with the state spread over HBM).
template <bool kNT, class T>
__device__ __forceinline__ T ld_stream(const T* p) {
    if constexpr (kNT)
        return __builtin_nontemporal_load(p);
    else
        return *p;
}
template <bool kNT, class T>
__device__ __forceinline__ void st_stream(T* p, T v) {
    if constexpr (kNT)
        __builtin_nontemporal_store(v, p);
    else
        *p = v;
}

// Ring stores: the ring is only read back by the copy engine, so bypass the
// caches' retention policy with nontemporal stores.  `off` < 2*ring_bytes.
__device__ __forceinline__ void ring_st16(const PackPlan& pk, uint64_t off, u32x4 v) {
    if (off >= pk.ring_bytes) off -= pk.ring_bytes;
    u32x4* dst = reinterpret_cast<u32x4*>(pk.ring + off);
    if (pk.ring_nt)
        __builtin_nontemporal_store(v, dst);
    else
        *dst = v;
}
__device__ __forceinline__ void ring_st_f32x8(const PackPlan& pk, uint64_t off, f32x4 lo, f32x4 hi) {
    u32x4 a = __builtin_bit_cast(u32x4, lo);
    u32x4 b = __builtin_bit_cast(u32x4, hi);
    ring_st16(pk, off, a);
    ring_st16(pk, off + 16, b);
}
__device__ __forceinline__ void ring_st_u16(const PackPlan& pk, uint64_t off, uint16_t v) {
    if (off >= pk.ring_bytes) off -= pk.ring_bytes;
    *reinterpret_cast<uint16_t*>(pk.ring + off) = v;
}
__device__ __forceinline__ void ring_st_f32(const PackPlan& pk, uint64_t off, float v) {
    if (off >= pk.ring_bytes) off -= pk.ring_bytes;
    *reinterpret_cast<float*>(pk.ring + off) = v;
}

// ---------------------------------------------------------------------------
// Block reductions (4 wavefronts of 64).
// ---------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

template <int kThreads>
__device__ __forceinline__ void block_reduce(double& sum, uint32_t& flag) {
    static_assert(kThreads % 64 == 0, "wave multiple");
    constexpr int kWaves = kThreads / 64;
    __shared__ double s_sum[kWaves];
    __shared__ uint32_t s_flag[kWaves];
    sum = wave_sum(sum);
    flag = __any(flag != 0u) ? 1u : 0u;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    if (lane == 0) {
        s_sum[wave] = sum;
        s_flag[wave] = flag;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
        uint32_t f = 0u;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            t += s_sum[w];
            f |= s_flag[w];
        }
        sum = t;
        flag = f;
    }
}

// ---------------------------------------------------------------------------
// Prepass: inf/NaN flag + sum of squares of the unscaled gradient.
// ---------------------------------------------------------------------------
// Gradient value for the norm: fp16 through the hardware conversion, which
// is exact for every finite value and infinity (the norm is telemetry; the
// update uses the contract's widening).
template <int kKind>
__device__ __forceinline__ float norm_value(uint16_t h) {
    if constexpr (kKind == kGradFP16)
        return static_cast<float>(__builtin_bit_cast(_Float16, h));
    else
        return bf16_to_f32(h);
}

template <int kKind>
__device__ __forceinline__ uint32_t word_nonfinite(uint32_t w) {
    // two 16-bit values; exponent field all ones means inf or NaN
    return (grad_nonfinite<kKind>(static_cast<uint16_t>(w & 0xFFFFu)) ? 1u : 0u) |
           (grad_nonfinite<kKind>(static_cast<uint16_t>(w >> 16)) ? 1u : 0u);
}

// ---------------------------------------------------------------------------
// Finalize: skip decision, loss scaler, step count, scalars, record.  Run by
// one whole block of kBlock threads over the partials of the step.
// ---------------------------------------------------------------------------
__device__ void finalize_block(uint8_t* __restrict__ ws, const Partial* __restrict__ parts, int nparts,
                               const FinalizeArgs& fa) {
    // Thread t sums partials t, t + kBlock, ... in that order; the loads of
    // eight of them are issued before any is added, so one block does not
    // wait out eight memory latencies in a row.
    double acc = 0.0;
    uint32_t bad = 0u;
    constexpr int kBatch = 8;
    for (int b0 = 0; b0 < nparts; b0 += kBlock * kBatch) {
        double v[kBatch];
        int32_t f[kBatch];
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            const int b = b0 + k * kBlock + static_cast<int>(threadIdx.x);
            v[k] = b < nparts ? parts[b].sumsq : 0.0;
            f[k] = b < nparts ? parts[b].nonfinite : 0;
        }
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            acc += v[k];
            bad |= static_cast<uint32_t>(f[k]);
        }
    }
    block_reduce<kBlock>(acc, bad);
    if (threadIdx.x != 0) return;
    // a caller-side overflow test replaces the scan (NaN counts as set)
    if (fa.found_inf != nullptr) bad = (*fa.found_inf != 0.0f) ? 1u : 0u;

    const ScalerCfg& sc = fa.sc;
    DevScaler* st = reinterpret_cast<DevScaler*>(ws + kWsScalerOff);
    gockpt_step_record* rec = reinterpret_cast<gockpt_step_record*>(ws + kWsRecordsOff) + fa.slot;
    const float scale_used = st->scale;
    int64_t t = st->t;
    int64_t tracker = st->tracker;
    float scale = scale_used;
    const int skip = (sc.check_overflow != 0 && bad != 0u) ? 1 : 0;
    if (skip) {
        if (sc.dynamic_scale) {
            const float reduced = scale * sc.backoff_factor;
            scale = reduced < sc.min_scale ? sc.min_scale : reduced;
            tracker = 0;
        }
    } else {
        t = t + 1;
        if (sc.dynamic_scale) {
            tracker = tracker + 1;
            if (tracker == sc.growth_interval) {
                scale = scale * sc.growth_factor;
                tracker = 0;
            }
        }
    }
    st->t = t;
    st->tracker = tracker;
    st->scale = scale;

    const StepScalars s = step_scalars(fa.hp, fa.lr, t, scale_used);
    if (fa.raw) {  // bucket scans summed squares of the scaled gradients
        const double inv = static_cast<double>(s.inv_scale);
        acc = acc * inv * inv;
    }
    rec->t = t;
    rec->tracker = tracker;
    rec->scale_used = scale_used;
    rec->scale_next = scale;
    rec->lr = fa.lr;
    rec->skip = skip;
    rec->nonfinite = static_cast<int32_t>(bad);
    rec->window_step = fa.window_step;
    rec->gnorm2 = fa.norm_off ? -1.0 : acc;
    rec->step_size = s.step_size;
    rec->sqrt_bc2 = s.sqrt_bc2;
    rec->decay = s.decay;
    rec->inv_scale = s.inv_scale;
    // the host reads the decision from its own memory once the step's
    // finalize has completed (vector store, system scope)
    if (fa.skip_out != nullptr) __hip_atomic_store(fa.skip_out, skip, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// One 8-element group of gradients (16 B), nontemporal or cached.
template <bool kNT>
__device__ __forceinline__ u32x4 ld_group(const uint16_t* p) {
    return kNT ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)) : ld_u32x4(p);
}

template <bool kNT, int kKind>
__global__ __launch_bounds__(kBlock) void prepass_kernel(const uint16_t* __restrict__ g, int64_t n,
                                                         uint8_t* __restrict__ ws) {
    const DevScaler* st = reinterpret_cast<const DevScaler*>(ws + kWsScalerOff);
    Partial* parts = reinterpret_cast<Partial*>(ws + kWsPartialsOff);
    const float inv_scale = 1.0f / st->scale;
    const int64_t ngroups = n / kVec;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    double acc = 0.0;
    uint32_t bad = 0u;
    // the next group's load is issued before this group's arithmetic, so a
    // wave keeps a load in flight while it computes
    int64_t gi = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
    u32x4 next = (u32x4){0u, 0u, 0u, 0u};
    if (gi < ngroups) next = ld_group<kNT>(g + gi * kVec);
    for (; gi < ngroups; gi += stride) {
        const u32x4 raw = next;
        if (gi + stride < ngroups) next = ld_group<kNT>(g + (gi + stride) * kVec);
        float s = 0.0f;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t w = raw[k];
            bad |= word_nonfinite<kKind>(w);
            const float a = norm_value<kKind>(static_cast<uint16_t>(w & 0xFFFFu)) * inv_scale;
            const float b = norm_value<kKind>(static_cast<uint16_t>(w >> 16)) * inv_scale;
            s = s + a * a;
            s = s + b * b;
        }
        acc += static_cast<double>(s);
    }
    if (blockIdx.x == 0) {
        const int64_t i = ngroups * kVec + threadIdx.x;
        if (threadIdx.x < kVec && i < n) {
            const uint16_t h = g[i];
            bad |= grad_nonfinite<kKind>(h) ? 1u : 0u;
            const float a = norm_value<kKind>(h) * inv_scale;
            acc += static_cast<double>(a * a);
        }
    }
    block_reduce<kBlock>(acc, bad);
    // One partial per block; the finalize kernel reduces them.  (Having the
    // last block to finish run the finalize instead saves a launch, but needs
    // an agent-scope release per block, which on this chip writes back the
    // XCD's L2 each time: measured slower at every size.)
    if (threadIdx.x == 0) {
        parts[blockIdx.x].sumsq = acc;
        parts[blockIdx.x].nonfinite = static_cast<int32_t>(bad);
        parts[blockIdx.x].pad = 0;
    }
}

// ---------------------------------------------------------------------------
// Bucket scan: the prepass over [begin, end), begin a multiple of kVec (end
// too, unless it is n).  Squares are taken of the scaled values in fp64, so
// they cannot overflow; the finalize applies the step's inv_scale.
// ---------------------------------------------------------------------------
template <bool kNT, int kKind>
__global__ __launch_bounds__(kBlock) void scan_kernel(const uint16_t* __restrict__ g, int64_t begin, int64_t end,
                                                      Partial* __restrict__ parts) {
    const int64_t ngroups = (end - begin) / kVec;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock;
    const uint16_t* base = g + begin;
    double acc = 0.0;
    uint32_t bad = 0u;
    int64_t gi = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;  // next load in flight, as the prepass
    u32x4 next = (u32x4){0u, 0u, 0u, 0u};
    if (gi < ngroups) next = ld_group<kNT>(base + gi * kVec);
    for (; gi < ngroups; gi += stride) {
        const u32x4 raw = next;
        if (gi + stride < ngroups) next = ld_group<kNT>(base + (gi + stride) * kVec);
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const uint32_t w = raw[k];
            bad |= word_nonfinite<kKind>(w);
            const double a = static_cast<double>(norm_value<kKind>(static_cast<uint16_t>(w & 0xFFFFu)));
            const double b = static_cast<double>(norm_value<kKind>(static_cast<uint16_t>(w >> 16)));
            acc += a * a;
            acc += b * b;
        }
    }
    if (blockIdx.x == 0) {
        const int64_t i = begin + ngroups * kVec + threadIdx.x;
        if (threadIdx.x < kVec && i < end) {
            const uint16_t h = g[i];
            bad |= grad_nonfinite<kKind>(h) ? 1u : 0u;
            const double a = static_cast<double>(norm_value<kKind>(h));
            acc += a * a;
        }
    }
    block_reduce<kBlock>(acc, bad);
    if (threadIdx.x == 0) {
        parts[blockIdx.x].sumsq = acc;
        parts[blockIdx.x].nonfinite = static_cast<int32_t>(bad);
        parts[blockIdx.x].pad = 0;
    }
}

// ---------------------------------------------------------------------------
// Finalize on its own (bucket scans, a caller's flag, or no prepass at all).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void finalize_kernel(uint8_t* __restrict__ ws, const Partial* __restrict__ parts,
                                                          int nparts, FinalizeArgs fa) {
    finalize_block(ws, parts, nparts, fa);
}

// ---------------------------------------------------------------------------
// Gate of the staged copies: the copy stream goes on once the host has moved
// enough earlier copies out of their staging slots.  One wavefront polls the
// host's counter (system-scope loads, never cached) and sleeps between polls;
// every wave leaves after the deadline or an iteration cap at the latest.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void gate_kernel(const uint64_t* released, uint64_t target, uint64_t max_ticks,
                                                  uint32_t* timed_out) {
    const uint64_t t0 = wall_clock64();
    const uint64_t max_iter = max_ticks;  // at least one clock tick per iteration
    bool ok = false;
    for (uint64_t it = 0; it < max_iter; ++it) {
        const uint64_t v = __hip_atomic_load(released, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_SYSTEM);
        if (v >= target) {
            ok = true;
            break;
        }
        if (wall_clock64() - t0 >= max_ticks) break;
        __builtin_amdgcn_s_sleep(16);
    }
    if (!ok && threadIdx.x == 0) __hip_atomic_store(timed_out, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// ---------------------------------------------------------------------------
// Fused AdamW update + window pack.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
    return static_cast<uint32_t>(f32_to_bf16_rne(a)) | (static_cast<uint32_t>(f32_to_bf16_rne(b)) << 16);
}

__device__ __forceinline__ void ring_st8(const PackPlan& pk, uint64_t off, u32x2 v) {
    if (off >= pk.ring_bytes) off -= pk.ring_bytes;
    u32x2* dst = reinterpret_cast<u32x2*>(pk.ring + off);
    if (pk.ring_nt)
        __builtin_nontemporal_store(v, dst);
    else
        *dst = v;
}

__device__ __forceinline__ void ring_st_f32x4(const PackPlan& pk, uint64_t off, f32x4 v) {
    ring_st16(pk, off, __builtin_bit_cast(u32x4, v));
}

// A quad is 4 consecutive elements.  A block of kB threads owns a tile of
// kB * kQ quads; thread t takes quads t, t + kB, ..., so every load and store
// instruction of a wavefront covers 64 consecutive quads (1 KiB of fp32,
// 512 B of bf16) and concurrently running blocks walk memory in order.  All
// loads of a thread are issued before any arithmetic.  Chunk bounds are
// multiples of 8, so a quad never straddles a part boundary.
template <bool kHasW, int kQ, int kKind, bool kNT, int kB>
__global__ __launch_bounds__(kB) void fused_kernel(FusedArgs a) {
    const gockpt_step_record* rec = a.rec;
    const int skip = rec->skip;
    StepScalars s;
    s.b1 = a.b1;
    s.b2 = a.b2;
    s.omb1 = a.omb1;
    s.omb2 = a.omb2;
    s.eps = a.eps;
    s.decay = rec->decay;
    s.step_size = rec->step_size;
    s.sqrt_bc2 = rec->sqrt_bc2;
    s.inv_scale = rec->inv_scale;
    const PackPlan& pk = a.pack;

    const int64_t nquads = a.n / 4;
    const int64_t q_base = static_cast<int64_t>(blockIdx.x) * (kB * kQ) + threadIdx.x;

    u32x2 graw[kQ];
    f32x4 pv[kQ], mv[kQ], vv[kQ];
    bool live[kQ], pk_g[kQ], pk_p[kQ], pk_m[kQ], pk_v[kQ];
#pragma unroll
    for (int h = 0; h < kQ; ++h) {
        const int64_t q = q_base + static_cast<int64_t>(h) * kB;
        const int64_t i = q * 4;
        live[h] = q < nquads;
        pk_g[h] = live[h] && !skip && i < pk.g_end;  // a skipped step's gradients are never replayed
        const bool in_c = live[h] && i >= pk.cb;
        pk_p[h] = in_c && i < pk.s_end[0];
        pk_m[h] = in_c && i < pk.s_end[1];
        pk_v[h] = in_c && i < pk.s_end[2];
        graw[h] = (u32x2){0u, 0u};
        pv[h] = mv[h] = vv[h] = (f32x4){0.f, 0.f, 0.f, 0.f};
        if (live[h] && !skip) graw[h] = ld_stream<kNT>(reinterpret_cast<const u32x2*>(a.g + i));
        if (live[h] && (!skip || pk_p[h] || pk_m[h] || pk_v[h])) {
            pv[h] = ld_stream<kNT>(reinterpret_cast<const f32x4*>(a.p + i));
            mv[h] = ld_stream<kNT>(reinterpret_cast<const f32x4*>(a.m + i));
            vv[h] = ld_stream<kNT>(reinterpret_cast<const f32x4*>(a.v + i));
        }
    }
#pragma unroll
    for (int h = 0; h < kQ; ++h) {
        if (!live[h]) continue;
        const int64_t i = (q_base + static_cast<int64_t>(h) * kB) * 4;
        if (!skip) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const uint32_t word = graw[h][e >> 1];
                const uint16_t gb = static_cast<uint16_t>((e & 1) ? (word >> 16) : (word & 0xFFFFu));
                float p = pv[h][e], m = mv[h][e], v = vv[h][e];
                adamw_update<kKind>(s, gb, p, m, v);
                pv[h][e] = p;
                mv[h][e] = m;
                vv[h][e] = v;
            }
            st_stream<kNT>(reinterpret_cast<f32x4*>(a.p + i), pv[h]);
            st_stream<kNT>(reinterpret_cast<f32x4*>(a.m + i), mv[h]);
            st_stream<kNT>(reinterpret_cast<f32x4*>(a.v + i), vv[h]);
            if (kHasW) {
                const u32x2 wv = {pack2_bf16(pv[h][0], pv[h][1]), pack2_bf16(pv[h][2], pv[h][3])};
                st_stream<kNT>(reinterpret_cast<u32x2*>(a.w + i), wv);
            }
        }
        if (pk_g[h]) ring_st8(pk, pk.off_g + 2ull * static_cast<uint64_t>(i), graw[h]);
        const uint64_t rel = 4ull * static_cast<uint64_t>(i - pk.cb);
        if (pk_p[h]) ring_st_f32x4(pk, pk.off_s[0] + rel, pv[h]);
        if (pk_m[h]) ring_st_f32x4(pk, pk.off_s[1] + rel, mv[h]);
        if (pk_v[h]) ring_st_f32x4(pk, pk.off_s[2] + rel, vv[h]);
    }

    // Ragged tail: the last n % 4 elements, one per thread of block 0.
    if (blockIdx.x == 0 && threadIdx.x < 4) {
        const int64_t i = nquads * 4 + threadIdx.x;
        if (i < a.n) {
            const bool pack_g = !skip && i < pk.g_end;
            const bool in_c = i >= pk.cb;
            const uint16_t gb = a.g[i];
            float p = a.p[i], m = a.m[i], v = a.v[i];
            if (!skip) {
                adamw_update<kKind>(s, gb, p, m, v);
                a.p[i] = p;
                a.m[i] = m;
                a.v[i] = v;
                if (kHasW) a.w[i] = f32_to_bf16_rne(p);
            }
            if (pack_g) ring_st_u16(pk, pk.off_g + 2ull * static_cast<uint64_t>(i), gb);
            if (in_c) {
                const uint64_t rel = 4ull * static_cast<uint64_t>(i - pk.cb);
                if (i < pk.s_end[0]) ring_st_f32(pk, pk.off_s[0] + rel, p);
                if (i < pk.s_end[1]) ring_st_f32(pk, pk.off_s[1] + rel, m);
                if (i < pk.s_end[2]) ring_st_f32(pk, pk.off_s[2] + rel, v);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Launchers.
// ---------------------------------------------------------------------------
static int env_int(const char* name, int dflt) {
    const char* s = getenv(name);
    if (s == nullptr || *s == '\0') return dflt;
    return atoi(s);
}

int prepass_blocks_for(int64_t n) {
    const int64_t groups = n / kVec;
    int64_t b = (groups + kBlock - 1) / kBlock;
    if (b < 1) b = 1;
    if (b > kPrepassMaxBlocks) b = kPrepassMaxBlocks;
    return static_cast<int>(b);
}

int scan_blocks_for(int64_t count, int max_blocks) {
    // at least four 8-element groups per lane
    int64_t b = (count / kVec + 4 * kBlock - 1) / (4 * kBlock);
    if (b < 1) b = 1;
    if (b > max_blocks) b = max_blocks;
    return static_cast<int>(b);
}

int launch_scan(const uint16_t* g, int64_t begin, int64_t end, void* parts, int nblocks, int nt, int grad_kind,
                void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    Partial* p = static_cast<Partial*>(parts);
    if (grad_kind == kGradFP16) {
        if (nt)
            hipLaunchKernelGGL((scan_kernel<true, kGradFP16>), dim3(nblocks), dim3(kBlock), 0, s, g, begin, end, p);
        else
            hipLaunchKernelGGL((scan_kernel<false, kGradFP16>), dim3(nblocks), dim3(kBlock), 0, s, g, begin, end, p);
    } else {
        if (nt)
            hipLaunchKernelGGL((scan_kernel<true, kGradBF16>), dim3(nblocks), dim3(kBlock), 0, s, g, begin, end, p);
        else
            hipLaunchKernelGGL((scan_kernel<false, kGradBF16>), dim3(nblocks), dim3(kBlock), 0, s, g, begin, end, p);
    }
    return static_cast<int>(hipGetLastError());
}

Knobs default_knobs() {
    Knobs k;
    k.quads_per_thread = env_int("GOCKPT_QUADS", 1);
    k.ring_nt = env_int("GOCKPT_RING_NT", 1);
    k.prepass_nt = env_int("GOCKPT_PREPASS_NT", 1);
    k.fused_nt = env_int("GOCKPT_FUSED_NT", 1);
    k.fused_block = env_int("GOCKPT_FUSED_BLOCK", 0);
    return k;
}

int launch_prepass(const uint16_t* g, int64_t n, void* workspace, int nblocks, int nt, int grad_kind,
                   void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint8_t* ws = static_cast<uint8_t*>(workspace);
    if (nblocks < 1 || nblocks > kPrepassMaxBlocks) return static_cast<int>(hipErrorInvalidValue);
    if (grad_kind == kGradFP16) {
        if (nt)
            hipLaunchKernelGGL((prepass_kernel<true, kGradFP16>), dim3(nblocks), dim3(kBlock), 0, s, g, n, ws);
        else
            hipLaunchKernelGGL((prepass_kernel<false, kGradFP16>), dim3(nblocks), dim3(kBlock), 0, s, g, n, ws);
    } else {
        if (nt)
            hipLaunchKernelGGL((prepass_kernel<true, kGradBF16>), dim3(nblocks), dim3(kBlock), 0, s, g, n, ws);
        else
            hipLaunchKernelGGL((prepass_kernel<false, kGradBF16>), dim3(nblocks), dim3(kBlock), 0, s, g, n, ws);
    }
    return static_cast<int>(hipGetLastError());
}

int launch_finalize(void* workspace, const void* parts, int nparts, const FinalizeArgs& fin, void* stream) {
    hipLaunchKernelGGL(finalize_kernel, dim3(1), dim3(kBlock), 0, static_cast<hipStream_t>(stream),
                       static_cast<uint8_t*>(workspace), static_cast<const Partial*>(parts), nparts, fin);
    return static_cast<int>(hipGetLastError());
}

int launch_gate(const uint64_t* released, uint64_t target, uint64_t max_ticks, uint32_t* timed_out, void* stream) {
    hipLaunchKernelGGL(gate_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream), released, target,
                       max_ticks, timed_out);
    return static_cast<int>(hipGetLastError());
}

template <int kQ, int kKind, bool kNT, int kB>
static int launch_fused_q(const FusedArgs& a, hipStream_t s) {
    // one tile of kB * kQ quads per block (at least one block for the ragged
    // tail); the launch holds at most 2^32 - 1 threads, i.e. n < 1.7e10 * kQ
    // elements, beyond what three fp32 arrays fit in HBM
    const int64_t per_block = static_cast<int64_t>(kB) * kQ * 4;
    int64_t tiles = (a.n + per_block - 1) / per_block;
    if (tiles < 1) tiles = 1;
    if (tiles > static_cast<int64_t>(0xFFFFFFFFu / kB)) return static_cast<int>(hipErrorInvalidValue);
    const unsigned grid = static_cast<unsigned>(tiles);
    if (a.w != nullptr)
        hipLaunchKernelGGL((fused_kernel<true, kQ, kKind, kNT, kB>), dim3(grid), dim3(kB), 0, s, a);
    else
        hipLaunchKernelGGL((fused_kernel<false, kQ, kKind, kNT, kB>), dim3(grid), dim3(kB), 0, s, a);
    return static_cast<int>(hipGetLastError());
}

// Blocks of 1024 threads (16 wavefronts) only with one quad per lane, the
// measured best; every other shape uses kBlock.
template <int kKind, bool kNT>
static int launch_fused_nt(const FusedArgs& a, hipStream_t s) {
    switch (a.quads_per_thread) {
        case 4: return launch_fused_q<4, kKind, kNT, kBlock>(a, s);
        case 2: return launch_fused_q<2, kKind, kNT, kBlock>(a, s);
        default:
            return a.block == kFusedWideBlock ? launch_fused_q<1, kKind, kNT, kFusedWideBlock>(a, s)
                                              : launch_fused_q<1, kKind, kNT, kBlock>(a, s);
    }
}

template <int kKind>
static int launch_fused_kind(const FusedArgs& a, hipStream_t s) {
    return a.nt ? launch_fused_nt<kKind, true>(a, s) : launch_fused_nt<kKind, false>(a, s);
}

int launch_fused(const FusedArgs& a, void* stream) {
    hipStream_t s = static_cast<hipStream_t>(stream);
    return a.grad_kind == kGradFP16 ? launch_fused_kind<kGradFP16>(a, s) : launch_fused_kind<kGradBF16>(a, s);
}

}  // namespace gockpt
