// gockpt_internal.h -- layouts shared by the runtime and the kernels.
#pragma once

#include <stdint.h>
#include <stddef.h>

#include "../../include/gockpt.h"
#include "gockpt_contract.h"

namespace gockpt {

constexpr int kBlock = 256;             // threads per block, 4 wavefronts
constexpr int kFusedWideBlock = 1024;   // the fused kernel's optional wide block, 16 wavefronts
constexpr int kVec = 8;                 // elements per thread per group
constexpr int kPrepassMaxBlocks = 2048; // partial sums slots
constexpr int kFinalizeThreads = 256;
constexpr int kScanSlots = 8192;        // partials of the bucket scans of one step
constexpr int kScanMaxBlocks = 256;     // blocks of a bucket scan beside the backward (one per compute unit)

// Device-resident loss-scaler state (workspace offset 0).
struct alignas(64) DevScaler {
    int64_t t;
    int64_t tracker;
    float scale;
    int32_t pad0;
    int64_t pad1[5];
};
static_assert(sizeof(DevScaler) == 64, "DevScaler");

// Per-block partial of the prepass.
struct alignas(16) Partial {
    double sumsq;
    int32_t nonfinite;
    int32_t pad;
};
static_assert(sizeof(Partial) == 16, "Partial");

static_assert(sizeof(gockpt_step_record) == 64, "record size");

// Workspace layout: [DevScaler | pad to 256][records: (MAX_K+1) x 64]
// [prepass partials][bucket-scan partials: two banks, alternating by step,
// so the scans of the next step never overwrite what this step's finalize
// still has to read]
constexpr size_t kWsScalerOff = 0;
constexpr size_t kWsRecordsOff = 256;
constexpr size_t kWsPartialsOff = kWsRecordsOff + (GOCKPT_MAX_K + 1) * sizeof(gockpt_step_record);
constexpr size_t kWsScanOff = kWsPartialsOff + kPrepassMaxBlocks * sizeof(Partial);
constexpr size_t kWsBytes = kWsScanOff + 2 * kScanSlots * sizeof(Partial);

// Page-locked, host-coherent control page of a context (4 KiB).  The device
// writes each window step's skip decision there (finalize), and gate kernels
// on the copy stream read how many staged copies the host has moved out of
// their staging slots.
struct alignas(64) CtrlPage {
    uint64_t released;      // staged copies whose slot is free again, in copy order (host writes)
    uint64_t pad0[7];
    uint32_t gate_timeout;  // a gate kernel gave up waiting (device writes 1)
    uint32_t pad1[15];
    int32_t skip[GOCKPT_MAX_K + 1];  // finalize: skip decision of window step s (device writes)
};
static_assert(sizeof(CtrlPage) <= 4096, "control page");

// Loss-scaler settings the finalize needs.
struct ScalerCfg {
    int32_t check_overflow;
    int32_t dynamic_scale;
    float growth_factor;
    float backoff_factor;
    float min_scale;
    int32_t pad;
    int64_t growth_interval;
};

// Which elements one step packs into the ring, and where.  The step's pack
// list is [grads of elements 0..gb) | master, exp_avg, exp_avg_sq of the
// chunk [cb, ce)].  A prefix of that list goes to the ring; the rest is copied
// straight from the live buffers.  Elements [0, g_end) of the gradients and
// [cb, s_end[k]) of state array k go to the ring, at ring byte offsets
// (physical, < ring_bytes) off_g + 2*i and off_s[k] + 4*(i - cb), taken
// modulo ring_bytes.
struct PackPlan {
    int64_t g_end;
    int64_t cb;
    int64_t s_end[3];
    uint64_t off_g;
    uint64_t off_s[3];
    uint8_t* ring;
    uint64_t ring_bytes;
    int32_t ring_nt;      // 1: nontemporal ring stores
    int32_t pad;
};

struct FusedArgs {
    float* p;
    float* m;
    float* v;
    uint16_t* w;
    const uint16_t* g;
    int64_t n;
    const gockpt_step_record* rec;  // this step's record (skip, scalars)
    float b1, b2, omb1, omb2, eps;  // step-independent scalars
    int32_t quads_per_thread;       // 1, 2 or 4 quads (4 elements) per thread
    int32_t grad_kind;              // kGradBF16 or kGradFP16
    int32_t nt;                     // nontemporal state loads and stores
    int32_t block;                  // threads per block: kBlock or kFusedWideBlock (one quad per lane)
    PackPlan pack;
};

// Launch-shape choices of a context (fixed at create).
struct Knobs {
    int quads_per_thread;  // fused kernel: quads of 4 elements per thread
    int ring_nt;      // nontemporal ring stores
    int prepass_nt;   // nontemporal gradient loads in the prepass
    int fused_nt;     // nontemporal loads and stores of the state in the fused kernel
    int fused_block;  // fused kernel threads per block: kBlock (default) or kFusedWideBlock
};

// What the finalize of one step needs besides the partials.
struct FinalizeArgs {
    int32_t raw;        // partials hold squares of the scaled gradients (bucket scans)
    int32_t norm_off;
    const float* found_inf;
    int32_t slot;       // record slot (window step s, 0 outside a window)
    int32_t window_step;
    float lr;
    int32_t pad;
    HParams hp;
    ScalerCfg sc;
    int32_t* skip_out;  // host-coherent slot for this step's skip decision, or null
};

// Launchers (gockpt_kernels.hip).  All stream-ordered, no host sync.
int launch_prepass(const uint16_t* g, int64_t n, void* workspace, int nblocks, int nt, int grad_kind, void* stream);
// parts: the partials to reduce (nparts of them, in order); raw: they hold
// squares of the scaled gradients (bucket scans), which the finalize unscales.
int launch_finalize(void* workspace, const void* parts, int nparts, const FinalizeArgs& fin, void* stream);
// One wavefront on `stream` that waits until *released >= target (host-
// coherent memory the host advances), at most max_ticks of the 100 MHz
// constant clock; on giving up it sets *timed_out.
int launch_gate(const uint64_t* released, uint64_t target, uint64_t max_ticks, uint32_t* timed_out, void* stream);
int launch_scan(const uint16_t* g, int64_t begin, int64_t end, void* parts, int nblocks, int nt, int grad_kind,
                void* stream);
int scan_blocks_for(int64_t count, int max_blocks);
int launch_fused(const FusedArgs& a, void* stream);
int prepass_blocks_for(int64_t n);
Knobs default_knobs();

}  // namespace gockpt
