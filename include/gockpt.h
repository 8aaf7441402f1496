/*
 * gockpt.h -- C ABI of the MI355X GoCkpt hot path.
 *
 * GoCkpt (arXiv 2511.07035) saves a checkpoint of the model and optimizer
 * state across K training steps instead of one: the state is split into K
 * parts, one part is sent to host memory per step, and at every step the
 * 16-bit gradients of the parts already sent are sent as well (Sec. 4.2.1,
 * Fig. transfer_update).  After the window the host replays AdamW on each
 * stale part with the saved gradients, which yields the checkpoint a blocking
 * snapshot after the last step would hold (Sec. 4.3.1, Fig. update_backend).
 * The paper's framework hooks are save_checkpoint, backward_begin and
 * update_begin (Sec. 4.6); here they are gockpt_begin_window,
 * gockpt_backward_begin and gockpt_step.
 *
 * On the device, one kernel per step applies the mixed-precision AdamW update
 * (fp32 master weights and moments, bf16 working weights, bf16 or fp16
 * gradients; Sec. 2.2) and, in the same pass over HBM, writes the step's part
 * of the state and the gradients of the parts already sent into a device
 * staging ring.  A copy stream drains the ring into host memory while the
 * next step computes (the overlap of Sec. 4.2.4); what does not fit the ring
 * is copied straight from the live buffers.  A small prepass before it finds
 * non-finite gradients (loss-scale skip) and the gradient norm; a context
 * that wants neither (check_overflow = 0, grad_norm_off = 1) runs none.
 *
 * Around that path: wait policies that reproduce the paper's comparison
 * schemes (Sec. 4.2.3-4.2.4), an event model of a window and a planner for K
 * and the part bounds (Sec. 4.2.3), in-window replay and staging into
 * pageable host memory for windows larger than the host can pin, and
 * persistence and loading of the restored checkpoint (Sec. 4.4.3, 4.3.2).
 *
 * Arithmetic contract (both the device update and the host replay follow it,
 * so the restored checkpoint is bit-identical to the device state):
 *   per step, with t the Adam step count after the step and lr the step's
 *   learning rate (fp32):
 *     bc1 = 1 - beta1^t, bc2 = 1 - beta2^t   (fp64, beta^t by binary
 *                                            exponentiation, high bit first)
 *     step_size = (float)(lr / bc1)          (fp64 division, rounded)
 *     sqrt_bc2  = sqrtf((float)bc2)
 *     decay     = (float)(1 - lr * weight_decay)        (fp64)
 *     b1 = (float)beta1, omb1 = (float)(1 - beta1)      (fp64, rounded)
 *     b2 = (float)beta2, omb2 = (float)(1 - beta2), e = (float)eps
 *     inv_scale = 1.0f / scale_used
 *   per element, every line one fp32 operation rounded to nearest even, no
 *   fused multiply-add, subnormals kept:
 *     g = float(grad_bits) * inv_scale        (bf16 or fp16 widened exactly)
 *     m = b1*m + omb1*g ;  v = b2*v + omb2*(g*g) ;  p = p*decay
 *     p = p - step_size * (m / (sqrtf(v)/sqrt_bc2 + e))
 *     w = bf16_round_nearest_even(p)  (every NaN -> 0x7FC0)
 *   A step whose gradients hold an inf/NaN is skipped when check_overflow is
 *   set: state unchanged, t unchanged; with dynamic scaling the scale backs
 *   off (max(scale*backoff, min_scale)), else every growth_interval applied
 *   steps it grows by growth_factor.
 *
 * Conventions
 *   - Every function returns an int status: GOCKPT_OK (0), GOCKPT_EAGAIN (1)
 *     or a negative error.  gockpt_last_error(ctx) gives a message for the
 *     last failing call on that context.  No C++ exception crosses this ABI.
 *   - "device" pointers are HIP device memory of the current device;
 *     "host" pointers are ordinary host memory; "pinned" means page-locked
 *     host memory (hipHostMalloc or torch pin_memory=True).
 *   - The caller owns every buffer it passes (state, gradients, ring,
 *     workspace, host arena, restore outputs) and keeps it alive until
 *     gockpt_destroy, or until the gockpt_restore (gockpt_restore_wait) that
 *     consumes it returns.
 *     The context owns its HIP events, its host bookkeeping and one 4 KiB
 *     page-locked control page (the device writes each window step's skip
 *     decision there, and the copy stream reads the staging-slot counter).
 *   - One host thread drives a context.  gockpt_restore uses its own worker
 *     threads internally.
 *   - Streams are hipStream_t passed as void*.  NULL means the null stream.
 *
 * State machine:  IDLE --begin_window--> WINDOW (steps 1..K) --K-th step-->
 *   DRAINING --drain--> DRAINED --restore--> IDLE (or --restore_async-->
 *   RESTORING --restore_wait--> IDLE).  gockpt_abort_window goes
 *   back to IDLE from any window state and discards the window.  A HIP error
 *   during a window marks it FAILED: drain and restore refuse it
 *   (GOCKPT_EFAILED); abort clears it.  Plain steps (no packing) are allowed
 *   in IDLE, DRAINING, DRAINED and RESTORING.
 */
#ifndef GOCKPT_H
#define GOCKPT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define GOCKPT_OK 0
#define GOCKPT_EAGAIN 1     /* non-blocking drain: copies still in flight */
#define GOCKPT_EINVAL (-1)  /* bad argument (sizes, alignment, bounds) */
#define GOCKPT_ESTATE (-2)  /* call made in the wrong state */
#define GOCKPT_EBUSY (-3)   /* a previous window is not restored/aborted */
#define GOCKPT_ENOMEM (-4)  /* a caller buffer is too small */
#define GOCKPT_EHIP (-5)    /* HIP runtime error (message has the HIP text) */
#define GOCKPT_EFAILED (-6) /* window poisoned by an earlier error */

#define GOCKPT_MAX_K 256           /* longest save window */
#define GOCKPT_ALIGN_ELEMS 8       /* chunk bounds are multiples of this */
#define GOCKPT_DEFAULT_COPY_BYTES ((size_t)64 << 20)

typedef struct gockpt_ctx gockpt_ctx;

/* Everything a context is created with. */
typedef struct {
    int64_t n;               /* elements in the flat parameter space, >= 0 */
    float* master;           /* device fp32[n], master weights (in place) */
    float* exp_avg;          /* device fp32[n], AdamW first moment */
    float* exp_avg_sq;       /* device fp32[n], AdamW second moment */
    uint16_t* weight_bf16;   /* device bf16[n] working weights, or NULL */
    const uint16_t* grad16;  /* device [n] 16-bit gradients (bf16 or fp16,
                                per grad_dtype), multiplied by the current
                                loss scale */
    double beta1, beta2, eps, weight_decay;
    int32_t check_overflow;  /* 1: skip steps with inf/NaN gradients */
    int32_t dynamic_scale;   /* 1: dynamic loss scaling (see contract) */
    float init_scale;        /* loss scale of the first step (>0) */
    float growth_factor, backoff_factor, min_scale;
    int64_t growth_interval; /* >= 1 */
    int64_t init_step;       /* Adam step count already taken (resume), >= 0 */
    int64_t init_tracker;    /* growth tracker at create (resume), >= 0 */
    void* ring;              /* device staging ring, 256-byte aligned, or NULL */
    size_t ring_bytes;       /* multiple of 256 (0 if ring is NULL) */
    size_t copy_bytes;       /* largest single D2H copy; 0 = default 64 MiB;
                                multiple of 256 */
    void* workspace;         /* device, gockpt_workspace_bytes(n) bytes */
    size_t workspace_bytes;
    void* compute_stream;    /* hipStream_t the update runs on */
    void* copy_stream;       /* hipStream_t the D2H copies run on; must not
                                be the compute stream */
    int32_t timing;          /* 1: time copies and kernels with HIP events
                                (fills the timing fields of the stats) */
    int32_t copy_threads;    /* staged windows: host threads moving landed
                                staging slots into the pageable arena
                                (<= 0: 8) */
    void* host_staging;      /* pinned host memory (gockpt_host_alloc) used to
                                stage copies into a pageable host arena, or
                                NULL; sliced into copy_bytes slots (>= 2) */
    size_t host_staging_bytes;
    int32_t grad_dtype;      /* GOCKPT_GRAD_BF16 (0) or GOCKPT_GRAD_FP16 (1):
                                the training run's gradient format (Sec. 2.2:
                                FP16 or BF16).  fp16 gradients are widened
                                exactly; their inf/NaN test is the fp16
                                exponent field.  Packed and sent as raw bits
                                either way. */
    int32_t grad_norm_off;   /* 0: every step computes the sum of squares of
                                its unscaled gradients (the records' gnorm2);
                                1: it does not (gnorm2 = -1).  With
                                check_overflow = 0 as well, nothing needs the
                                gradients before the update, and the step
                                skips the prepass, its 2 bytes per element of
                                reading. */
    const float* found_inf;  /* device, nullable.  With check_overflow = 1:
                                the caller has already tested the gradients
                                (a gradient scaler's found-inf flag, written
                                on the compute stream before gockpt_step),
                                and a step is skipped exactly when
                                *found_inf != 0 (a NaN flag counts as set);
                                the prepass then does not scan for inf/NaN,
                                and with grad_norm_off = 1 it does not run.
                                Ignored with check_overflow = 0. */
} gockpt_config;

#define GOCKPT_GRAD_BF16 0
#define GOCKPT_GRAD_FP16 1

/* Options of one save window (gockpt_begin_window_ex). */
typedef struct {
    int32_t replay_every;    /* R.  0 (default) or >= K: the gradients of all K
                                steps are kept and replayed by gockpt_restore.
                                1 <= R < K: during the window, after every R
                                steps have landed, a library thread replays
                                them onto the parts already received, so the
                                arena keeps R steps of gradients instead of K
                                (host memory 12 n + 2 R bounds[K-1] bytes);
                                the copies of a step wait for the replay of
                                the batch whose gradient slots they reuse */
    int32_t replay_threads;  /* threads of that in-window replay (<= 0: 8) */
    int32_t wait_policy;     /* when the compute stream waits for the window's
                                copies (GOCKPT_WAIT_*; other than LAZY needs a
                                pinned arena) */
    int32_t ring_off;        /* 1: this window leaves the staging ring unused
                                and copies everything straight from the live
                                buffers */
    int32_t late_plan;       /* ring plan: how much of the staging ring a
                                window step may fill (GOCKPT_RING_*; 0 =
                                GOCKPT_RING_QUERY) */
    int32_t no_timing;       /* 1: this window records no timing events even
                                when the context has timing on (its step
                                times are then not available) */
    int32_t defer_copies;    /* 1: a window step's copies are queued on the
                                copy stream at the next call into the
                                library (gockpt_backward_begin, gockpt_step
                                or gockpt_drain) instead of by gockpt_step
                                itself.  Copies queued before the device
                                reaches the update wait for it on the copy
                                engine, and that wait slows the dispatch of
                                short kernels on the compute stream: a loop
                                that launches many short kernels and runs
                                less than a step ahead of the device loses
                                less time this way.  Needs GOCKPT_WAIT_LAZY.
                                A step's copies then start no earlier than
                                that next call, the gradients taken straight
                                from the gradient buffer included */
    int32_t reserved_[1];    /* must be 0 */
} gockpt_window_opts;

/* Wait policies (gockpt_window_opts.wait_policy).  They change only when the
 * compute stream may go on, never what reaches the host.
 *   LAZY  (default): data copied straight from a live buffer is waited for
 *         just before that buffer is overwritten -- state before the next
 *         update, gradients before the next backward (gockpt_backward_begin).
 *         The gradient transfer hides behind the next forward pass: the
 *         paper's GoCkpt-O (Sec. 4.2.4).
 *   GRADS: at the end of every window step the compute stream waits until that
 *         step's gradients are on the host: the explicit gradient wait of the
 *         paper's GoCkpt, whose only visible cost is the gradient transfer
 *         (Sec. 4.2.3).
 *   ALL:  at the end of every window step the compute stream waits for all of
 *         the step's copies.  With K = 1 and the ring off this is a blocking
 *         snapshot of the whole state (the Async baseline of Sec. 4.2.3 and
 *         Sec. 5.2); K = 1 with LAZY is Async-O (the copy overlaps one
 *         step). */
#define GOCKPT_WAIT_LAZY 0
#define GOCKPT_WAIT_GRADS 1
#define GOCKPT_WAIT_ALL 2

/* Ring plans (gockpt_window_opts.late_plan).  Each window step packs as much
 * of its pack list (the gradients of the parts already sent, then its own
 * part's master, m, v; Sec. 4.2.1) into the staging ring as the plan allows;
 * the rest is copied straight from the live buffers.  The checkpoint is the
 * same bytes under every plan.
 *   QUERY       (default) the ring space whose earlier copies have finished
 *               when the host calls gockpt_step.  Never blocks, but a host
 *               that runs steps ahead of the device sees little space freed.
 *   HOST_WAIT   the same decision taken once the device reaches the update:
 *               gockpt_step blocks the calling thread until the compute
 *               stream has finished the step's finalize.  The step's skip
 *               decision is then known too, and a skipped step sends no
 *               gradients.
 *   DEVICE_WAIT the whole ring, as if every earlier copy had finished by the
 *               update; the compute stream waits (on the device) for the
 *               copies of the ring ranges the step overwrites.  Never blocks
 *               the calling thread (the transfers stay off the training
 *               thread, Sec. 4.4.1); costs device time only when the link
 *               has not kept up with the earlier steps' copies. */
#define GOCKPT_RING_QUERY 0
#define GOCKPT_RING_HOST_WAIT 1
#define GOCKPT_RING_DEVICE_WAIT 2

/* One per step, written by the device, copied into the host arena.  64 B. */
typedef struct {
    int64_t t;            /* Adam step count after the step */
    int64_t tracker;      /* growth tracker after the step */
    float scale_used;     /* loss scale the step's gradients carried */
    float scale_next;     /* loss scale after the step */
    float lr;             /* learning rate of the step */
    int32_t skip;         /* 1: step skipped (inf/NaN gradient) */
    int32_t nonfinite;    /* 1: some gradient was inf/NaN, or the found_inf
                             flag was set when one is given; 0 when nothing
                             looked (check_overflow = 0, grad_norm_off = 1) */
    int32_t window_step;  /* s in 1..K inside a window, 0 otherwise */
    double gnorm2;        /* sum of squares of the unscaled gradients; -1
                             with grad_norm_off */
    float step_size;      /* scalars the device used (see the contract) */
    float sqrt_bc2;
    float decay;
    float inv_scale;
} gockpt_step_record;

/* Counters of the last window (bytes and, with timing on, milliseconds). */
typedef struct {
    int32_t K;
    int32_t steps_done;
    int32_t skipped;
    int32_t n_gates;          /* staged windows: gate kernels queued on the copy
                                 stream (a copy reusing a staging slot waits
                                 there until the host has emptied it) */
    uint64_t bytes_ring;      /* bytes planned into the ring (a skipped step
                                 packs none of its gradients) */
    uint64_t bytes_spilled;   /* bytes copied straight from live buffers */
    uint64_t bytes_d2h;       /* all bytes copied to the host arena */
    uint64_t n_copies;        /* hipMemcpyAsync calls */
    double copy_ms;           /* sum over steps of copy-stream busy time */
    double prepass_ms;        /* sum over steps of the time before the update:
                                 prepass (or the wait for the bucket scans)
                                 and finalize */
    double update_ms;         /* sum of fused update+pack kernel times */
    double wait_ms;           /* host time blocked in gockpt_drain */
    uint64_t bytes_host_copied;  /* staged windows: bytes the worker threads
                                    moved from staging slots into the arena */
    double host_copy_ms;      /* sum over worker threads of the time spent in
                                 those copies (workers run in parallel: the
                                 aggregate rate is up to copy_threads times
                                 bytes_host_copied / host_copy_ms) */
    double replay_ms;         /* in-window replay: time the replayer spent
                                 applying batches (0 without it) */
} gockpt_window_stats;

/* The restored checkpoint's scalar state. */
typedef struct {
    int64_t t;            /* Adam step count of the checkpoint */
    int64_t tracker;      /* growth tracker of the checkpoint */
    float scale;          /* loss scale of the checkpoint */
    int32_t K;            /* window length the checkpoint came from */
    int32_t skipped;      /* skipped steps inside the window */
    int32_t reserved_;
    double restore_ms;    /* host wall time of the replay */
    int64_t element_updates; /* AdamW element updates replayed */
} gockpt_ckpt_meta;

/* Byte offsets of the pieces of a window's host arena (pinned). */
typedef struct {
    uint64_t records;      /* gockpt_step_record[K] */
    uint64_t master;       /* fp32[n]: part j lands at [bounds[j-1], bounds[j]) */
    uint64_t exp_avg;      /* fp32[n] */
    uint64_t exp_avg_sq;   /* fp32[n] */
    uint64_t grads;        /* start of the gradient blocks */
    uint64_t total;        /* arena size in bytes */
} gockpt_arena_layout;

/* ---- sizes and planning (host only, no device calls) -------------------- */

/* Device workspace bytes a context over n elements needs. */
size_t gockpt_workspace_bytes(int64_t n);

/* Host arena layout for a K-step window with chunk bounds bounds[0..K] and
 * in-window replay every replay_every steps (0 = keep all gradients; see
 * gockpt_window_opts).  grad_offsets as in gockpt_arena_layout_for. */
int gockpt_arena_layout_ex(int K, const int64_t* bounds, int64_t n, int replay_every,
                           gockpt_arena_layout* out, uint64_t* grad_offsets);

/* Host arena layout for a K-step window with chunk bounds bounds[0..K].
 * grad_offsets (nullable, K entries): byte offset of step s's gradient block
 * (bf16 gradients of elements [0, bounds[s-1]), s = 1..K; step 1's is empty).
 * Returns GOCKPT_EINVAL for bad K or bounds. */
int gockpt_arena_layout_for(int K, const int64_t* bounds, int64_t n,
                            gockpt_arena_layout* out, uint64_t* grad_offsets);

/* Split [0, n) into K parts, one per window step (Sec. 4.2.1; Sec. 4.2.2
 * organises the state into blocks).  Every state
 * byte per element costs the same, so a byte-balanced split is an element-
 * balanced one.  tensor_ends (nullable, n_tensors entries, increasing, last
 * == n) restricts interior bounds to tensor boundaries: each bound is the
 * tensor boundary nearest to j*n/K that keeps the bounds strictly increasing.
 * Otherwise bounds are j*n/K rounded down to a multiple of `align` elements
 * (align: a multiple of 8).  Boundaries that are not multiples of 8 are
 * rejected (GOCKPT_EINVAL).  bounds_out holds K+1 entries. */
int gockpt_plan_bounds(int K, int64_t n, const int64_t* tensor_ends, int n_tensors,
                       int64_t align, int64_t* bounds_out);

/* ---- pinned host memory for the arena ------------------------------------ */

/* Page-locked host allocation of `bytes` (hipHostMalloc, portable, 4 KiB
 * aligned) for a window's host arena; the D2H copies need page-locked
 * destinations to run asynchronously on the copy engines (Sec. 4.4.2 pins the
 * host buffers for the same reason).  The memory is zeroed with several
 * threads before returning, so its CPU pages are mapped up front.  *out is
 * NULL on failure (GOCKPT_EHIP).  Free with gockpt_host_free. */
int gockpt_host_alloc(size_t bytes, void** out);
int gockpt_host_free(void* p);

/* ---- context ------------------------------------------------------------ */

/* Validate cfg, create events, upload the scaler state into the workspace.
 * Synchronous.  Errors: EINVAL (null/unaligned pointers: every device buffer
 * 16-byte aligned; ring and workspace 256-byte aligned), ENOMEM (workspace too
 * small), EHIP. *out is NULL on failure. */
int gockpt_create(const gockpt_config* cfg, gockpt_ctx** out);

/* gockpt_create for callers that cannot allocate memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * context's device workspace is the library's own static scratch array
 * (gockpt_workspace_bytes(n) = 304.5 KiB whatever n is; one per GPU,
 * kept until the process ends) instead of cfg->workspace, and no control page
 * is allocated.  It calls no hipMalloc, hipFree or hipHostMalloc; it creates
 * the context's HIP events and host bookkeeping like gockpt_create.
 * cfg->workspace must be NULL and cfg->workspace_bytes 0; cfg->host_staging
 * must be NULL (staged windows need the control page), and skipped steps'
 * gradients are always sent (the skip decision has no host-visible slot).
 * Otherwise the context behaves as one from gockpt_create, bit for bit.
 * Every context made this way on one GPU would share that GPU's array, and
 * the array keeps what the last context left there (the loss-scaler state is
 * cleared at create): only one may live per device at a time -- a second one
 * gets GOCKPT_EBUSY until the first is destroyed.  Errors: EINVAL (config,
 * workspace or staging given), ENOMEM (a workspace larger than the static
 * array), EBUSY, EHIP. */
int gockpt_create_noalloc(const gockpt_config* cfg, gockpt_ctx** out);

/* Wait for all work of the context, release its events.  Accepts NULL. */
int gockpt_destroy(gockpt_ctx* ctx);

/* Message for the last failing call on ctx.  With ctx NULL: the calling
 * thread's last failing call that takes no context (gockpt_create, host
 * memory, checkpoint files, replay of an arena).  Valid until the next such
 * call. */
const char* gockpt_last_error(const gockpt_ctx* ctx);

/* ---- window planner (Sec. 4.2.3) --------------------------------------------
 * An event model of a window on the compute and copy streams, following the
 * library's own rules: per step, forward (t_fwd_ms) -> the lazy gradient wait
 * -> backward (t_bwd_ms) -> the lazy state wait -> the update (t_upd_ms plus
 * the pack stores at pack_gbs) -> the wait of the chosen policy.  The copy
 * stream moves, at link_gbs in copy_bytes pieces, the step's gradients that
 * did not fit the ring from when the update starts, then after the update
 * the ring's gradients and state and the rest of the state.  Ring use
 * follows ring_plan: QUERY and HOST_WAIT take the ring space whose copies
 * have finished when the update starts (HOST_WAIT's rule exactly; QUERY
 * decides earlier, on the host, so it may find less); DEVICE_WAIT takes the
 * whole ring and the update waits for the copies of the bytes it
 * overwrites.  Ring space is freed per segment (one pack segment's copies
 * finish together), as the library does; a part's state counts as one
 * segment.  With staging_bytes > 0 (a pageable
 * arena) every copy lands in one of staging_bytes / copy_bytes slots in
 * turn, starts only once the host has emptied the slot's previous copy, and
 * the host empties slots in copy order at host_gbs.  The predicted stall
 * is the compute-stream time of the window's K steps and the step after it
 * minus K + 1 plain steps; the in-window replay is not modelled.
 * With 14 B of state and 2 B of gradient per element, no ring and one part's
 * transfer lasting one step, it reproduces Sec. 4.2.3's (N-1) T_step for
 * Async-O and N(N-1)/14 T_step for GoCkpt. */
typedef struct {
    int64_t n;                  /* elements */
    const int64_t* tensor_ends; /* nullable: bounds restricted to these ends
                                   (increasing, last == n) */
    int32_t n_tensors;
    int32_t wait_policy;        /* GOCKPT_WAIT_* of the window */
    int64_t align;              /* bound alignment without tensor_ends
                                   (multiple of 8; <= 0: 256) */
    double t_fwd_ms;            /* end of an update -> gockpt_backward_begin */
    double t_bwd_ms;            /* gockpt_backward_begin -> start of the update
                                   (backward, gradient writes, prepass) */
    double t_upd_ms;            /* the update without the pack */
    double pack_gbs;            /* rate of the pack stores (<= 0: free) */
    double link_gbs;            /* device -> host rate (> 0) */
    uint64_t ring_bytes;        /* staging ring (0: none; multiple of 256) */
    uint64_t copy_bytes;        /* copy piece (0: GOCKPT_DEFAULT_COPY_BYTES) */
    double state_bytes;         /* bytes sent per element of a part (<= 0: 12) */
    double grad_bytes;          /* bytes sent per gradient (<= 0: 2) */
    int32_t max_K;              /* planner: longest window tried (<= 0: 7, the
                                   cap of Sec. 4.2.3) */
    int32_t ring_plan;          /* GOCKPT_RING_* of the window (see above) */
    uint64_t staging_bytes;     /* pinned staging of a pageable arena (0: the
                                   arena is pinned; else >= copy_bytes) */
    double host_gbs;            /* staged: rate at which the library threads
                                   together move landed copies into the arena
                                   (<= 0: at once) */
} gockpt_plan_params;

typedef struct {
    int32_t K;
    int32_t reserved_;
    double stall_ms;      /* predicted checkpoint stall (see above) */
    double latency_ms;    /* window start -> last copy on the host */
    double d2h_bytes;     /* bytes copied to the host */
    double spilled_bytes; /* of which copied straight from the live buffers */
} gockpt_plan_result;

/* Predicted stall of a K-step window with the given bounds (rules as
 * gockpt_begin_window).  step_stall_ms (nullable, K+1 entries): each step's
 * delay over a plain step, the last entry being the step after the window.
 * Host only.  Errors: EINVAL (parameters or bounds). */
int gockpt_simulate_window(const gockpt_plan_params* params, int K, const int64_t* bounds,
                           gockpt_plan_result* out, double* step_stall_ms);

/* Choose K (1..max_K) and the bounds that minimise the predicted stall; ties
 * go to fewer bytes copied, then an earlier last copy, then a shorter window.
 * Candidates per K: equal parts, and parts that keep every step's copy volume
 * equal (part s holds n q^(s-1)(1-q)/(1-q^K) elements, q = 1 - grad/state
 * bytes, so the growing gradient share is offset by shrinking parts), each
 * refined by moving one bound at a time.  bounds_out holds max_K + 1
 * entries.  Host only.  Errors: EINVAL. */
int gockpt_plan_window(const gockpt_plan_params* params, int64_t* bounds_out, gockpt_plan_result* out);

/* ---- the hot path -------------------------------------------------------- */

/* Open a K-step save window (save_checkpoint hook, Sec. 4.6).  bounds:
 * K+1 host int64, bounds[0] = 0, bounds[K] = n, strictly increasing, interior
 * bounds multiples of 8.  host_arena: at least gockpt_arena_layout_for(...)
 * .total bytes, 256-byte aligned.  A pinned arena receives the D2H copies
 * directly.  A pageable arena (larger than the host can pin) needs
 * cfg.host_staging: copies then land in the pinned staging slots and library
 * threads move them into the arena.  No device work.  Errors: EINVAL (bounds,
 * alignment, pageable arena without staging), ENOMEM (arena too small),
 * EBUSY (a window not restored or aborted), EFAILED. */
int gockpt_begin_window(gockpt_ctx* ctx, int K, const int64_t* bounds,
                        void* host_arena, size_t arena_bytes);

/* gockpt_begin_window with options (opts may be NULL).  The arena must be at
 * least gockpt_arena_layout_ex(K, bounds, n, opts->replay_every).total. */
int gockpt_begin_window_ex(gockpt_ctx* ctx, int K, const int64_t* bounds,
                           void* host_arena, size_t arena_bytes,
                           const gockpt_window_opts* opts);

/* Call before the backward pass writes the gradient buffer (backward_begin
 * hook, Sec. 4.6).  If the previous step had to copy gradients straight from
 * the gradient buffer (ring full), `stream` (NULL: the compute stream) waits
 * for those copies.  Cheap no-op otherwise, and always after gockpt_drain
 * (every copy of the window has finished by then).  In a window with
 * defer_copies it first queues the previous step's copies. */
int gockpt_backward_begin(gockpt_ctx* ctx, void* stream);

/* The overflow test and norm of the coming step over one bucket of
 * gradients, [begin, end), queued on `stream` (NULL: the compute stream) as
 * soon as the backward has written that bucket -- so the test overlaps the
 * rest of the backward instead of running before the update, where it would
 * read all 2n bytes of gradients on the step's critical path.  The stream
 * must be ordered after the writes of the bucket.  When the scans of a step
 * cover [0, n) exactly (any order, no overlap), gockpt_step runs no prepass:
 * it waits for the scans and reduces their partials in call order (the skip
 * decision does not depend on the order; the norm, telemetry, sums in fp64).
 * begin and end are multiples of 8 (end may be n).  Errors: EINVAL (range),
 * ESTATE (overlap with an earlier scan of the step, or more than 8192 scan
 * blocks in one step), EHIP. */
int gockpt_scan_grads(gockpt_ctx* ctx, int64_t begin, int64_t end, void* stream);

/* One optimizer step (update_begin hook, Sec. 4.6), stream-ordered on the
 * compute stream.  Reads the gradient buffer as it stands in stream order.
 * Inside a window, window step s packs part s of the updated state and the
 * gradients of parts 1..s-1 and queues their copies to the host arena on the
 * copy stream; after the K-th step the window is DRAINING.  Outside a window
 * it is the plain fused update: three kernels on the compute stream and no
 * host-side decision, so it may be captured in a HIP graph (stream capture
 * of the compute stream) and replayed; lr is fixed at capture, while the step
 * count and the loss scale live on the device and advance with every replay.
 * Window steps cannot be captured (their copies are planned on the host).
 * Step records are read after the drain
 * (gockpt_window_records).  The calling thread does not wait for the device,
 * except: with the HOST_WAIT ring plan (until the device has finished the
 * step's finalize); with in-window replay into a pinned arena (until the
 * replay of the batch whose gradient slots this step reuses).  In staged
 * windows every copy is queued here; a copy that reuses a staging slot waits
 * on the device (a gate kernel on the copy stream) until a library thread
 * has emptied the slot.  With defer_copies the step's copies are queued by
 * the next call into the library (this function queues the previous step's
 * first).
 * Errors: EINVAL (lr not finite), ESTATE (bucket scans made for this step
 * that do not cover [0, n); or the previous window step copies
 * gradients straight from the gradient buffer and gockpt_backward_begin was
 * not called since; not after the window is drained), EHIP (window becomes
 * FAILED). */
int gockpt_step(gockpt_ctx* ctx, float lr);

/* Completion of the window's GPU-to-CPU transfer, which must be on the host
 * before the CPU update of the parts (Sec. 4.3.1) and before persistence
 * (Sec. 4.4.1, Sec. 4.4.3; the commit waits for the previous checkpoint,
 * Sec. 4.2.3).  Waits for the window's copies -- staged ones moved into the
 * arena, and with in-window replay the replay of the last batch -- (blocking
 * = 1) or polls them (blocking = 0, returns GOCKPT_EAGAIN while in flight);
 * a deferring window's last copies are queued first.
 * On success the window is DRAINED and stats (nullable) is filled.  Errors:
 * ESTATE (not DRAINING/DRAINED), EFAILED, EHIP. */
int gockpt_drain(gockpt_ctx* ctx, int blocking, gockpt_window_stats* stats);

/* CPU reconstruction (Sec. 4.3.1): bring every part to the state after the
 * window's last step by replaying the saved gradients with each step's
 * record.  Host only, nthreads worker threads (<= 0: 16).  Outputs are host
 * arrays of n elements; any of master_out/exp_avg_out/exp_avg_sq_out may be
 * NULL to restore that array in place inside the host arena (the arena's
 * master/exp_avg/exp_avg_sq areas then hold the checkpoint).  w_bf16_out
 * (nullable) receives bf16_rne(master).  meta (nullable) receives t, scale,
 * tracker.  Afterwards the context is IDLE.  Errors: ESTATE (not DRAINED),
 * EFAILED, EINVAL. */
int gockpt_restore(gockpt_ctx* ctx, float* master_out, float* exp_avg_out,
                   float* exp_avg_sq_out, uint16_t* w_bf16_out,
                   gockpt_ckpt_meta* meta, int nthreads);

/* gockpt_restore in a library thread, so training goes on while the host
 * replays (the CPU update runs beside the GPU's training, Sec. 4.3.1).
 * Returns at once; the context is RESTORING until gockpt_restore_wait.
 * Meanwhile plain steps may run (they touch neither the arena nor the
 * outputs); gockpt_begin_window, gockpt_persist, gockpt_load,
 * gockpt_abort_window and gockpt_destroy first wait for the restore.  The
 * outputs must stay valid, and unread, until the wait returns.  Errors:
 * ESTATE (not DRAINED), EFAILED. */
int gockpt_restore_async(gockpt_ctx* ctx, float* master_out, float* exp_avg_out,
                         float* exp_avg_sq_out, uint16_t* w_bf16_out, int nthreads);

/* Wait for gockpt_restore_async; meta (nullable) as in gockpt_restore.
 * Afterwards the context is IDLE.  Errors: those of gockpt_restore (the
 * window is then FAILED), ESTATE (no restore running). */
int gockpt_restore_wait(gockpt_ctx* ctx, gockpt_ckpt_meta* meta);

/* Discard the current window (any window state) and return to IDLE after
 * waiting for its copies, including those the library threads still had
 * queued after an error.  Clears FAILED.  When it returns GOCKPT_OK no copy
 * or library thread touches the arena, the staging memory or the live
 * buffers any more: the caller may free the arena, and new gradients may be
 * written without gockpt_backward_begin.  Errors: EHIP (the copy stream
 * reported an error while it was waited for; the context is IDLE anyway). */
int gockpt_abort_window(gockpt_ctx* ctx);

/* ---- inspection ------------------------------------------------------- */

/* Synchronize the compute stream and read the device-resident scaler state. */
int gockpt_get_scaler(gockpt_ctx* ctx, int64_t* t, float* scale, int64_t* tracker);

/* Copy of the drained window's records (K entries) into records_out (host). */
int gockpt_window_records(gockpt_ctx* ctx, gockpt_step_record* records_out, int capacity);

/* Per-step figures of the drained window (needs cfg.timing = 1):
 * out[5*(s-1) + 0] = prepass + finalize ms, [+1] = fused update+pack kernel
 * ms, [+2] = copy-stream ms from the step's first copy to its last, [+3] =
 * bytes the update packed into the ring (the rest of the step's pack was
 * copied straight from the live buffers), [+4] = compute-stream ms between
 * the finalize and the update kernel (with HOST_WAIT the host's round trip;
 * with DEVICE_WAIT any wait for earlier ring copies), for s = 1..K; out
 * holds 5*capacity doubles.  Errors: ESTATE (not drained, or timing off for
 * the context or the window), ENOMEM. */
int gockpt_window_step_times(gockpt_ctx* ctx, double* out, int capacity);

/* Replay a drained host arena without a context (same code as
 * gockpt_restore): for callers that persisted the arena and restore in
 * another process, and for host-only tests.  The arena layout must match
 * gockpt_arena_layout_for(K, bounds, n); grad_dtype as in gockpt_config;
 * outputs as in gockpt_restore (NULL = in place). */
int gockpt_replay_arena(int K, const int64_t* bounds, int64_t n, void* host_arena,
                        size_t arena_bytes, double beta1, double beta2, double eps,
                        double weight_decay, int grad_dtype, float* master_out, float* exp_avg_out,
                        float* exp_avg_sq_out, uint16_t* w_bf16_out,
                        gockpt_ckpt_meta* meta, int nthreads);

/* ---- persistence and loading (Sec. 4.4.3, Sec. 4.3.2) ---------------------
 * A checkpoint is a directory: data.bin (master | exp_avg | exp_avg_sq,
 * fp32[n] each, every array at a 4 KiB-aligned offset), an optional `user`
 * file of caller text, and `meta` (text: scalar state, hyperparameters as
 * exact hexadecimal floats, layout, a CRC-32C per piece of data.bin).  `meta`
 * is written last (to meta.tmp, synced, renamed, directory synced), so a
 * checkpoint is complete exactly when `meta` exists.  A checkpoint is written
 * into a sibling directory (`dir`.gockpt-tmp) and put at `dir` only when
 * complete -- exchanged with the one already there in a single rename -- so
 * `dir` never stops holding a complete checkpoint while a new one is written.
 * `dir` is the checkpoint's own directory.  Pieces are written and read by
 * several threads at their own offsets.  The bf16 weights are not stored: loading
 * re-derives them as bf16_rne(master), bit-identical to what the update
 * writes. */
typedef struct {
    int64_t n;
    int64_t t;              /* Adam step count */
    int64_t tracker;        /* loss-scaler growth tracker */
    float scale;            /* loss scale */
    int32_t K;              /* window the checkpoint came from (0: none) */
    int32_t skipped;        /* skipped steps inside that window */
    int32_t has_user;       /* 1: a user file is present */
    double beta1, beta2, eps, weight_decay;
    uint64_t piece_bytes;   /* write/read/checksum unit (0 on write: 64 MiB;
                               a multiple of 4096) */
    uint64_t data_bytes;    /* size of data.bin (filled on read) */
} gockpt_ckpt_info;

typedef struct {
    double bytes;   /* payload bytes written or read */
    double ms;      /* wall time, sync included */
    int64_t pieces;
} gockpt_io_stats;

/* Write a checkpoint of three host arrays (fp32[info->n] each) into `dir`
 * (created if missing) with nthreads writers (<= 0: 16).  user_meta: NUL-
 * terminated text or NULL.  Host only.  Errors: EINVAL, EFAILED (I/O; the
 * message names the call and errno).  On any error `meta` is absent. */
int gockpt_write_checkpoint(const char* dir, const float* master, const float* exp_avg,
                            const float* exp_avg_sq, const gockpt_ckpt_info* info,
                            const char* user_meta, int nthreads, gockpt_io_stats* stats);

/* Scalar state and layout of a complete checkpoint.  Errors: EFAILED (no
 * `meta`: not a complete checkpoint; malformed). */
int gockpt_read_checkpoint_info(const char* dir, gockpt_ckpt_info* info);

/* Read a complete checkpoint of n elements into three host arrays, checking
 * every piece's CRC-32C.  Errors: EINVAL (n differs), EFAILED (incomplete,
 * short file, checksum mismatch -- the message names the array and byte). */
int gockpt_read_checkpoint(const char* dir, int64_t n, float* master, float* exp_avg,
                           float* exp_avg_sq, gockpt_ckpt_info* info, int nthreads,
                           gockpt_io_stats* stats);

/* The checkpoint's user text: *length gets its size; buf (nullable) gets it
 * NUL-terminated.  Errors: EFAILED, ENOMEM (capacity < length + 1). */
int gockpt_read_checkpoint_user(const char* dir, char* buf, size_t capacity, size_t* length);

/* The complete checkpoint with the largest step count among the immediate
 * subdirectories of `root` (ties: the greatest name); its path goes to out.
 * Incomplete ones (no `meta`) are skipped.  Errors: EFAILED (none found),
 * ENOMEM (capacity). */
int gockpt_find_latest_checkpoint(const char* root, char* out, size_t capacity);

/* Persist the checkpoint the last gockpt_restore left in the arena (restore
 * in place, window IDLE) to `dir`: the background persistence of Sec. 4.4.3.
 * async = 1 returns at once and writes from a library thread;
 * gockpt_persist_wait joins it.  A persist still running is waited for before
 * another persist, before gockpt_begin_window (the arena is about to be
 * reused; Sec. 4.4.3 waits for the previous checkpoint before a new one),
 * before gockpt_load and in gockpt_destroy.  The arena must stay allocated
 * until then.  Errors: ESTATE (no in-place restore since the last window),
 * EINVAL, and with async = 0 those of gockpt_write_checkpoint. */
int gockpt_persist(gockpt_ctx* ctx, const char* dir, const char* user_meta, int nthreads, int async);

/* Wait for the running persist (if any); returns its status (its message via
 * gockpt_last_error(ctx)) and fills stats.  OK when none ran. */
int gockpt_persist_wait(gockpt_ctx* ctx, gockpt_io_stats* stats);

/* Checkpoint loading (Sec. 4.3.2): read a complete checkpoint into host_buf
 * (>= 12 n bytes: master | exp_avg | exp_avg_sq), copy it into the context's
 * device buffers, re-derive the bf16 weights on the device and set the
 * device loss-scaler state (t, tracker, scale), all on the compute stream,
 * which is synchronized before returning.  Training resumes at step t + 1.
 * Window must be IDLE.  Errors: EINVAL (n or hyperparameters differ from the
 * context's, buffer too small), EFAILED (as gockpt_read_checkpoint), EHIP. */
int gockpt_load(gockpt_ctx* ctx, const char* dir, void* host_buf, size_t host_bytes, int nthreads,
                gockpt_ckpt_info* info);

#ifdef __cplusplus
}
#endif

#endif /* GOCKPT_H */
