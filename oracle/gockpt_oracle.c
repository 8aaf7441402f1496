/*
 * gockpt_oracle.c -- plain, slow CPU oracle for the GoCkpt hot path
 * (arXiv 2511.07035).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
 * the benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the HIP library; the two meet only at the
 * seeded inputs the tests hand to both.
 *
 * What it computes (and where the paper says so):
 *   - one mixed-precision AdamW step over a flat parameter space: fp32
 *     master weights and fp32 first/second moments, 16-bit gradients and
 *     16-bit working weights (Sec. 2.2, Mixed-Precision Training; the
 *     optimizer is AdamW, Sec. 4.3.1);
 *   - the loss-scaling skip rule that mixed-precision training relies on
 *     (Sec. 2.2: loss scaling against underflow);
 *   - a synchronous run of K steps -- the checkpoint a blocking snapshot at
 *     the end of the window would hold (Sec. 2.1: step N uses and produces
 *     versioned states M^N, O^N);
 *   - the multi-step window: part j of the state is sent after step j, and at
 *     each later step the gradients of the parts already sent are sent too
 *     (Sec. 4.2.1, Fig. transfer_update);
 *   - the CPU reconstruction: each stale part is brought forward by replaying
 *     AdamW with the saved gradients, which must give the synchronous result
 *     (Sec. 4.3.1, Fig. update_backend).
 *
 * Precision: fp32 for every per-element operation, one IEEE-754 operation per
 * statement, round to nearest even, no fused multiply-add (build with
 * -ffp-contract=off), no flush-to-zero.  fp64 only for the bias-correction
 * powers, where the arithmetic contract places it.  The paper does not print
 * an operation order; the order used here is PyTorch's documented AdamW with
 * decoupled weight decay, one rounding per operation as written out in
 * adamw_element below, and the HIP path follows the same contract
 * from its own code.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fPIC -shared (no -ffast-math).
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#include <math.h>

/* ------------------------------------------------------------------------ */
/* 16-bit floating-point format (bfloat16) -- Sec. 2.2 stores gradients and  */
/* working weights in 16 bits.                                               */
/* ------------------------------------------------------------------------ */

/* bf16 -> fp32 is exact: the bf16 pattern is the top half of the fp32 one. */
float oracle_bf16_to_f32(uint16_t b)
{
    uint32_t u = ((uint32_t)b) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* fp32 -> bf16, round to nearest, ties to even.  Keep the top 16 bits; round
 * up when the dropped low half is above one half of the last kept bit, or
 * exactly one half and the kept pattern is odd.  A carry out of the mantissa
 * moves into the exponent, which is the correct next representable value
 * (and turns the largest finite values into infinity when they round up).
 * Every NaN becomes the canonical quiet NaN 0x7FC0. */
uint16_t oracle_bf16_rne(float x)
{
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    int is_nan = ((u & 0x7F800000u) == 0x7F800000u) && ((u & 0x007FFFFFu) != 0u);
    if (is_nan)
        return 0x7FC0u;
    uint32_t kept = u >> 16;
    uint32_t dropped = u & 0xFFFFu;
    int round_up = 0;
    if (dropped > 0x8000u)
        round_up = 1;
    if (dropped == 0x8000u && (kept & 1u) != 0u)
        round_up = 1;
    if (round_up)
        kept = kept + 1u;
    return (uint16_t)kept;
}

void oracle_bf16_rne_array(size_t n, const float* x, uint16_t* out)
{
    for (size_t i = 0; i < n; i++)
        out[i] = oracle_bf16_rne(x[i]);
}

/* ------------------------------------------------------------------------ */
/* IEEE-754 binary16 (fp16) -- Sec. 2.2 allows FP16 or BF16 gradients.       */
/* ------------------------------------------------------------------------ */

/* binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.  Every
 * binary16 value is exactly representable in fp32:
 *   exponent 0:       (-1)^s * fraction * 2^-24          (zero, subnormals)
 *   exponent 1..30:   (-1)^s * (1024 + fraction) * 2^(e - 25)
 *   exponent 31:      infinity (fraction 0) or NaN.
 * The integer significands (< 2048) and the powers of two are exact in fp32,
 * so each value below is computed without rounding. */
float oracle_fp16_to_f32(uint16_t h)
{
    int sign = (h >> 15) & 1;
    int e = (h >> 10) & 0x1F;
    int f = h & 0x3FF;
    float mag;
    if (e == 0) {
        mag = ldexpf((float)f, -24);
    } else if (e < 31) {
        mag = ldexpf((float)(1024 + f), e - 25);
    } else if (f == 0) {
        mag = INFINITY;
    } else {
        /* quiet NaN carrying the fraction in its top bits */
        uint32_t u = 0x7FC00000u | ((uint32_t)f << 13);
        memcpy(&mag, &u, sizeof mag);
    }
    return sign ? -mag : mag;
}

/* A gradient is non-finite when its exponent field is all ones (inf or NaN):
 * bits 7..14 for bf16, bits 10..14 for fp16. */
static int grad_is_nonfinite(uint16_t b, int fp16)
{
    if (fp16)
        return (b & 0x7C00u) == 0x7C00u;
    return (b & 0x7F80u) == 0x7F80u;
}

static float grad_to_f32(uint16_t b, int fp16)
{
    return fp16 ? oracle_fp16_to_f32(b) : oracle_bf16_to_f32(b);
}

/* ------------------------------------------------------------------------ */
/* Per-step scalars.                                                        */
/* ------------------------------------------------------------------------ */

/* beta^t by binary exponentiation in fp64, scanning the exponent's bits from
 * the most significant one down: square, then multiply by beta where the bit
 * is set.  The fixed order makes the result reproducible on any IEEE-754
 * machine. */
double oracle_powi(double beta, int64_t t)
{
    double r = 1.0;
    for (int bit = 62; bit >= 0; bit--) {
        r = r * r;
        if (((t >> bit) & 1) != 0)
            r = r * beta;
    }
    return r;
}

typedef struct {
    float b1;        /* beta1 rounded to fp32 */
    float b2;        /* beta2 rounded to fp32 */
    float omb1;      /* (1 - beta1) computed in fp64, rounded to fp32 */
    float omb2;      /* (1 - beta2) computed in fp64, rounded to fp32 */
    float eps;       /* eps rounded to fp32 */
    float decay;     /* (1 - lr * wd) computed in fp64, rounded to fp32 */
    float step_size; /* lr / (1 - beta1^t) computed in fp64, rounded to fp32 */
    float sqrt_bc2;  /* sqrt of (1 - beta2^t) rounded to fp32, fp32 sqrt */
    float inv_scale; /* 1 / loss scale, fp32 division */
} oracle_scalars_t;

/* Adam's bias corrections 1 - beta^t for the step count t, the learning rate
 * and the decoupled weight decay factor for this step, and the reciprocal
 * of the loss scale the gradients carry (Sec. 2.2). */
void oracle_step_scalars(double beta1, double beta2, double eps, double weight_decay,
                         float lr, int64_t t, float loss_scale, oracle_scalars_t* s)
{
    double bc1 = 1.0 - oracle_powi(beta1, t);
    double bc2 = 1.0 - oracle_powi(beta2, t);
    double lr_d = (double)lr;
    s->b1 = (float)beta1;
    s->b2 = (float)beta2;
    s->omb1 = (float)(1.0 - beta1);
    s->omb2 = (float)(1.0 - beta2);
    s->eps = (float)eps;
    s->decay = (float)(1.0 - lr_d * weight_decay);
    s->step_size = (float)(lr_d / bc1);
    float bc2_f = (float)bc2;
    s->sqrt_bc2 = sqrtf(bc2_f);
    s->inv_scale = 1.0f / loss_scale;
}

/* ------------------------------------------------------------------------ */
/* One AdamW update of one element.                                         */
/* ------------------------------------------------------------------------ */

/* The gradient is unscaled first (it arrives multiplied by the loss scale),
 * then the moments are updated, the decoupled weight decay shrinks the
 * master weight, and the bias-corrected Adam step is subtracted. */
static void adamw_element(const oracle_scalars_t* s, uint16_t grad_bits, int fp16,
                          float* p_io, float* m_io, float* v_io)
{
    float p = *p_io;
    float m = *m_io;
    float v = *v_io;

    float g = grad_to_f32(grad_bits, fp16);
    g = g * s->inv_scale;

    float m_keep = s->b1 * m;
    float m_new = s->omb1 * g;
    m = m_keep + m_new;

    float g2 = g * g;
    float v_keep = s->b2 * v;
    float v_new = s->omb2 * g2;
    v = v_keep + v_new;

    p = p * s->decay;

    float root = sqrtf(v);
    float denom = root / s->sqrt_bc2;
    denom = denom + s->eps;
    float ratio = m / denom;
    float delta = s->step_size * ratio;
    p = p - delta;

    *p_io = p;
    *m_io = m;
    *v_io = v;
}

/* ------------------------------------------------------------------------ */
/* Hyperparameters, loss scaler, per-step record.                           */
/* ------------------------------------------------------------------------ */

typedef struct {
    double beta1, beta2, eps, weight_decay;
    int32_t check_overflow;   /* skip a step whose gradients hold inf/NaN */
    int32_t dynamic_scale;    /* grow/back off the loss scale */
    float growth_factor;
    float backoff_factor;
    float min_scale;
    int32_t grad_fp16;        /* 1: gradients are binary16, 0: bfloat16 */
    int64_t growth_interval;
} oracle_hparams_t;

typedef struct {
    int64_t t;        /* Adam step count (advances only on applied steps) */
    float scale;      /* loss scale the next step's gradients carry */
    int32_t pad_;
    int64_t tracker;  /* consecutive applied steps since the last change */
} oracle_scaler_t;

typedef struct {
    int64_t t;          /* step count used by this step (after the advance) */
    int32_t skip;       /* 1: step skipped, state unchanged */
    float scale_used;   /* loss scale the step's gradients carried */
    float lr;           /* learning rate of the step */
    int32_t pad_;
    double gnorm2;      /* sum of squares of the unscaled gradient (fp64) */
} oracle_record_t;

/* Decide skip, advance t, and move the loss scale (dynamic loss scaling as in
 * mixed-precision training, Sec. 2.2).  Returns the skip flag. */
static int scaler_advance(const oracle_hparams_t* hp, oracle_scaler_t* st, int nonfinite)
{
    int skip = (hp->check_overflow != 0) && (nonfinite != 0);
    if (skip) {
        if (hp->dynamic_scale) {
            float reduced = st->scale * hp->backoff_factor;
            st->scale = reduced < hp->min_scale ? hp->min_scale : reduced;
            st->tracker = 0;
        }
    } else {
        st->t = st->t + 1;
        if (hp->dynamic_scale) {
            st->tracker = st->tracker + 1;
            if (st->tracker == hp->growth_interval) {
                st->scale = st->scale * hp->growth_factor;
                st->tracker = 0;
            }
        }
    }
    return skip;
}

int oracle_any_nonfinite(size_t n, const uint16_t* g, int fp16)
{
    for (size_t i = 0; i < n; i++)
        if (grad_is_nonfinite(g[i], fp16))
            return 1;
    return 0;
}

double oracle_grad_norm2(size_t n, const uint16_t* g, float inv_scale, int fp16)
{
    double acc = 0.0;
    for (size_t i = 0; i < n; i++) {
        double x = (double)grad_to_f32(g[i], fp16) * (double)inv_scale;
        acc += x * x;
    }
    return acc;
}

/* ------------------------------------------------------------------------ */
/* One full optimizer step over the flat space.                             */
/* ------------------------------------------------------------------------ */

/* nonfinite_override: -1 scans the given gradients; 0 or 1 forces the global
 * flag (used when only a sample of a large parameter space is passed in and
 * the flag comes from the whole gradient). */
void oracle_adamw_step(size_t n, float* p, float* m, float* v, uint16_t* w,
                       const uint16_t* g, float lr, int nonfinite_override,
                       const oracle_hparams_t* hp, oracle_scaler_t* st,
                       oracle_record_t* rec)
{
    int nonfinite = nonfinite_override >= 0 ? nonfinite_override : oracle_any_nonfinite(n, g, hp->grad_fp16);
    float scale_used = st->scale;
    int skip = scaler_advance(hp, st, nonfinite);
    rec->t = st->t;
    rec->skip = skip;
    rec->scale_used = scale_used;
    rec->lr = lr;
    rec->pad_ = 0;
    oracle_scalars_t s;
    oracle_step_scalars(hp->beta1, hp->beta2, hp->eps, hp->weight_decay, lr, st->t, scale_used, &s);
    rec->gnorm2 = oracle_grad_norm2(n, g, s.inv_scale, hp->grad_fp16);
    if (skip)
        return;
    for (size_t i = 0; i < n; i++) {
        adamw_element(&s, g[i], hp->grad_fp16, &p[i], &m[i], &v[i]);
        if (w != NULL)
            w[i] = oracle_bf16_rne(p[i]);
    }
}

/* K synchronous steps: the state a blocking checkpoint taken after the K-th
 * step would hold.  grads holds K rows of n gradients, row s-1 for step s. */
void oracle_sync_run(size_t n, int K, float* p, float* m, float* v, uint16_t* w,
                     const uint16_t* grads, const float* lrs, const int32_t* nonfinite,
                     const oracle_hparams_t* hp, oracle_scaler_t* st, oracle_record_t* recs)
{
    for (int s = 1; s <= K; s++) {
        int override = nonfinite != NULL ? nonfinite[s - 1] : -1;
        oracle_adamw_step(n, p, m, v, w, grads + (size_t)(s - 1) * n, lrs[s - 1],
                          override, hp, st, &recs[s - 1]);
    }
}

/* Offset, in elements, of step s's gradient block in the packed gradient
 * store: step s sends the gradients of parts 1..s-1, i.e. of elements
 * [0, bounds[s-1]); the blocks are laid end to end for s = 1..K. */
int64_t oracle_sent_offset(const int64_t* bounds, int s)
{
    int64_t off = 0;
    for (int r = 1; r < s; r++)
        off += bounds[r - 1];
    return off;
}

/* The multi-step window (Sec. 4.2.1): the state is split into K parts
 * [bounds[j-1], bounds[j]).  At window step s the step runs, then part s of
 * the freshly updated state is captured, and the gradients this step used for
 * the parts already captured (parts 1..s-1) are captured too.  A skipped step
 * uses no gradients, so none are captured for it. */
void oracle_window_capture(size_t n, int K, const int64_t* bounds,
                           float* p, float* m, float* v, uint16_t* w,
                           const uint16_t* grads, const float* lrs, const int32_t* nonfinite,
                           const oracle_hparams_t* hp, oracle_scaler_t* st, oracle_record_t* recs,
                           float* snap_p, float* snap_m, float* snap_v, uint16_t* sent)
{
    for (int s = 1; s <= K; s++) {
        const uint16_t* g = grads + (size_t)(s - 1) * n;
        int override = nonfinite != NULL ? nonfinite[s - 1] : -1;
        oracle_adamw_step(n, p, m, v, w, g, lrs[s - 1], override, hp, st, &recs[s - 1]);
        for (int64_t i = bounds[s - 1]; i < bounds[s]; i++) {
            snap_p[i] = p[i];
            snap_m[i] = m[i];
            snap_v[i] = v[i];
        }
        if (!recs[s - 1].skip) {
            int64_t off = oracle_sent_offset(bounds, s);
            for (int64_t i = 0; i < bounds[s - 1]; i++)
                sent[off + i] = g[i];
        }
    }
}

/* CPU reconstruction (Sec. 4.3.1): part j was captured after step j; replay
 * steps j+1..K on it with the captured gradients and each step's recorded
 * step count, learning rate and loss scale.  Skipped steps are not replayed.
 * The result is the state after step K for every part; the 16-bit working
 * weights are re-derived from the master weights. */
void oracle_replay_restore(size_t n, int K, const int64_t* bounds,
                           const float* snap_p, const float* snap_m, const float* snap_v,
                           const uint16_t* sent, const oracle_record_t* recs,
                           const oracle_hparams_t* hp,
                           float* out_p, float* out_m, float* out_v, uint16_t* out_w)
{
    (void)n;
    for (int j = 1; j <= K; j++) {
        for (int64_t i = bounds[j - 1]; i < bounds[j]; i++) {
            out_p[i] = snap_p[i];
            out_m[i] = snap_m[i];
            out_v[i] = snap_v[i];
        }
        for (int s = j + 1; s <= K; s++) {
            const oracle_record_t* r = &recs[s - 1];
            if (r->skip)
                continue;
            oracle_scalars_t sc;
            oracle_step_scalars(hp->beta1, hp->beta2, hp->eps, hp->weight_decay,
                                r->lr, r->t, r->scale_used, &sc);
            const uint16_t* g = sent + oracle_sent_offset(bounds, s);
            for (int64_t i = bounds[j - 1]; i < bounds[j]; i++)
                adamw_element(&sc, g[i], hp->grad_fp16, &out_p[i], &out_m[i], &out_v[i]);
        }
        if (out_w != NULL)
            for (int64_t i = bounds[j - 1]; i < bounds[j]; i++)
                out_w[i] = oracle_bf16_rne(out_p[i]);
    }
}
