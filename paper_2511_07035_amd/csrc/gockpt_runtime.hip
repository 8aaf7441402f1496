// gockpt_runtime.hip -- host runtime of the GoCkpt hot path: context, window
// state machine, staging-ring planning, the side-stream D2H drain, the staged
// path into pageable host memory and the in-window replay.
//
// Per step (update_begin hook, Sec. 4.6) on the compute stream:
//   [wait for last step's direct copies of state] -> prepass -> finalize
//   -> fused update+pack -> event.
// Inside a window the copies of the step follow on the copy stream: first
// the gradients the ring could not take, straight from the gradient buffer,
// as soon as the gradients are complete (they overlap the update and the
// next forward pass, Sec. 4.2.4); then, after the update, the step record,
// the ring part of the pack list and the rest of the state straight from the
// live buffers, overlapping the next step's forward/backward.  Gradient
// copies come first (Sec. 4.2.2 gives gradient transfers priority).
//
// Ring accounting: the ring is a byte stream written at a monotonically
// increasing logical offset; physical offset = logical mod ring_bytes.  How
// much of it a step may use is the ring plan of the window:
//   QUERY        the space whose earlier copies have completed when the host
//                calls gockpt_step (queried, never waited for);
//   HOST_WAIT    the same, decided once the device reaches the update (the
//                calling thread blocks until then);
//   DEVICE_WAIT  the whole ring, as if every earlier copy had finished by the
//                update; the compute stream waits for the copies of the ring
//                ranges the step overwrites (never blocks the host).
// What does not fit is copied straight from the live buffers ("direct
// spill"); the next update then waits for the state copies, and the next
// backward -- via gockpt_backward_begin -- for the gradient copies.
//
// Host side: a pinned arena receives the copies directly ("direct" window).
// A pageable arena -- larger than what the host can pin -- is reached through
// pinned staging slots ("staged" window): copy q lands in slot q mod nslots,
// and worker threads move landed slots into the arena in copy order.  Every
// copy is queued by gockpt_step itself; before a copy that reuses a slot the
// copy stream runs a gate kernel that waits until the host has released the
// slot's previous copy (a counter in the context's host-coherent control
// page), so neither the caller nor a library thread waits for staging space.
// With in-window replay (replay_every = R < K) a replayer thread applies
// every batch of R landed steps to the parts already received (the CPU update
// of Sec. 4.3.1, run during the window), so only R steps of gradients are
// kept.
//
// Deadlock freedom: device-side waits are only on events recorded earlier in
// program order, and a gate only on the release of copies queued before it
// (their landing needs nothing queued after the gate); host threads wait only
// for work that is already queued on the device or on another host thread
// that does not wait on them.
#include <hip/hip_runtime.h>

#include <dlfcn.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <chrono>
#include <condition_variable>
#include <deque>
#include <iterator>
#include <map>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "gockpt_internal.h"

namespace gockpt {
void arena_layout(int K, const int64_t* b, int64_t n, int R, gockpt_arena_layout* lay, uint64_t* goff);
bool valid_bounds(int K, const int64_t* b, int64_t n);
int check_records(int K, const gockpt_step_record* rec, int upto, const HParams& hp, StepScalars* sc,
                  std::string& err);
int64_t replay_parts(int K, const int64_t* bounds, const gockpt_step_record* rec, const StepScalars* sc,
                     const uint16_t* const* gblk, int first_part, int last_part, int s_lo, int s_hi,
                     const float* ip, const float* im, const float* iv, float* op, float* om, float* ov,
                     uint16_t* w_out, int nthreads, int grad_kind);
int replay_window(int K, const int64_t* bounds, int64_t n, uint8_t* arena, size_t arena_bytes, int R,
                  int s_first, const HParams& hp, int grad_kind, float* p_out, float* m_out, float* v_out,
                  uint16_t* w_out, gockpt_ckpt_meta* meta, int nthreads, int64_t earlier_updates,
                  std::string& err);
int launch_cast_bf16(const float* p, uint16_t* w, int64_t n, hipStream_t stream);
void set_host_error(const std::string& msg);
void copy_to_arena(void* dst, const void* src, size_t len);
}  // namespace gockpt

using namespace gockpt;

namespace {

enum class WinState { Idle, Window, Draining, Drained, Restoring, Failed };

struct RingCopy {
    uint64_t lbeg, lend;  // logical ring range this copy drains
    hipEvent_t ev;        // set once the copy is queued (staged windows queue it later)
};

// One device -> host copy of at most copy_bytes that never crosses the
// ring's end.
struct Job {
    const uint8_t* src;
    uint64_t dst_off;  // byte offset in the arena
    uint64_t bytes;
    RingCopy* ring;    // the ring segment's bookkeeping entry, on its last copy only (records its event)
    bool grad;         // a gradient block (its slot may wait for a replay)
    bool from_ring;    // the source is the staging ring
};

struct StepTiming {
    hipEvent_t pre0, pre1, upd0, upd1, cp0, cp1;
    bool has_copy;
    uint64_t ring_bytes;       // bytes planned into the ring this step
    uint64_t ring_grad_bytes;  // of which gradients (not packed when the step is skipped)
};

// The copies of one window step, planned by gockpt_step and queued on the
// copy stream at once or, with defer_copies, at the library's next call.
struct StepCopies {
    bool active = false;
    int s = 0;
    std::vector<Job> jobs;  // in copy order
    StepTiming tm{};
    bool timed = false;
    int first_after_kernel = 0;  // jobs before it need only the gradients
    int last_spill_g = -1, last_spill_s = -1, last_grad_job = -1;
    bool grads_ready_ev = false;  // ev_grads_ready was recorded for this step
};

// A staged copy: after `ev` its bytes are in `slot`; a worker moves them to
// the arena and releases copy number `seq`.
struct Landing {
    hipEvent_t ev;
    uint8_t* slot;
    uint64_t dst_off;
    uint64_t len;
    uint64_t seq;
    int step;
    bool grad;
};

// Longest a gate kernel waits for the host to free a staging slot (ticks of
// the 100 MHz constant clock): 120 s.  A gate that gives up marks the window
// failed.
constexpr uint64_t kGateTicks = 120ull * 100000000ull;

thread_local std::string g_create_error;

// Optional roctx ranges around the library's phases (GOCKPT_ROCTX=1): the
// marker library is opened at run time, so nothing links against it and a
// context without the variable pays one null test per range.
struct Roctx {
    int (*push)(const char*) = nullptr;
    int (*pop)() = nullptr;
};
Roctx g_roctx;
std::once_flag g_roctx_once;

void load_roctx() {
    std::call_once(g_roctx_once, [] {
        void* h = dlopen("librocprofiler-sdk-roctx.so.1", RTLD_NOW | RTLD_LOCAL);
        if (h == nullptr) h = dlopen("libroctx64.so", RTLD_NOW | RTLD_LOCAL);
        if (h == nullptr) return;
        g_roctx.push = reinterpret_cast<int (*)(const char*)>(dlsym(h, "roctxRangePushA"));
        g_roctx.pop = reinterpret_cast<int (*)()>(dlsym(h, "roctxRangePop"));
        if (g_roctx.push == nullptr || g_roctx.pop == nullptr) g_roctx = Roctx{};
    });
}

// A roctx range for the scope's duration when `on`.
struct Range {
    bool on;
    Range(bool enabled, const char* fmt, ...) : on(enabled && g_roctx.push != nullptr) {
        if (!on) return;
        char buf[96];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        g_roctx.push(buf);
    }
    ~Range() {
        if (on) g_roctx.pop();
    }
    Range(const Range&) = delete;
    Range& operator=(const Range&) = delete;
};

constexpr size_t kStepFields = 5;  // per step in gockpt_window_step_times

uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

// Error text of the host-only calls, read with gockpt_last_error(NULL).
void gockpt::set_host_error(const std::string& msg) { g_create_error = msg; }

struct gockpt_ctx {
    gockpt_config cfg;
    HParams hp;
    ScalerCfg sc;
    StepScalars konst;
    hipStream_t cs = nullptr, xs = nullptr;
    uint8_t* ws = nullptr;
    int pre_blocks = 1;
    Knobs knobs{1, 1, 1, 1, kBlock};
    size_t copy_bytes = GOCKPT_DEFAULT_COPY_BYTES;
    std::string err;

    // ---- window (main thread) ----
    WinState st = WinState::Idle;
    int K = 0, s = 0;
    std::vector<int64_t> bounds;
    uint8_t* arena = nullptr;
    size_t arena_bytes = 0;
    gockpt_arena_layout lay{};
    std::vector<uint64_t> goff;
    bool staged = false;
    int R = 0;  // in-window replay batch (0: none)
    int wait_policy = GOCKPT_WAIT_LAZY;
    bool ring_off = false;  // this window copies everything from the live buffers
    int ring_plan = GOCKPT_RING_QUERY;  // how a step decides its ring use
    bool win_timing = false;  // this window records timing events (cfg.timing, unless the window opts out)
    bool defer = false;       // defer_copies of the window
    StepCopies deferred;      // a window step's copies not queued yet (defer)
    uint64_t ring_waited = 0;  // DEVICE_WAIT: logical ring offset the compute stream has waited through
    int replay_threads = 8;
    uint64_t head = 0;  // ring logical write offset
    hipEvent_t ev_kernel = nullptr, ev_last_copy = nullptr, ev_grads_copied = nullptr;
    hipEvent_t ev_fin = nullptr;  // after each window step's finalize (its skip decision is on the host)
    hipEvent_t ev_grads_ready = nullptr;
    hipEvent_t ev_grad_spill = nullptr, ev_state_spill = nullptr;
    bool grad_spill_pending = false, state_spill_pending = false, backward_called = true;
    bool any_copy = false;
    std::vector<StepTiming> timing;
    gockpt_window_stats stats{};  // bytes_host_copied, host_copy_ms, replay_ms: written by library threads under mu
    std::vector<gockpt_step_record> records;
    std::vector<uint64_t> ring_grad_bytes;  // per window step: gradient bytes planned into the ring
    std::vector<double> step_ms;  // kStepFields per step after drain (timing on)

    // ---- shared with the library threads (guarded by mu) ----
    std::mutex mu;
    std::condition_variable cv;
    std::deque<RingCopy> inflight;
    std::vector<hipEvent_t> event_pool;
    std::vector<hipEvent_t> timing_pool;
    std::vector<hipEvent_t> all_events;
    std::deque<Landing> land_q;
    uint64_t landings_open = 0;         // staged copies queued and not yet handled by a worker
    std::vector<int> pending;           // per step: staged copies not yet landed
    std::vector<char> issued;           // per step: all copies queued on the device
    std::vector<hipEvent_t> step_done;  // direct windows: per step, after its copies
    int issued_through = 0, landed_through = 0, replayed_through = 0;
    int64_t replay_updates = 0;
    // staging slots (staged windows): copy number q uses slot q mod nslots
    uint8_t* staging = nullptr;
    uint64_t nslots = 0;
    uint64_t seq = 0;           // staged copies queued over the context's life (main thread)
    uint64_t gate_through = 0;  // copies below gate_through + nslots need no further gate (main thread)
    uint64_t released = 0;      // copies released in order (mu)
    std::vector<char> slot_done;  // released out of order, waiting for the earlier ones (mu)
    // host-coherent control page (gockpt_create allocates it; none without)
    CtrlPage* ctrl = nullptr;
    CtrlPage* ctrl_dev = nullptr;
    bool scratch_ws = false;  // the workspace is the library's static scratch (gockpt_create_noalloc)
    int device = 0;
    bool thread_error = false;
    std::string thread_err;
    bool shutdown = false, cancel = false;
    // Fault injection for tests of the error paths: the copy with this
    // 1-based index (counted over the context's life, GOCKPT_TEST_FAIL_COPY)
    // reports an error without reaching the device; 0 = off.
    int64_t fail_copy_at = 0;
    // Debug switches read at create: GOCKPT_DEBUG_POISON=1 fills every ring
    // range and staging slot with 0xFF bytes (a NaN pattern) once its copy
    // has been taken, so a copy that reads a range before the pack wrote it,
    // or a pack that overwrites one before its copy, shows up as a parity
    // failure; GOCKPT_DEBUG_CHECKS=1 checks the ring and staging order
    // invariants on the host at every window step; GOCKPT_ROCTX=1 wraps the
    // library's phases in roctx ranges.
    bool dbg_poison = false, dbg_checks = false, roctx = false;
    std::atomic<int64_t> copies_issued{0};
    std::thread replayer;
    std::vector<std::thread> workers;

    // ---- bucket scans of the coming step (see gockpt_scan_grads) ----
    int scan_bank = 0;       // which of the two partial banks this step's scans fill
    int scan_used = 0;       // partial slots used in that bank
    int64_t scan_covered = 0;
    std::map<int64_t, int64_t> scan_ranges;  // begin -> end
    // one event per stream other than the compute stream, re-recorded after
    // each scan on it: stream order makes the last one cover them all
    std::vector<std::pair<hipStream_t, hipEvent_t>> scan_events;

    // ---- background restore (main thread joins; the thread writes only
    // the restore_* results) ----
    std::thread restorer;
    int restore_rc = GOCKPT_OK;
    std::string restore_err;
    gockpt_ckpt_meta restore_meta{};
    bool restore_in_place = false;

    // ---- persistence ----
    bool ckpt_in_arena = false;  // the last restore left the checkpoint in the arena
    gockpt_ckpt_meta last_meta{};
    std::thread persister;
    int persist_rc = GOCKPT_OK;
    std::string persist_err;
    gockpt_io_stats persist_stats{};

    // Every window copy goes through here.
    hipError_t copy_d2h(void* dst, const void* src, size_t bytes) {
        if (fail_copy_at > 0 && copies_issued.fetch_add(1) + 1 == fail_copy_at) return hipErrorInvalidValue;
        return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, xs);
    }
    int fail(int code, const char* fmt, ...) {
        char buf[512];
        va_list ap;
        va_start(ap, fmt);
        vsnprintf(buf, sizeof buf, fmt, ap);
        va_end(ap);
        err = buf;
        return code;
    }
    int hip_fail(hipError_t e, const char* what) {
        if (st == WinState::Window || st == WinState::Draining) st = WinState::Failed;
        return fail(GOCKPT_EHIP, "%s: %s", what, hipGetErrorString(e));
    }
    // Call with mu held.
    hipEvent_t take_event_locked() {
        if (!event_pool.empty()) {
            hipEvent_t e = event_pool.back();
            event_pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreateWithFlags(&e, hipEventDisableTiming) != hipSuccess) return nullptr;
        all_events.push_back(e);
        return e;
    }
    hipEvent_t take_event() {
        std::lock_guard<std::mutex> lk(mu);
        return take_event_locked();
    }
    hipEvent_t take_timing_event() {
        std::lock_guard<std::mutex> lk(mu);
        if (!timing_pool.empty()) {
            hipEvent_t e = timing_pool.back();
            timing_pool.pop_back();
            return e;
        }
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        all_events.push_back(e);
        return e;
    }
    void recycle_timing() {
        std::lock_guard<std::mutex> lk(mu);
        for (auto& t : timing) {
            timing_pool.push_back(t.pre0);
            timing_pool.push_back(t.pre1);
            timing_pool.push_back(t.upd0);
            timing_pool.push_back(t.upd1);
            if (t.has_copy) {
                timing_pool.push_back(t.cp0);
                timing_pool.push_back(t.cp1);
            }
        }
        timing.clear();
    }
    // Pop ring copies that have finished; returns the oldest logical offset
    // still in use (head if none).  An entry whose copy is not queued yet
    // (staged windows) is still in use.
    uint64_t reclaim() {
        std::lock_guard<std::mutex> lk(mu);
        while (!inflight.empty()) {
            hipEvent_t ev = inflight.front().ev;
            if (ev == nullptr) break;
            hipError_t q = hipEventQuery(ev);
            if (q != hipSuccess) {
                if (q != hipErrorNotReady) (void)hipGetLastError();
                break;
            }
            event_pool.push_back(ev);
            inflight.pop_front();
        }
        return inflight.empty() ? head : inflight.front().lbeg;
    }
    // mu held.  Copy `q` is out of its staging slot; publish how many copies
    // are released in order (gate kernels read it).
    void release_locked(uint64_t q) {
        slot_done[q % nslots] = 1;
        while (slot_done[released % nslots] && released < seq_snapshot_locked()) {
            slot_done[released % nslots] = 0;
            ++released;
        }
        publish_released(released);
    }
    uint64_t queued_seq = 0;  // copies pushed to land_q (mu): released never passes it
    uint64_t seq_snapshot_locked() const { return queued_seq; }
    void publish_released(uint64_t v) {
        if (ctrl != nullptr) __atomic_store_n(&ctrl->released, v, __ATOMIC_RELEASE);
    }
    // mu held.  Advance landed_through over steps whose copies all landed.
    void advance_landed_locked() {
        while (landed_through < K && issued[landed_through + 1] && pending[landed_through + 1] == 0)
            ++landed_through;
    }
    void set_thread_error(const std::string& m) {
        std::lock_guard<std::mutex> lk(mu);
        if (!thread_error) thread_err = m;
        thread_error = true;
        cv.notify_all();
    }
    bool has_thread_error() {
        std::lock_guard<std::mutex> lk(mu);
        return thread_error;
    }
    int thread_fail() {
        std::string m;
        {
            std::lock_guard<std::mutex> lk(mu);
            m = thread_err;
        }
        if (st == WinState::Window || st == WinState::Draining || st == WinState::Drained) st = WinState::Failed;
        return fail(GOCKPT_EFAILED, "window failed in a library thread: %s", m.c_str());
    }
};

namespace {

// ---------------------------------------------------------------------------
// Library threads.
// ---------------------------------------------------------------------------

void drop_deferred(gockpt_ctx* c);

// Staged windows: move landed slots into the pageable arena, in copy order.
// A gradient copy with in-window replay first waits until the replay of the
// batch whose arena slot it reuses is done (that batch's copies all came
// earlier, so workers handling them are never behind this one).  After an
// error or a cancel the slot is only released: nothing more is written to
// the arena.
void worker_loop(gockpt_ctx* c) {
    for (;;) {
        Landing L;
        {
            std::unique_lock<std::mutex> lk(c->mu);
            c->cv.wait(lk, [&] { return c->shutdown || !c->land_q.empty(); });
            if (c->land_q.empty()) return;
            L = c->land_q.front();
            c->land_q.pop_front();
        }
        hipError_t e = hipEventSynchronize(L.ev);
        std::string why;
        if (e != hipSuccess) why = std::string("staged landing: ") + hipGetErrorString(e);
        if (why.empty() && __atomic_load_n(&c->ctrl->gate_timeout, __ATOMIC_ACQUIRE) != 0u)
            why = "a staging gate timed out waiting for the host to free a slot";
        bool write = why.empty();
        if (write && L.grad && c->R > 0) {
            const int need = (L.step - 1) / c->R * c->R;
            std::unique_lock<std::mutex> lk(c->mu);
            c->cv.wait(lk, [&] { return c->thread_error || c->cancel || c->replayed_through >= need; });
            write = !c->thread_error && !c->cancel;
        } else if (write) {
            std::lock_guard<std::mutex> lk(c->mu);
            write = !c->thread_error && !c->cancel;
        }
        double copy_ms = 0.0;
        if (write) {
            const auto t0 = std::chrono::steady_clock::now();
            copy_to_arena(c->arena + L.dst_off, L.slot, L.len);
            copy_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
        }
        if (c->dbg_poison) memset(L.slot, 0xFF, L.len);  // a copy landing late, or read early, now reads NaNs
        std::lock_guard<std::mutex> lk(c->mu);
        if (write) {
            c->stats.bytes_host_copied += L.len;
            c->stats.host_copy_ms += copy_ms;
        }
        c->event_pool.push_back(L.ev);
        c->pending[L.step]--;
        c->landings_open--;
        c->release_locked(L.seq);
        if (!why.empty() && !c->thread_error) {
            c->thread_error = true;
            c->thread_err = why;
        }
        c->advance_landed_locked();
        c->cv.notify_all();
    }
}

// In-window replay: after every R landed steps, apply them to the parts
// already received.
void replayer_loop(gockpt_ctx* c) {
    const int K = c->K, R = c->R;
    std::vector<StepScalars> scal(K);
    std::vector<const uint16_t*> gblk(K);
    for (int s = 1; s <= K; ++s) gblk[s - 1] = reinterpret_cast<const uint16_t*>(c->arena + c->goff[s - 1]);
    float* ap = reinterpret_cast<float*>(c->arena + c->lay.master);
    float* am = reinterpret_cast<float*>(c->arena + c->lay.exp_avg);
    float* av = reinterpret_cast<float*>(c->arena + c->lay.exp_avg_sq);
    const gockpt_step_record* rec = reinterpret_cast<const gockpt_step_record*>(c->arena + c->lay.records);
    int done = 0;
    while (done < K) {
        const int b = done + R < K ? done + R : K;
        if (!c->staged) {
            // direct window: step b's copies are the last of steps <= b on the copy stream
            hipEvent_t ev = nullptr;
            {
                std::unique_lock<std::mutex> lk(c->mu);
                c->cv.wait(lk, [&] { return c->cancel || c->thread_error || c->issued_through >= b; });
                if (c->cancel || c->thread_error) return;
                ev = c->step_done[b];
            }
            hipError_t e = hipEventSynchronize(ev);
            if (e != hipSuccess) {
                c->set_thread_error(std::string("replay wait: ") + hipGetErrorString(e));
                return;
            }
        } else {
            std::unique_lock<std::mutex> lk(c->mu);
            c->cv.wait(lk, [&] { return c->cancel || c->thread_error || c->landed_through >= b; });
            if (c->cancel || c->thread_error) return;
        }
        std::string err;
        if (check_records(K, rec, b, c->hp, scal.data(), err) != GOCKPT_OK) {
            c->set_thread_error(err);
            return;
        }
        const auto t0 = std::chrono::steady_clock::now();
        const int64_t u = replay_parts(K, c->bounds.data(), rec, scal.data(), gblk.data(), 1, b - 1, done + 1, b, ap,
                                       am, av, ap, am, av, nullptr, c->replay_threads, c->cfg.grad_dtype);
        const double ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
        std::lock_guard<std::mutex> lk(c->mu);
        c->stats.replay_ms += ms;
        c->replay_updates += u;
        c->replayed_through = b;
        c->cv.notify_all();
        done = b;
    }
}

// own_ws: the workspace is the library's static scratch (the caller passes
// none).
int check_config(const gockpt_config* c, std::string& e, bool own_ws = false) {
    char buf[256];
    auto bad = [&](const char* m) {
        e = m;
        return GOCKPT_EINVAL;
    };
    if (c == nullptr) return bad("config is NULL");
    if (c->n < 0) return bad("n < 0");
    if (c->n > 0) {
        if (!c->master || !c->exp_avg || !c->exp_avg_sq || !c->grad16)
            return bad("master, exp_avg, exp_avg_sq and grad16 are required");
        if (!aligned(c->master, 16) || !aligned(c->exp_avg, 16) || !aligned(c->exp_avg_sq, 16) ||
            !aligned(c->grad16, 16) || (c->weight_bf16 && !aligned(c->weight_bf16, 16)))
            return bad("device state buffers must be 16-byte aligned");
    }
    if (!(c->beta1 >= 0.0 && c->beta1 < 1.0) || !(c->beta2 >= 0.0 && c->beta2 < 1.0))
        return bad("betas must lie in [0, 1)");
    if (!(c->eps >= 0.0) || !isfinite(c->eps) || !isfinite(c->weight_decay)) return bad("eps/weight_decay");
    if (!(c->init_scale > 0.0f) || !isfinite(c->init_scale)) return bad("init_scale must be finite and > 0");
    if (c->dynamic_scale) {
        if (!(c->growth_factor > 0.0f) || !(c->backoff_factor > 0.0f) || !(c->min_scale > 0.0f))
            return bad("scaler factors must be > 0");
        if (c->growth_interval < 1) return bad("growth_interval must be >= 1");
    }
    if (c->init_step < 0 || c->init_tracker < 0) return bad("init_step/init_tracker < 0");
    if (c->grad_dtype != GOCKPT_GRAD_BF16 && c->grad_dtype != GOCKPT_GRAD_FP16) return bad("unknown grad_dtype");
    if (c->grad_norm_off != 0 && c->grad_norm_off != 1) return bad("grad_norm_off must be 0 or 1");
    if (c->found_inf != nullptr && !aligned(c->found_inf, 4)) return bad("found_inf must be 4-byte aligned");
    if (c->ring != nullptr) {
        if (!aligned(c->ring, 256) || c->ring_bytes % 256 != 0) return bad("ring must be 256-byte aligned and sized");
    } else if (c->ring_bytes != 0) {
        return bad("ring_bytes without ring");
    }
    if (c->copy_bytes % 256 != 0) return bad("copy_bytes must be a multiple of 256");
    if (own_ws) {
        if (c->workspace != nullptr || c->workspace_bytes != 0)
            return bad("gockpt_create_noalloc uses the library's scratch workspace: workspace must be NULL, 0 bytes");
        if (c->host_staging != nullptr)
            return bad("gockpt_create_noalloc takes no host staging (staged windows need a control page it does not "
                       "allocate)");
    } else if (c->workspace == nullptr || !aligned(c->workspace, 256)) {
        return bad("workspace must be 256-byte aligned");
    } else if (c->workspace_bytes < gockpt_workspace_bytes(c->n)) {
        snprintf(buf, sizeof buf, "workspace has %zu bytes, needs %zu", c->workspace_bytes,
                 gockpt_workspace_bytes(c->n));
        e = buf;
        return GOCKPT_ENOMEM;
    }
    if (c->compute_stream == c->copy_stream) return bad("copy stream must differ from the compute stream");
    if (c->host_staging != nullptr) {
        const size_t slot = c->copy_bytes ? c->copy_bytes : GOCKPT_DEFAULT_COPY_BYTES;
        if (!aligned(c->host_staging, 256) || c->host_staging_bytes < 2 * slot)
            return bad("host_staging must be 256-byte aligned and hold at least two copy_bytes slots");
    }
    return GOCKPT_OK;
}

// Wait for a background persist; its status stays in persist_rc.
void join_persist(gockpt_ctx* c) {
    if (c->persister.joinable()) c->persister.join();
}

// The replay of a drained window (restore): steps not replayed during the
// window, onto every part; outputs NULL = in place in the arena.
int run_restore(gockpt_ctx* c, float* p, float* m, float* v, uint16_t* w, int nthreads, gockpt_ckpt_meta* meta,
                std::string& err) {
    const int s_first = c->R > 0 ? c->K + 1 : 2;  // the in-window replay already applied every step
    return replay_window(c->K, c->bounds.data(), c->cfg.n, c->arena, c->arena_bytes, c->R, s_first, c->hp,
                         c->cfg.grad_dtype, p, m, v, w, meta, nthreads, c->replay_updates, err);
}

// Wait for a background restore and take its result: IDLE on success,
// FAILED otherwise.  GOCKPT_OK when none was running.
int finish_restore(gockpt_ctx* c) {
    if (!c->restorer.joinable()) return GOCKPT_OK;
    c->restorer.join();
    if (c->restore_rc != GOCKPT_OK) {
        c->st = WinState::Failed;
        return c->fail(c->restore_rc, "%s", c->restore_err.c_str());
    }
    c->last_meta = c->restore_meta;
    c->ckpt_in_arena = c->restore_in_place;
    c->st = WinState::Idle;
    return GOCKPT_OK;
}

void stop_threads(gockpt_ctx* c) {
    {
        std::lock_guard<std::mutex> lk(c->mu);
        c->shutdown = true;
        c->cancel = true;
        c->cv.notify_all();
    }
    if (c->replayer.joinable()) c->replayer.join();
    for (auto& w : c->workers)
        if (w.joinable()) w.join();
    c->workers.clear();
}

// Wait until every staged copy queued so far has been handled by a worker,
// then stop the replayer (optionally cancelling the batches it has not
// started); used by abort and destroy.  With cancel_replay the gates on the
// copy stream are opened first (the released counter jumps ahead) and the
// workers only release their slots, so the wait ends even after an error --
// and no library thread or copy touches the arena or the staging slots once
// it returns, even when the caller frees them next.  The counter is then set
// back to the copies actually released.
void quiesce(gockpt_ctx* c, bool cancel_replay) {
    if (cancel_replay) {
        std::lock_guard<std::mutex> lk(c->mu);
        c->cancel = true;
        c->publish_released(UINT64_MAX / 2);
        c->cv.notify_all();
    }
    if (c->staged || c->landings_open > 0) {
        std::unique_lock<std::mutex> lk(c->mu);
        c->cv.wait(lk, [&] { return c->land_q.empty() && c->landings_open == 0; });
    }
    if (c->replayer.joinable()) c->replayer.join();
    // a gate queued just before a copy that then failed to queue has no
    // landing: let the copy stream run out before the counter goes back
    if (cancel_replay && c->ctrl != nullptr && c->any_copy) (void)hipStreamSynchronize(c->xs);
    std::lock_guard<std::mutex> lk(c->mu);
    c->publish_released(c->released);
    if (c->ctrl != nullptr) __atomic_store_n(&c->ctrl->gate_timeout, 0u, __ATOMIC_RELEASE);
    c->cancel = false;
}

}  // namespace

extern "C" {

const char* gockpt_last_error(const gockpt_ctx* ctx) {
    return ctx != nullptr ? ctx->err.c_str() : g_create_error.c_str();
}

}  // extern "C"

// The device workspace of contexts made by gockpt_create_noalloc, one per
// GPU the library runs on, held until the process ends.  In host code this
// name is only a stand-in for the symbol: its device address on each GPU
// comes from hipGetSymbolAddress and is the only form passed to kernels or
// copies.
static __device__ __align__(256) uint8_t scratch[(kWsBytes + 255) / 256 * 256];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t* g_scratch_ptr[kMaxDevices];  // device address of `scratch` on each GPU (set once, with that GPU current)
bool g_scratch_busy[kMaxDevices];     // a live no-alloc context holds that GPU's scratch

// A context over the device workspace `ws`: the caller's (cfg->workspace)
// or the library's static scratch.  with_ctrl: allocate the control page (the
// only memory a context allocates; staged windows and skip-aware transfers
// need it).
int create_ctx(const gockpt_config* cfg, uint8_t* ws, bool with_ctrl, gockpt_ctx** out) {
    gockpt_ctx* c = new gockpt_ctx();
    c->cfg = *cfg;
    c->hp = HParams{cfg->beta1, cfg->beta2, cfg->eps, cfg->weight_decay};
    c->sc = ScalerCfg{cfg->check_overflow, cfg->dynamic_scale, cfg->growth_factor, cfg->backoff_factor,
                      cfg->min_scale, 0, cfg->growth_interval};
    c->konst = step_scalars(c->hp, 0.0f, 1, 1.0f);
    c->cs = static_cast<hipStream_t>(cfg->compute_stream);
    c->xs = static_cast<hipStream_t>(cfg->copy_stream);
    c->ws = ws;
    c->pre_blocks = prepass_blocks_for(cfg->n);
    c->knobs = default_knobs();
    // the fused kernel's block: kBlock unless asked for the 16-wavefront one
    // (a few tenths of a percent faster on a GPU running nothing else, but a
    // block that size cannot start on a compute unit another kernel partly
    // holds, so it slows down badly beside concurrent kernels)
    if (c->knobs.fused_block != kFusedWideBlock) c->knobs.fused_block = kBlock;
    if (const char* f = getenv("GOCKPT_TEST_FAIL_COPY")) c->fail_copy_at = atoll(f);
    auto env_on = [](const char* name) {
        const char* v = getenv(name);
        return v != nullptr && *v != '\0' && *v != '0';
    };
    c->dbg_poison = env_on("GOCKPT_DEBUG_POISON");
    c->dbg_checks = env_on("GOCKPT_DEBUG_CHECKS");
    c->roctx = env_on("GOCKPT_ROCTX");
    if (c->roctx) load_roctx();
    c->copy_bytes = cfg->copy_bytes ? cfg->copy_bytes : GOCKPT_DEFAULT_COPY_BYTES;

    hipError_t he = hipGetDevice(&c->device);
    hipEvent_t* evs[] = {&c->ev_kernel, &c->ev_last_copy, &c->ev_grad_spill, &c->ev_state_spill,
                         &c->ev_grads_copied, &c->ev_grads_ready, &c->ev_fin};
    for (hipEvent_t* ev : evs) {
        if (he != hipSuccess) break;
        he = hipEventCreateWithFlags(ev, hipEventDisableTiming);
        if (he == hipSuccess) c->all_events.push_back(*ev);
    }
    if (he == hipSuccess && with_ctrl) {
        // host-coherent, so the device's stores and the host's counter are
        // seen across PCIe without cache maintenance
        void* page = nullptr;
        he = hipHostMalloc(&page, 4096, hipHostMallocCoherent | hipHostMallocMapped);
        if (he == hipSuccess) {
            memset(page, 0, 4096);
            c->ctrl = static_cast<CtrlPage*>(page);
            void* dev = nullptr;
            he = hipHostGetDevicePointer(&dev, page, 0);
            c->ctrl_dev = static_cast<CtrlPage*>(dev);
        }
    }
    if (he == hipSuccess) {
        DevScaler init{};
        init.t = cfg->init_step;
        init.tracker = cfg->init_tracker;
        init.scale = cfg->init_scale;
        he = hipMemcpyAsync(c->ws + kWsScalerOff, &init, sizeof init, hipMemcpyHostToDevice, c->cs);
        if (he == hipSuccess) he = hipStreamSynchronize(c->cs);
    }
    if (he != hipSuccess) {
        g_create_error = std::string("gockpt_create: ") + hipGetErrorString(he);
        for (hipEvent_t ev : c->all_events) (void)hipEventDestroy(ev);
        if (c->ctrl != nullptr) (void)hipHostFree(c->ctrl);
        delete c;
        return GOCKPT_EHIP;
    }
    if (cfg->host_staging != nullptr) {
        c->staging = static_cast<uint8_t*>(cfg->host_staging);
        c->nslots = cfg->host_staging_bytes / c->copy_bytes;
        c->slot_done.assign(c->nslots, 0);
        const int nw = cfg->copy_threads > 0 ? cfg->copy_threads : 8;
        for (int i = 0; i < nw; ++i) c->workers.emplace_back(worker_loop, c);
    }
    *out = c;
    return GOCKPT_OK;
}

}  // namespace

extern "C" {

int gockpt_create(const gockpt_config* cfg, gockpt_ctx** out) {
    if (out == nullptr) {
        g_create_error = "out is NULL";
        return GOCKPT_EINVAL;
    }
    *out = nullptr;
    std::string e;
    int rc = check_config(cfg, e);
    if (rc != GOCKPT_OK) {
        g_create_error = e;
        return rc;
    }
    return create_ctx(cfg, static_cast<uint8_t*>(cfg->workspace), true, out);
}

int gockpt_create_noalloc(const gockpt_config* cfg, gockpt_ctx** out) {
    if (out == nullptr) {
        g_create_error = "out is NULL";
        return GOCKPT_EINVAL;
    }
    *out = nullptr;
    std::string e;
    int rc = check_config(cfg, e, true);
    if (rc != GOCKPT_OK) {
        g_create_error = e;
        return rc;
    }
    const size_t need = gockpt_workspace_bytes(cfg->n);
    if (need > sizeof(scratch)) {
        char buf[160];
        snprintf(buf, sizeof buf, "gockpt_create_noalloc: n = %lld needs a %zu-byte workspace, the static one holds %zu",
                 static_cast<long long>(cfg->n), need, sizeof(scratch));
        g_create_error = buf;
        return GOCKPT_ENOMEM;
    }
    int dev = 0;
    hipError_t he = hipGetDevice(&dev);
    if (he != hipSuccess) {
        g_create_error = std::string("gockpt_create_noalloc: ") + hipGetErrorString(he);
        return GOCKPT_EHIP;
    }
    if (dev < 0 || dev >= kMaxDevices) {
        g_create_error = "gockpt_create_noalloc: device index beyond the library's table";
        return GOCKPT_EINVAL;
    }
    uint8_t* ws = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_scratch_mu);
        if (g_scratch_ptr[dev] == nullptr) {
            // once per device, with that device current: each GPU holds its
            // own copy of the array at its own address
            void* p = nullptr;
            he = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (he != hipSuccess || p == nullptr) {
                g_create_error = std::string("gockpt_create_noalloc: hipGetSymbolAddress: ") +
                                 hipGetErrorString(he);
                return GOCKPT_EHIP;
            }
            g_scratch_ptr[dev] = static_cast<uint8_t*>(p);
        }
        if (g_scratch_busy[dev]) {
            g_create_error = "gockpt_create_noalloc: another no-alloc context lives on this device (they would share "
                             "its scratch workspace)";
            return GOCKPT_EBUSY;
        }
        g_scratch_busy[dev] = true;
        ws = g_scratch_ptr[dev];
    }
    rc = create_ctx(cfg, ws, false, out);
    if (rc != GOCKPT_OK) {
        std::lock_guard<std::mutex> lk(g_scratch_mu);
        g_scratch_busy[dev] = false;
        return rc;
    }
    (*out)->scratch_ws = true;
    return GOCKPT_OK;
}

int gockpt_destroy(gockpt_ctx* c) {
    if (c == nullptr) return GOCKPT_OK;
    int rc = GOCKPT_OK;
    if (c->restorer.joinable()) c->restorer.join();
    drop_deferred(c);
    quiesce(c, true);
    stop_threads(c);
    join_persist(c);
    if (c->any_copy && hipStreamSynchronize(c->xs) != hipSuccess) rc = GOCKPT_EHIP;
    if (hipStreamSynchronize(c->cs) != hipSuccess) rc = GOCKPT_EHIP;
    for (hipEvent_t ev : c->all_events) (void)hipEventDestroy(ev);
    if (c->ctrl != nullptr && hipHostFree(c->ctrl) != hipSuccess) rc = GOCKPT_EHIP;
    if (c->scratch_ws) {
        std::lock_guard<std::mutex> lk(g_scratch_mu);
        g_scratch_busy[c->device] = false;
    }
    delete c;
    return rc;
}

int gockpt_begin_window_ex(gockpt_ctx* c, int K, const int64_t* bounds, void* host_arena, size_t arena_bytes,
                           const gockpt_window_opts* opts) {
    if (c == nullptr) return GOCKPT_EINVAL;
    if (c->st == WinState::Restoring && finish_restore(c) != GOCKPT_OK) return GOCKPT_EFAILED;
    if (c->st == WinState::Failed) return c->fail(GOCKPT_EFAILED, "window failed earlier; call gockpt_abort_window");
    if (c->st != WinState::Idle) return c->fail(GOCKPT_EBUSY, "previous window not restored or aborted");
    join_persist(c);  // the previous checkpoint is written before the arena is reused
    if (!valid_bounds(K, bounds, c->cfg.n))
        return c->fail(GOCKPT_EINVAL, "bad window: K in 1..%d, bounds[0]=0, bounds[K]=n, increasing, x8",
                       GOCKPT_MAX_K);
    if (opts != nullptr && opts->reserved_[0] != 0)
        return c->fail(GOCKPT_EINVAL, "gockpt_window_opts.reserved_ must be 0");
    int R = opts ? opts->replay_every : 0;
    if (R < 0) return c->fail(GOCKPT_EINVAL, "replay_every < 0");
    if (R >= K) R = 0;
    const int policy = opts ? opts->wait_policy : GOCKPT_WAIT_LAZY;
    if (policy < GOCKPT_WAIT_LAZY || policy > GOCKPT_WAIT_ALL) return c->fail(GOCKPT_EINVAL, "unknown wait_policy");
    gockpt_arena_layout lay;
    std::vector<uint64_t> goff(K);
    arena_layout(K, bounds, c->cfg.n, R, &lay, goff.data());
    if (host_arena == nullptr || !aligned(host_arena, 256))
        return c->fail(GOCKPT_EINVAL, "host arena must be non-NULL and 256-byte aligned");
    if (arena_bytes < lay.total)
        return c->fail(GOCKPT_ENOMEM, "host arena has %zu bytes, window needs %llu", arena_bytes,
                       static_cast<unsigned long long>(lay.total));
    hipPointerAttribute_t attr;
    hipError_t pe = hipPointerGetAttributes(&attr, host_arena);
    const bool pinned = pe == hipSuccess && attr.type == hipMemoryTypeHost;
    if (pe != hipSuccess) (void)hipGetLastError();
    if (!pinned && c->cfg.host_staging == nullptr)
        return c->fail(GOCKPT_EINVAL, "host arena is not pinned and the context has no host staging");
    if (!pinned && c->ctrl == nullptr)
        return c->fail(GOCKPT_EINVAL, "a pageable host arena needs a context made by gockpt_create (control page)");
    const int plan = opts ? opts->late_plan : GOCKPT_RING_QUERY;
    if (plan < GOCKPT_RING_QUERY || plan > GOCKPT_RING_DEVICE_WAIT) return c->fail(GOCKPT_EINVAL, "unknown ring plan");
    if (!pinned && policy != GOCKPT_WAIT_LAZY)
        return c->fail(GOCKPT_EINVAL, "wait policies other than GOCKPT_WAIT_LAZY need a pinned host arena");
    const bool defer = opts != nullptr && opts->defer_copies != 0;
    if (defer && policy != GOCKPT_WAIT_LAZY)
        return c->fail(GOCKPT_EINVAL, "defer_copies needs GOCKPT_WAIT_LAZY (the other policies wait for the copies "
                       "at once)");
    c->K = K;
    c->s = 0;
    c->bounds.assign(bounds, bounds + K + 1);
    c->arena = static_cast<uint8_t*>(host_arena);
    c->arena_bytes = arena_bytes;
    c->lay = lay;
    c->goff = goff;
    c->staged = !pinned;
    c->R = R;
    c->wait_policy = policy;
    c->ring_off = opts != nullptr && opts->ring_off != 0;
    c->ring_plan = plan;
    c->ring_waited = 0;
    c->win_timing = c->cfg.timing != 0 && !(opts != nullptr && opts->no_timing != 0);
    c->defer = defer;
    c->deferred = StepCopies{};
    c->replay_threads = opts && opts->replay_threads > 0 ? opts->replay_threads : 8;
    c->head = 0;
    c->recycle_timing();
    c->records.clear();
    c->ring_grad_bytes.assign(K + 1, 0);
    c->step_ms.clear();
    memset(&c->stats, 0, sizeof c->stats);
    c->stats.K = K;
    {
        std::lock_guard<std::mutex> lk(c->mu);
        for (auto& r : c->inflight)
            if (r.ev) c->event_pool.push_back(r.ev);
        c->inflight.clear();
        for (hipEvent_t ev : c->step_done)
            if (ev) c->event_pool.push_back(ev);
        c->step_done.assign(K + 1, nullptr);
        c->pending.assign(K + 1, 0);
        c->issued.assign(K + 1, 0);
        c->issued_through = c->landed_through = c->replayed_through = 0;
        c->replay_updates = 0;
        c->cancel = false;
    }
    if (R > 0) c->replayer = std::thread(replayer_loop, c);
    c->ckpt_in_arena = false;
    c->st = WinState::Window;
    return GOCKPT_OK;
}

int gockpt_begin_window(gockpt_ctx* c, int K, const int64_t* bounds, void* host_arena, size_t arena_bytes) {
    return gockpt_begin_window_ex(c, K, bounds, host_arena, arena_bytes, nullptr);
}

}  // extern "C"

namespace {

// Queue one window step's copies on the copy stream (Sec. 4.2.2's order:
// gradients first).  c->ev_kernel (and c->ev_grads_ready when d says so)
// still mark that step's update (and gradients) on the compute stream: they
// are recorded again only by the next gockpt_step, which first queues any
// deferred copies.
int issue_copies(gockpt_ctx* c, StepCopies& d) {
    const int s = d.s;
    std::vector<Job>& jobs = d.jobs;
    StepTiming& tm = d.tm;
    const bool timed = d.timed;
    const int first_after_kernel = d.first_after_kernel;
    const int last_spill_g = d.last_spill_g, last_spill_s = d.last_spill_s, last_grad_job = d.last_grad_job;
    const bool grads_ready_ev = d.grads_ready_ev;
    gockpt_window_stats& stt = c->stats;
    hipError_t e;
    d.active = false;
    if (timed) {
        tm.cp0 = c->take_timing_event();
        tm.cp1 = c->take_timing_event();
        tm.has_copy = true;
        if (!tm.cp0 || !tm.cp1) return c->hip_fail(hipErrorOutOfMemory, "timing events");
    }
    // (the update leaves the gradient buffer as it was, so without the
    // gradients-ready event the update's event covers those copies too)
    if ((e = hipStreamWaitEvent(c->xs, first_after_kernel > 0 && grads_ready_ev ? c->ev_grads_ready : c->ev_kernel,
                                0)) != hipSuccess)
        return c->hip_fail(e, "copy wait");
    if (timed && (e = hipEventRecord(tm.cp0, c->xs)) != hipSuccess) return c->hip_fail(e, "event record");
    if (c->R > 0 && !c->staged) {
        // the gradient slot of this step in the pinned arena was last used by
        // step s - R: its replay must be done before the copies land there
        const int need = (s - 1) / c->R * c->R;
        std::unique_lock<std::mutex> lk(c->mu);
        c->cv.wait(lk, [&] { return c->thread_error || c->replayed_through >= need; });
        if (c->thread_error) {
            lk.unlock();
            return c->thread_fail();
        }
    }
    for (size_t k = 0; k < jobs.size(); ++k) {
        if (k > 0 && static_cast<int>(k) == first_after_kernel &&
            (e = hipStreamWaitEvent(c->xs, c->ev_kernel, 0)) != hipSuccess)
            return c->hip_fail(e, "copy wait");
        const Job& j = jobs[k];
        uint8_t* dst = c->arena + j.dst_off;
        uint64_t q = 0;
        if (c->staged) {
            // staging slot q mod nslots; its previous copy must be out of it
            q = c->seq;
            dst = c->staging + (q % c->nslots) * c->copy_bytes;
            if (q >= c->nslots && c->gate_through + c->nslots <= q) {
                const uint64_t rel = __atomic_load_n(&c->ctrl->released, __ATOMIC_ACQUIRE);
                if (rel + c->nslots > q && rel <= q) {
                    c->gate_through = rel;
                } else {
                    // open the gate for a batch of slots at once; every copy
                    // the target counts is queued before the gate
                    const uint64_t batch = c->nslots / 4 > 0 ? c->nslots / 4 : 1;
                    uint64_t target = q - c->nslots + batch;
                    if (target > q) target = q;
                    e = static_cast<hipError_t>(
                        launch_gate(&c->ctrl_dev->released, target, kGateTicks, &c->ctrl_dev->gate_timeout, c->xs));
                    if (e != hipSuccess) return c->hip_fail(e, "gate launch");
                    c->gate_through = target;
                    stt.n_gates++;
                }
            }
        }
        if (c->staged && c->dbg_checks && q >= c->nslots && c->gate_through + c->nslots <= q) {
            c->st = WinState::Failed;
            return c->fail(GOCKPT_EFAILED, "debug check: staged copy %llu reuses a slot no gate covers",
                           static_cast<unsigned long long>(q));
        }
        e = c->copy_d2h(dst, j.src, j.bytes);
        if (e != hipSuccess) return c->hip_fail(e, "copy");
        stt.n_copies++;
        if (j.from_ring && c->dbg_poison) {
            // the copy has its bytes: poison them before the range counts as free
            e = hipMemsetAsync(const_cast<uint8_t*>(j.src), 0xFF, j.bytes, c->xs);
            if (e != hipSuccess) return c->hip_fail(e, "poison");
        }
        if (c->staged) {
            hipEvent_t ev = c->take_event();
            if (ev == nullptr) return c->hip_fail(hipErrorOutOfMemory, "event create");
            if ((e = hipEventRecord(ev, c->xs)) != hipSuccess) return c->hip_fail(e, "event record");
            std::lock_guard<std::mutex> lk(c->mu);
            c->land_q.push_back({ev, dst, j.dst_off, j.bytes, q, s, j.grad});
            c->seq = q + 1;
            c->queued_seq = q + 1;
            c->pending[s]++;
            c->landings_open++;
            c->cv.notify_one();
        }
        if (j.ring) {
            hipEvent_t ev = c->take_event();
            if (ev == nullptr) return c->hip_fail(hipErrorOutOfMemory, "event create");
            if ((e = hipEventRecord(ev, c->xs)) != hipSuccess) return c->hip_fail(e, "event record");
            std::lock_guard<std::mutex> lk(c->mu);
            j.ring->ev = ev;
        }
        if (static_cast<int>(k) == last_spill_g && (e = hipEventRecord(c->ev_grad_spill, c->xs)) != hipSuccess)
            return c->hip_fail(e, "event record");
        if (static_cast<int>(k) == last_spill_s && (e = hipEventRecord(c->ev_state_spill, c->xs)) != hipSuccess)
            return c->hip_fail(e, "event record");
        if (static_cast<int>(k) == last_grad_job && c->wait_policy == GOCKPT_WAIT_GRADS &&
            (e = hipEventRecord(c->ev_grads_copied, c->xs)) != hipSuccess)
            return c->hip_fail(e, "event record");
    }
    if (timed && (e = hipEventRecord(tm.cp1, c->xs)) != hipSuccess) return c->hip_fail(e, "event record");
    if ((e = hipEventRecord(c->ev_last_copy, c->xs)) != hipSuccess) return c->hip_fail(e, "event record");
    // Explicit waits of the blocking schemes: the compute stream goes on
    // only once the step's gradients (or all of its copies) are on the host.
    if (c->wait_policy == GOCKPT_WAIT_GRADS && (e = hipStreamWaitEvent(c->cs, c->ev_grads_copied, 0)) != hipSuccess)
        return c->hip_fail(e, "wait for gradient copies");
    if (c->wait_policy == GOCKPT_WAIT_ALL && (e = hipStreamWaitEvent(c->cs, c->ev_last_copy, 0)) != hipSuccess)
        return c->hip_fail(e, "wait for the step's copies");
    hipEvent_t done_ev = c->take_event();
    if (done_ev == nullptr) return c->hip_fail(hipErrorOutOfMemory, "event create");
    if ((e = hipEventRecord(done_ev, c->xs)) != hipSuccess) return c->hip_fail(e, "event record");
    {
        std::lock_guard<std::mutex> lk(c->mu);
        c->step_done[s] = done_ev;
        c->issued[s] = 1;
        c->issued_through = s;
        c->advance_landed_locked();
        c->cv.notify_all();
    }
    c->any_copy = true;
    if (last_spill_g >= 0) {
        c->grad_spill_pending = true;
        c->backward_called = false;
    }
    if (last_spill_s >= 0) c->state_spill_pending = true;
    if (timed) c->timing.push_back(tm);
    return GOCKPT_OK;
}

// The copies a deferring window still holds, queued now.
int flush_deferred(gockpt_ctx* c) {
    if (!c->deferred.active) return GOCKPT_OK;
    StepCopies d = std::move(c->deferred);
    c->deferred = StepCopies{};
    return issue_copies(c, d);
}

// A window given up: its deferred copies are never queued (their timing
// events go back to the pool with the window's others).
void drop_deferred(gockpt_ctx* c) {
    if (c->deferred.active && c->deferred.timed) c->timing.push_back(c->deferred.tm);
    c->deferred = StepCopies{};
}

}  // namespace

extern "C" {

int gockpt_backward_begin(gockpt_ctx* c, void* stream) {
    if (c == nullptr) return GOCKPT_EINVAL;
    Range range(c->roctx, "gockpt_backward_begin");
    if (c->deferred.active) {
        const int rc = flush_deferred(c);
        if (rc != GOCKPT_OK) return rc;
    }
    if (c->grad_spill_pending) {
        hipStream_t s = stream ? static_cast<hipStream_t>(stream) : c->cs;
        hipError_t e = hipStreamWaitEvent(s, c->ev_grad_spill, 0);
        if (e != hipSuccess) return c->hip_fail(e, "gockpt_backward_begin");
        c->grad_spill_pending = false;
    }
    c->backward_called = true;
    return GOCKPT_OK;
}

int gockpt_scan_grads(gockpt_ctx* c, int64_t begin, int64_t end, void* stream) {
    if (c == nullptr) return GOCKPT_EINVAL;
    const int64_t n = c->cfg.n;
    if (!(0 <= begin && begin < end && end <= n) || begin % kVec != 0 || (end % kVec != 0 && end != n))
        return c->fail(GOCKPT_EINVAL, "scan range [%lld, %lld): need 0 <= begin < end <= n, both multiples of 8 "
                                      "(end may be n)", static_cast<long long>(begin), static_cast<long long>(end));
    // the ranges so far are disjoint: only the neighbours in begin order can overlap
    auto next = c->scan_ranges.lower_bound(begin);
    const std::pair<const int64_t, int64_t>* clash = nullptr;
    if (next != c->scan_ranges.end() && next->first < end) clash = &*next;
    if (clash == nullptr && next != c->scan_ranges.begin() && std::prev(next)->second > begin) clash = &*std::prev(next);
    if (clash != nullptr)
        return c->fail(GOCKPT_ESTATE, "scan range [%lld, %lld) overlaps [%lld, %lld) of this step",
                       static_cast<long long>(begin), static_cast<long long>(end),
                       static_cast<long long>(clash->first), static_cast<long long>(clash->second));
    hipStream_t st = stream ? static_cast<hipStream_t>(stream) : c->cs;
    // beside the backward a scan keeps to one block per compute unit; on the
    // compute stream it is on the step's critical path and takes the device
    int nb = scan_blocks_for(end - begin, st == c->cs ? kPrepassMaxBlocks : kScanMaxBlocks);
    if (nb > kScanSlots - c->scan_used) nb = kScanSlots - c->scan_used;
    if (nb < 1) return c->fail(GOCKPT_ESTATE, "more than %d scan blocks in one step", kScanSlots);
    uint8_t* parts = c->ws + kWsScanOff + (static_cast<size_t>(c->scan_bank) * kScanSlots + c->scan_used) *
                                              sizeof(Partial);
    hipError_t e = static_cast<hipError_t>(launch_scan(static_cast<const uint16_t*>(c->cfg.grad16), begin, end, parts,
                                                       nb, c->knobs.prepass_nt, c->cfg.grad_dtype, st));
    if (e != hipSuccess) return c->hip_fail(e, "scan launch");
    if (st != c->cs) {
        hipEvent_t ev = nullptr;
        for (const auto& se : c->scan_events)
            if (se.first == st) ev = se.second;
        if (ev == nullptr) {
            ev = c->take_event();
            if (ev == nullptr) return c->hip_fail(hipErrorOutOfMemory, "event create");
            c->scan_events.emplace_back(st, ev);
        }
        if ((e = hipEventRecord(ev, st)) != hipSuccess) return c->hip_fail(e, "event record");
    }
    c->scan_used += nb;
    c->scan_covered += end - begin;
    c->scan_ranges.emplace(begin, end);
    return GOCKPT_OK;
}

int gockpt_step(gockpt_ctx* c, float lr) {
    if (c == nullptr) return GOCKPT_EINVAL;
    if (!isfinite(lr)) return c->fail(GOCKPT_EINVAL, "lr is not finite");
    if (c->st == WinState::Failed) return c->fail(GOCKPT_EFAILED, "window failed earlier");
    if (c->has_thread_error()) return c->thread_fail();
    if (c->deferred.active) {
        // before anything of this step is queued: the previous step's events
        // are recorded again below
        const int rc = flush_deferred(c);
        if (rc != GOCKPT_OK) return rc;
    }
    if (c->grad_spill_pending && !c->backward_called)
        return c->fail(GOCKPT_ESTATE,
                       "gradients of the previous step are still being copied from the gradient buffer; "
                       "call gockpt_backward_begin before writing new gradients");
    if (!c->scan_ranges.empty() && c->scan_covered != c->cfg.n)
        return c->fail(GOCKPT_ESTATE, "the bucket scans of this step cover %lld of %lld elements",
                       static_cast<long long>(c->scan_covered), static_cast<long long>(c->cfg.n));
    const gockpt_config& cfg = c->cfg;
    const int64_t n = cfg.n;
    const bool in_window = c->st == WinState::Window;
    const int s = in_window ? c->s + 1 : 0;
    hipError_t e;
    Range range(c->roctx, "gockpt_step %d/%d", s, in_window ? c->K : 0);

    const uint64_t R = cfg.ring && !c->ring_off ? cfg.ring_bytes : 0;

    // The gradients are complete here in stream order: copies that take them
    // straight from the gradient buffer may start now, ahead of the update
    // (the gradient transfer overlaps the update and the next forward pass,
    // Sec. 4.2.4).  The event marking this point is recorded only when the
    // step may send gradients that way: under DEVICE_WAIT the gradients come
    // first in the ring and all of them fit whenever 2 * b_{s-1} bytes do.
    const int64_t gb0 = in_window ? c->bounds[s - 1] : 0;
    const bool grads_ready_ev =
        in_window && gb0 > 0 &&
        !(c->ring_plan == GOCKPT_RING_DEVICE_WAIT && R && round_up(static_cast<uint64_t>(gb0) * 2, 256) <= R);
    if (grads_ready_ev && (e = hipEventRecord(c->ev_grads_ready, c->cs)) != hipSuccess)
        return c->hip_fail(e, "event record");

    // The previous step's state copies straight from the live buffers must
    // finish before this update overwrites them.  Queued before any kernel of
    // this step, so a failure here leaves the step entirely undone (the
    // finalize would otherwise have advanced the step count for an update
    // that never ran).
    if (c->state_spill_pending) {
        if ((e = hipStreamWaitEvent(c->cs, c->ev_state_spill, 0)) != hipSuccess)
            return c->hip_fail(e, "wait for state copies");
        c->state_spill_pending = false;
    }

    StepTiming tm{};
    const bool timed = c->win_timing && in_window;
    if (timed) {
        tm.pre0 = c->take_timing_event();
        tm.pre1 = c->take_timing_event();
        tm.upd0 = c->take_timing_event();
        tm.upd1 = c->take_timing_event();
        if (!tm.pre0 || !tm.pre1 || !tm.upd0 || !tm.upd1) return c->hip_fail(hipErrorOutOfMemory, "timing events");
        if ((e = hipEventRecord(tm.pre0, c->cs)) != hipSuccess) return c->hip_fail(e, "event record");
    }
    // The prepass reads the gradients for the overflow test and the norm; with
    // neither wanted (or the test done by the caller, or the buckets already
    // scanned) nothing reads them before the update.
    FinalizeArgs fin{};
    fin.found_inf = cfg.check_overflow != 0 ? cfg.found_inf : nullptr;
    fin.norm_off = cfg.grad_norm_off;
    fin.slot = s;
    fin.window_step = s;
    fin.lr = lr;
    fin.hp = c->hp;
    fin.sc = c->sc;
    fin.skip_out = in_window && c->ctrl_dev != nullptr ? &c->ctrl_dev->skip[s] : nullptr;
    const bool scanned = !c->scan_ranges.empty();
    const bool prepass =
        !scanned && n > 0 && ((cfg.check_overflow != 0 && fin.found_inf == nullptr) || cfg.grad_norm_off == 0);
    if (prepass) {
        e = static_cast<hipError_t>(
            launch_prepass(cfg.grad16, n, c->ws, c->pre_blocks, c->knobs.prepass_nt, cfg.grad_dtype, c->cs));
        if (e != hipSuccess) return c->hip_fail(e, "prepass launch");
    }
    for (const auto& se : c->scan_events)
        if ((e = hipStreamWaitEvent(c->cs, se.second, 0)) != hipSuccess)
            return c->hip_fail(e, "wait for the bucket scans");
    const uint8_t* parts = c->ws + (scanned ? kWsScanOff + static_cast<size_t>(c->scan_bank) * kScanSlots *
                                                               sizeof(Partial)
                                            : kWsPartialsOff);
    fin.raw = scanned ? 1 : 0;
    e = static_cast<hipError_t>(
        launch_finalize(c->ws, parts, scanned ? c->scan_used : (prepass ? c->pre_blocks : 0), fin, c->cs));
    if (e != hipSuccess) return c->hip_fail(e, "finalize launch");
    if (scanned) {  // the next step's scans fill the other bank
        std::lock_guard<std::mutex> lk(c->mu);
        for (const auto& se : c->scan_events) c->event_pool.push_back(se.second);
        c->scan_events.clear();
        c->scan_ranges.clear();
        c->scan_used = 0;
        c->scan_covered = 0;
        c->scan_bank ^= 1;
    }
    if (timed && (e = hipEventRecord(tm.pre1, c->cs)) != hipSuccess) return c->hip_fail(e, "event record");

    // With HOST_WAIT the calling thread waits for the finalize: the ring
    // space freed meanwhile is then used instead of spilling, and the step's
    // skip decision is known (a skipped step's gradients are never replayed,
    // so then none are sent).
    bool skipped = false;
    if (in_window && c->ring_plan == GOCKPT_RING_HOST_WAIT && R) {
        if ((e = hipEventRecord(c->ev_fin, c->cs)) != hipSuccess) return c->hip_fail(e, "event record");
        if ((e = hipEventSynchronize(c->ev_fin)) != hipSuccess) return c->hip_fail(e, "wait for the device");
        if (c->ctrl != nullptr) skipped = __atomic_load_n(&c->ctrl->skip[s], __ATOMIC_ACQUIRE) != 0;
    }

    // Pack plan of this step.
    FusedArgs a{};
    a.p = cfg.master;
    a.m = cfg.exp_avg;
    a.v = cfg.exp_avg_sq;
    a.w = cfg.weight_bf16;
    a.g = cfg.grad16;
    a.grad_kind = cfg.grad_dtype;
    a.n = n;
    a.rec = reinterpret_cast<const gockpt_step_record*>(c->ws + kWsRecordsOff) + s;
    a.b1 = c->konst.b1;
    a.b2 = c->konst.b2;
    a.omb1 = c->konst.omb1;
    a.omb2 = c->konst.omb2;
    a.eps = c->konst.eps;
    a.quads_per_thread = c->knobs.quads_per_thread;
    a.nt = c->knobs.fused_nt;
    a.block = c->knobs.fused_block;
    PackPlan& pk = a.pack;
    pk.ring_nt = c->knobs.ring_nt;
    pk.g_end = 0;
    pk.cb = n;
    pk.s_end[0] = pk.s_end[1] = pk.s_end[2] = n;
    pk.ring = static_cast<uint8_t*>(cfg.ring);
    pk.ring_bytes = cfg.ring_bytes ? cfg.ring_bytes : 1;

    // Segment k: 0 = grads [0, b0) (none when the step is known skipped),
    // 1..3 = master/m/v of [b0, b1).
    int64_t seg_beg[4] = {0, 0, 0, 0}, seg_end[4] = {0, 0, 0, 0}, ring_end[4] = {0, 0, 0, 0};
    uint64_t seg_lstart[4] = {0, 0, 0, 0};
    if (in_window) {
        const int64_t b0 = c->bounds[s - 1], b1 = c->bounds[s];
        seg_beg[0] = 0;
        seg_end[0] = skipped ? 0 : b0;
        for (int k = 1; k < 4; ++k) {
            seg_beg[k] = b0;
            seg_end[k] = b1;
        }
        const uint64_t drained = c->reclaim();
        int64_t avail = 0;
        if (R) avail = c->ring_plan == GOCKPT_RING_DEVICE_WAIT ? static_cast<int64_t>(R)
                                                               : static_cast<int64_t>(R) - static_cast<int64_t>(c->head - drained);
        if (avail < 0) avail = 0;
        const uint64_t head0 = c->head;
        uint64_t lpos = head0;
        bool full = false;
        for (int k = 0; k < 4; ++k) {
            const uint64_t esz = k == 0 ? 2 : 4;
            const int64_t len = seg_end[k] - seg_beg[k];
            const uint64_t need = round_up(static_cast<uint64_t>(len) * esz, 256);
            seg_lstart[k] = lpos;
            if (!full && static_cast<int64_t>(need) <= avail) {
                ring_end[k] = seg_end[k];
                avail -= static_cast<int64_t>(need);
                lpos += need;
            } else {
                // Largest multiple of 8 elements that fits; the rest spills.
                int64_t fit = full ? 0 : avail / static_cast<int64_t>(esz * kVec) * kVec;
                if (fit > len) fit = len;
                ring_end[k] = seg_beg[k] + fit;
                lpos += static_cast<uint64_t>(fit) * esz;
                avail = 0;
                full = true;
            }
        }
        pk.g_end = ring_end[0];
        pk.cb = b0;
        for (int k = 0; k < 3; ++k) pk.s_end[k] = ring_end[k + 1];
        if (R) {
            pk.off_g = seg_lstart[0] % R;
            for (int k = 0; k < 3; ++k) pk.off_s[k] = seg_lstart[k + 1] % R;
        }
        c->head = round_up(lpos, 256);
        // DEVICE_WAIT: the step overwrites the physical bytes of logical
        // offsets [head0 - R, head - R).  Copies are queued in logical order,
        // so waiting for the last in-flight copy that starts below head - R
        // covers all of them.
        if (c->ring_plan == GOCKPT_RING_DEVICE_WAIT && R && c->head > R && c->head - R > c->ring_waited) {
            const uint64_t reuse_end = c->head - R;
            hipEvent_t wait_ev = nullptr;
            uint64_t wait_end = 0;
            bool unqueued = false;
            {
                std::lock_guard<std::mutex> lk(c->mu);
                for (const RingCopy& rc : c->inflight) {
                    if (rc.lbeg >= reuse_end) break;
                    wait_ev = rc.ev;
                    wait_end = rc.lend;
                    unqueued = rc.ev == nullptr;
                }
            }
            if (unqueued) return c->fail(GOCKPT_EFAILED, "ring range reused before its copy was queued");
            if (wait_ev != nullptr && wait_end > c->ring_waited) {
                if ((e = hipStreamWaitEvent(c->cs, wait_ev, 0)) != hipSuccess) return c->hip_fail(e, "ring wait");
                c->ring_waited = wait_end;
            }
        }
    }

    if (in_window && c->dbg_checks && R) {
        // every earlier copy of the ring bytes this step overwrites has
        // finished (QUERY, HOST_WAIT) or is waited for on the device before
        // the update (DEVICE_WAIT); earlier copies are in logical order
        const uint64_t reuse_end = c->head > R ? c->head - R : 0;
        std::lock_guard<std::mutex> lk(c->mu);
        uint64_t prev = 0;
        for (const RingCopy& rc : c->inflight) {
            if (rc.lbeg < prev)
                return c->fail(GOCKPT_EFAILED, "debug check: ring copies out of logical order at step %d", s);
            prev = rc.lbeg;
            if (rc.lbeg >= reuse_end) break;
            const bool waited = c->ring_plan == GOCKPT_RING_DEVICE_WAIT && rc.lend <= c->ring_waited;
            const bool done = rc.ev != nullptr && hipEventQuery(rc.ev) == hipSuccess;
            if (!waited && !done) {
                (void)hipGetLastError();
                c->st = WinState::Failed;
                return c->fail(GOCKPT_EFAILED, "debug check: step %d overwrites ring bytes [%llu, %llu) whose copy "
                               "has neither finished nor been waited for", s,
                               static_cast<unsigned long long>(rc.lbeg), static_cast<unsigned long long>(rc.lend));
            }
        }
    }
    if (timed && (e = hipEventRecord(tm.upd0, c->cs)) != hipSuccess) return c->hip_fail(e, "event record");
    if (n > 0) {
        if ((e = static_cast<hipError_t>(launch_fused(a, c->cs))) != hipSuccess) return c->hip_fail(e, "fused launch");
    }
    if (timed && (e = hipEventRecord(tm.upd1, c->cs)) != hipSuccess) return c->hip_fail(e, "event record");
    if (!in_window) return GOCKPT_OK;

    // ---- the step's copies, as a job list in copy order ----
    gockpt_window_stats& stt = c->stats;
    std::vector<Job> jobs;
    const uint64_t dst_base[4] = {c->goff[s - 1], c->lay.master, c->lay.exp_avg, c->lay.exp_avg_sq};
    const uint8_t* live[4] = {reinterpret_cast<const uint8_t*>(cfg.grad16),
                              reinterpret_cast<const uint8_t*>(cfg.master),
                              reinterpret_cast<const uint8_t*>(cfg.exp_avg),
                              reinterpret_cast<const uint8_t*>(cfg.exp_avg_sq)};
    // Copy order: the gradients that did not fit the ring, straight from the
    // gradient buffer (these need only the gradients, not the update); then,
    // after the update, the step record, the ring's gradients, the ring's
    // state and the rest of the state from the live buffers.  Gradients go
    // first (Sec. 4.2.2).  Ring ranges are registered now, before the copies
    // are queued.
    int last_spill_g = -1, last_spill_s = -1;
    auto emit_ring = [&](int k) {
        const uint64_t esz = k == 0 ? 2 : 4;
        const int64_t len = ring_end[k] - seg_beg[k];
        if (len <= 0) return;
        const uint64_t bytes = static_cast<uint64_t>(len) * esz;
        const uint64_t dst = dst_base[k] + static_cast<uint64_t>(seg_beg[k]) * esz;
        // one bookkeeping entry per segment, its event recorded after the
        // segment's last copy: copies run in order, so that event covers the
        // whole segment (one event per segment, not per copy)
        RingCopy* rcp;
        {
            std::lock_guard<std::mutex> lk(c->mu);
            c->inflight.push_back({seg_lstart[k], seg_lstart[k] + bytes, nullptr});
            rcp = &c->inflight.back();
        }
        uint64_t lcur = seg_lstart[k], done = 0;
        while (done < bytes) {
            const uint64_t phys = lcur % R;
            uint64_t len_b = bytes - done;
            if (len_b > R - phys) len_b = R - phys;  // stop at the ring's end
            if (len_b > c->copy_bytes) len_b = c->copy_bytes;
            jobs.push_back({static_cast<uint8_t*>(cfg.ring) + phys, dst + done, len_b,
                            done + len_b == bytes ? rcp : nullptr, k == 0, true});
            done += len_b;
            lcur += len_b;
        }
        stt.bytes_ring += bytes;
        stt.bytes_d2h += bytes;
        tm.ring_bytes += bytes;
        if (k == 0) {
            tm.ring_grad_bytes += bytes;
            c->ring_grad_bytes[s] += bytes;
        }
    };
    auto emit_spill = [&](int k) {
        const uint64_t esz = k == 0 ? 2 : 4;
        const int64_t len = seg_end[k] - ring_end[k];
        if (len <= 0) return;
        const uint64_t bytes = static_cast<uint64_t>(len) * esz;
        const uint64_t first = static_cast<uint64_t>(ring_end[k]) * esz;
        for (uint64_t done = 0; done < bytes;) {
            const uint64_t len_b = bytes - done < c->copy_bytes ? bytes - done : c->copy_bytes;
            jobs.push_back({live[k] + first + done, dst_base[k] + first + done, len_b, nullptr, k == 0, false});
            done += len_b;
        }
        (k == 0 ? last_spill_g : last_spill_s) = static_cast<int>(jobs.size()) - 1;
        stt.bytes_spilled += bytes;
        stt.bytes_d2h += bytes;
    };
    emit_spill(0);
    const int first_after_kernel = static_cast<int>(jobs.size());
    jobs.push_back({c->ws + kWsRecordsOff + static_cast<uint64_t>(s) * sizeof(gockpt_step_record),
                    c->lay.records + static_cast<uint64_t>(s - 1) * sizeof(gockpt_step_record),
                    sizeof(gockpt_step_record), nullptr, false, false});
    emit_ring(0);
    const int last_grad_job = static_cast<int>(jobs.size()) - 1;  // the record when the ring holds no gradients
    for (int k = 1; k < 4; ++k) emit_ring(k);
    for (int k = 1; k < 4; ++k) emit_spill(k);

    if ((e = hipEventRecord(c->ev_kernel, c->cs)) != hipSuccess) return c->hip_fail(e, "event record");
    StepCopies d;
    d.active = true;
    d.s = s;
    d.jobs = std::move(jobs);
    d.tm = tm;
    d.timed = timed;
    d.first_after_kernel = first_after_kernel;
    d.last_spill_g = last_spill_g;
    d.last_spill_s = last_spill_s;
    d.last_grad_job = last_grad_job;
    d.grads_ready_ev = grads_ready_ev;
    stt.steps_done = s;
    c->s = s;
    if (s == c->K) c->st = WinState::Draining;
    if (c->defer) {
        // queued at the next call into the library, by when the device has
        // usually finished this update: copies queued early wait on the copy
        // engine for the update, which slows the dispatch of short kernels
        c->deferred = std::move(d);
        return GOCKPT_OK;
    }
    return issue_copies(c, d);
}

int gockpt_drain(gockpt_ctx* c, int blocking, gockpt_window_stats* stats) {
    if (c == nullptr) return GOCKPT_EINVAL;
    Range range(c->roctx, "gockpt_drain %s", blocking ? "blocking" : "poll");
    if (c->st == WinState::Failed) return c->fail(GOCKPT_EFAILED, "window failed earlier");
    if (c->deferred.active) {
        const int rc = flush_deferred(c);
        if (rc != GOCKPT_OK) return rc;
    }
    if (c->st == WinState::Drained) {
        if (stats) *stats = c->stats;
        return GOCKPT_OK;
    }
    if (c->st != WinState::Draining) return c->fail(GOCKPT_ESTATE, "drain needs all K window steps issued");
    const auto t0 = std::chrono::steady_clock::now();
    hipError_t e;
    const int K = c->K;
    if (!blocking) {
        std::lock_guard<std::mutex> lk(c->mu);
        if (!c->thread_error && ((c->staged && c->landed_through < K) || (c->R > 0 && c->replayed_through < K)))
            return GOCKPT_EAGAIN;
    }
    if (!c->staged) {
        if (blocking) {
            e = hipEventSynchronize(c->ev_last_copy);
            if (e != hipSuccess) return c->hip_fail(e, "drain wait");
        } else {
            e = hipEventQuery(c->ev_last_copy);
            if (e == hipErrorNotReady) return GOCKPT_EAGAIN;
            if (e != hipSuccess) return c->hip_fail(e, "drain query");
        }
    }
    {
        std::unique_lock<std::mutex> lk(c->mu);
        c->cv.wait(lk, [&] {
            return c->thread_error ||
                   ((!c->staged || c->landed_through >= K) && (c->R == 0 || c->replayed_through >= K));
        });
    }
    if (c->has_thread_error()) return c->thread_fail();
    if (c->replayer.joinable()) c->replayer.join();
    c->stats.wait_ms += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    c->reclaim();
    const gockpt_step_record* rec = reinterpret_cast<const gockpt_step_record*>(c->arena + c->lay.records);
    c->records.assign(rec, rec + K);
    int skipped = 0;
    for (int s = 1; s <= K; ++s) {
        if (c->records[s - 1].window_step != s) {
            c->st = WinState::Failed;
            return c->fail(GOCKPT_EFAILED, "record of window step %d is missing", s);
        }
        if (c->records[s - 1].skip) {
            ++skipped;
            c->stats.bytes_ring -= c->ring_grad_bytes[s];  // the kernel packed none of them
        }
    }
    c->stats.skipped = skipped;
    c->step_ms.clear();
    for (size_t i = 0; i < c->timing.size(); ++i) {
        const StepTiming& t = c->timing[i];
        float a = 0.0f, b = 0.0f, d = 0.0f, g = 0.0f;
        if (hipEventElapsedTime(&a, t.pre0, t.pre1) != hipSuccess) a = 0.0f;
        if (hipEventElapsedTime(&b, t.upd0, t.upd1) != hipSuccess) b = 0.0f;
        if (hipEventElapsedTime(&g, t.pre1, t.upd0) != hipSuccess) g = 0.0f;
        if (!t.has_copy || hipEventElapsedTime(&d, t.cp0, t.cp1) != hipSuccess) d = 0.0f;
        (void)hipGetLastError();
        c->stats.prepass_ms += a;
        c->stats.update_ms += b;
        c->stats.copy_ms += d;
        c->step_ms.push_back(a);
        c->step_ms.push_back(b);
        c->step_ms.push_back(d);
        // a skipped step packs no gradients (the fused kernel leaves them out)
        const bool skip = i < c->records.size() && c->records[i].skip != 0;
        c->step_ms.push_back(static_cast<double>(skip ? t.ring_bytes - t.ring_grad_bytes : t.ring_bytes));
        c->step_ms.push_back(g);
    }
    c->recycle_timing();
    // every copy of the window has completed: later steps need not wait for
    // copies from the live buffers (and a plain step queues no cross-stream
    // wait, so it can be captured)
    c->grad_spill_pending = c->state_spill_pending = false;
    c->backward_called = true;
    c->st = WinState::Drained;
    if (stats) *stats = c->stats;
    return GOCKPT_OK;
}

int gockpt_restore(gockpt_ctx* c, float* master_out, float* exp_avg_out, float* exp_avg_sq_out,
                   uint16_t* w_bf16_out, gockpt_ckpt_meta* meta, int nthreads) {
    if (c == nullptr) return GOCKPT_EINVAL;
    Range range(c->roctx, "gockpt_restore");
    if (c->st == WinState::Failed) return c->fail(GOCKPT_EFAILED, "window failed earlier");
    if (c->st != WinState::Drained) return c->fail(GOCKPT_ESTATE, "restore needs a drained window");
    std::string err;
    gockpt_ckpt_meta m{};
    int rc = run_restore(c, master_out, exp_avg_out, exp_avg_sq_out, w_bf16_out, nthreads, &m, err);
    if (rc != GOCKPT_OK) {
        c->st = WinState::Failed;
        return c->fail(rc, "%s", err.c_str());
    }
    if (meta != nullptr) *meta = m;
    c->last_meta = m;
    c->ckpt_in_arena = master_out == nullptr && exp_avg_out == nullptr && exp_avg_sq_out == nullptr;
    c->st = WinState::Idle;
    return GOCKPT_OK;
}

int gockpt_restore_async(gockpt_ctx* c, float* master_out, float* exp_avg_out, float* exp_avg_sq_out,
                         uint16_t* w_bf16_out, int nthreads) {
    if (c == nullptr) return GOCKPT_EINVAL;
    if (c->st == WinState::Failed) return c->fail(GOCKPT_EFAILED, "window failed earlier");
    if (c->st != WinState::Drained) return c->fail(GOCKPT_ESTATE, "restore needs a drained window");
    c->restore_rc = GOCKPT_OK;
    c->restore_err.clear();
    c->restore_meta = gockpt_ckpt_meta{};
    c->restore_in_place = master_out == nullptr && exp_avg_out == nullptr && exp_avg_sq_out == nullptr;
    c->st = WinState::Restoring;
    c->restorer = std::thread([c, master_out, exp_avg_out, exp_avg_sq_out, w_bf16_out, nthreads]() {
        std::string err;
        gockpt_ckpt_meta m{};
        const int rc = run_restore(c, master_out, exp_avg_out, exp_avg_sq_out, w_bf16_out, nthreads, &m, err);
        c->restore_rc = rc;
        c->restore_err = err;
        c->restore_meta = m;
    });
    return GOCKPT_OK;
}

int gockpt_restore_wait(gockpt_ctx* c, gockpt_ckpt_meta* meta) {
    if (c == nullptr) return GOCKPT_EINVAL;
    if (c->st != WinState::Restoring || !c->restorer.joinable())
        return c->fail(GOCKPT_ESTATE, "no restore running");
    const int rc = finish_restore(c);
    if (rc != GOCKPT_OK) return rc;
    if (meta != nullptr) *meta = c->last_meta;
    return GOCKPT_OK;
}

int gockpt_abort_window(gockpt_ctx* c) {
    if (c == nullptr) return GOCKPT_EINVAL;
    if (c->restorer.joinable()) c->restorer.join();  // its result is discarded with the window
    int rc = GOCKPT_OK;
    c->ckpt_in_arena = false;
    drop_deferred(c);
    quiesce(c, true);
    if (c->any_copy) {
        // every copy queued so far, including those of a step whose later
        // copies failed to queue (the last-copy event may predate them)
        hipError_t e = hipStreamSynchronize(c->xs);
        if (e != hipSuccess) rc = c->fail(GOCKPT_EHIP, "abort wait: %s", hipGetErrorString(e));
    }
    if (rc == GOCKPT_OK) {
        // every copy from the live buffers has finished
        c->grad_spill_pending = c->state_spill_pending = false;
        c->backward_called = true;
    }
    {
        std::lock_guard<std::mutex> lk(c->mu);
        for (auto& r : c->inflight)
            if (r.ev) c->event_pool.push_back(r.ev);
        c->inflight.clear();
        c->thread_error = false;
        c->thread_err.clear();
    }
    c->recycle_timing();
    c->head = 0;
    c->K = 0;
    c->s = 0;
    c->st = WinState::Idle;
    return rc;
}

int gockpt_persist(gockpt_ctx* c, const char* dir, const char* user_meta, int nthreads, int async) {
    if (c == nullptr || dir == nullptr) return GOCKPT_EINVAL;
    join_persist(c);
    if (c->st == WinState::Restoring && finish_restore(c) != GOCKPT_OK) return GOCKPT_EFAILED;
    if (c->st != WinState::Idle || !c->ckpt_in_arena)
        return c->fail(GOCKPT_ESTATE, "persist needs the checkpoint of an in-place gockpt_restore");
    gockpt_ckpt_info info{};
    info.n = c->cfg.n;
    info.t = c->last_meta.t;
    info.tracker = c->last_meta.tracker;
    info.scale = c->last_meta.scale;
    info.K = c->last_meta.K;
    info.skipped = c->last_meta.skipped;
    info.beta1 = c->cfg.beta1;
    info.beta2 = c->cfg.beta2;
    info.eps = c->cfg.eps;
    info.weight_decay = c->cfg.weight_decay;
    const float* p = reinterpret_cast<const float*>(c->arena + c->lay.master);
    const float* m = reinterpret_cast<const float*>(c->arena + c->lay.exp_avg);
    const float* v = reinterpret_cast<const float*>(c->arena + c->lay.exp_avg_sq);
    std::string d(dir), u(user_meta ? user_meta : "");
    const bool has_user = user_meta != nullptr;
    auto job = [c, p, m, v, info, d, u, has_user, nthreads]() {
        gockpt_io_stats st{};
        const int rc = gockpt_write_checkpoint(d.c_str(), p, m, v, &info, has_user ? u.c_str() : nullptr, nthreads,
                                               &st);
        c->persist_rc = rc;
        c->persist_err = rc == GOCKPT_OK ? "" : gockpt_last_error(nullptr);
        c->persist_stats = st;
    };
    c->persist_rc = GOCKPT_OK;
    c->persist_err.clear();
    if (async) {
        c->persister = std::thread(job);
        return GOCKPT_OK;
    }
    job();
    if (c->persist_rc != GOCKPT_OK) return c->fail(c->persist_rc, "%s", c->persist_err.c_str());
    return GOCKPT_OK;
}

int gockpt_persist_wait(gockpt_ctx* c, gockpt_io_stats* stats) {
    if (c == nullptr) return GOCKPT_EINVAL;
    join_persist(c);
    if (stats != nullptr) *stats = c->persist_stats;
    if (c->persist_rc != GOCKPT_OK) return c->fail(c->persist_rc, "%s", c->persist_err.c_str());
    return GOCKPT_OK;
}

int gockpt_load(gockpt_ctx* c, const char* dir, void* host_buf, size_t host_bytes, int nthreads,
                gockpt_ckpt_info* info_out) {
    if (c == nullptr || dir == nullptr) return GOCKPT_EINVAL;
    if (c->st == WinState::Restoring && finish_restore(c) != GOCKPT_OK) return GOCKPT_EFAILED;
    if (c->st != WinState::Idle) return c->fail(GOCKPT_ESTATE, "load needs an idle context (no window)");
    join_persist(c);
    const int64_t n = c->cfg.n;
    gockpt_ckpt_info info{};
    int rc = gockpt_read_checkpoint_info(dir, &info);
    if (rc != GOCKPT_OK) return c->fail(rc, "%s", gockpt_last_error(nullptr));
    if (info.n != n) return c->fail(GOCKPT_EINVAL, "checkpoint holds %lld elements, context has %lld",
                                    static_cast<long long>(info.n), static_cast<long long>(n));
    if (info.beta1 != c->cfg.beta1 || info.beta2 != c->cfg.beta2 || info.eps != c->cfg.eps ||
        info.weight_decay != c->cfg.weight_decay)
        return c->fail(GOCKPT_EINVAL, "checkpoint hyperparameters differ from the context's");
    if (host_buf == nullptr || host_bytes < 12ull * static_cast<uint64_t>(n))
        return c->fail(GOCKPT_EINVAL, "host_buf must hold 12 n bytes");
    float* hp = static_cast<float*>(host_buf);
    rc = gockpt_read_checkpoint(dir, n, hp, hp + n, hp + 2 * n, &info, nthreads, nullptr);
    if (rc != GOCKPT_OK) return c->fail(rc, "%s", gockpt_last_error(nullptr));
    const gockpt_config& cfg = c->cfg;
    hipError_t e = hipSuccess;
    const size_t bytes = 4ull * static_cast<uint64_t>(n);
    if (n > 0) {
        e = hipMemcpyAsync(cfg.master, hp, bytes, hipMemcpyHostToDevice, c->cs);
        if (e == hipSuccess) e = hipMemcpyAsync(cfg.exp_avg, hp + n, bytes, hipMemcpyHostToDevice, c->cs);
        if (e == hipSuccess) e = hipMemcpyAsync(cfg.exp_avg_sq, hp + 2 * n, bytes, hipMemcpyHostToDevice, c->cs);
        if (e == hipSuccess && cfg.weight_bf16 != nullptr)
            e = static_cast<hipError_t>(launch_cast_bf16(static_cast<const float*>(cfg.master),
                                                         static_cast<uint16_t*>(cfg.weight_bf16), n, c->cs));
    }
    DevScaler sc{};
    sc.t = info.t;
    sc.tracker = info.tracker;
    sc.scale = info.scale;
    if (e == hipSuccess) e = hipMemcpyAsync(c->ws + kWsScalerOff, &sc, sizeof sc, hipMemcpyHostToDevice, c->cs);
    if (e == hipSuccess) e = hipStreamSynchronize(c->cs);
    if (e != hipSuccess) return c->fail(GOCKPT_EHIP, "load: %s", hipGetErrorString(e));
    c->ckpt_in_arena = false;
    if (info_out != nullptr) *info_out = info;
    return GOCKPT_OK;
}

int gockpt_get_scaler(gockpt_ctx* c, int64_t* t, float* scale, int64_t* tracker) {
    if (c == nullptr) return GOCKPT_EINVAL;
    DevScaler h{};
    hipError_t e = hipMemcpyAsync(&h, c->ws + kWsScalerOff, sizeof h, hipMemcpyDeviceToHost, c->cs);
    if (e == hipSuccess) e = hipStreamSynchronize(c->cs);
    if (e != hipSuccess) return c->hip_fail(e, "gockpt_get_scaler");
    if (t) *t = h.t;
    if (scale) *scale = h.scale;
    if (tracker) *tracker = h.tracker;
    return GOCKPT_OK;
}

int gockpt_window_records(gockpt_ctx* c, gockpt_step_record* out, int capacity) {
    if (c == nullptr || out == nullptr) return GOCKPT_EINVAL;
    if (c->st != WinState::Drained && c->st != WinState::Restoring && !(c->st == WinState::Idle && !c->records.empty()))
        return c->fail(GOCKPT_ESTATE, "records are available after drain");
    if (capacity < static_cast<int>(c->records.size())) return c->fail(GOCKPT_ENOMEM, "capacity < K");
    memcpy(out, c->records.data(), c->records.size() * sizeof(gockpt_step_record));
    return GOCKPT_OK;
}

int gockpt_window_step_times(gockpt_ctx* c, double* out, int capacity) {
    if (c == nullptr || out == nullptr) return GOCKPT_EINVAL;
    if (c->st != WinState::Drained && c->st != WinState::Idle && c->st != WinState::Restoring)
        return c->fail(GOCKPT_ESTATE, "times follow drain");
    if (c->step_ms.empty())
        return c->fail(GOCKPT_ESTATE, "no step times: create with timing = 1, do not opt the window out, and drain");
    const size_t k = c->step_ms.size() / kStepFields;
    if (static_cast<size_t>(capacity) < k) return c->fail(GOCKPT_ENOMEM, "capacity < K");
    memcpy(out, c->step_ms.data(), c->step_ms.size() * sizeof(double));
    return GOCKPT_OK;
}

int gockpt_host_alloc(size_t bytes, void** out) {
    if (out == nullptr) return GOCKPT_EINVAL;
    *out = nullptr;
    if (bytes == 0) bytes = 1;
    hipError_t e = hipHostMalloc(out, bytes, hipHostMallocPortable);
    if (e != hipSuccess) {
        *out = nullptr;
        g_create_error = std::string("gockpt_host_alloc: ") + hipGetErrorString(e);
        return GOCKPT_EHIP;
    }
    // The CPU side of the mapping is populated on first touch; zero the
    // arena with several threads now, so the first restore does not pay one
    // page fault per 4 KiB page.
    const size_t kThreads = bytes >= (size_t(1) << 30) ? 16 : 1;
    const size_t per = (bytes + kThreads - 1) / kThreads;
    std::vector<std::thread> th;
    for (size_t t = 0; t < kThreads; ++t) {
        const size_t a = t * per;
        if (a >= bytes) break;
        const size_t len = a + per <= bytes ? per : bytes - a;
        th.emplace_back([p = static_cast<char*>(*out) + a, len] { memset(p, 0, len); });
    }
    for (auto& x : th) x.join();
    return GOCKPT_OK;
}

int gockpt_host_free(void* p) {
    if (p == nullptr) return GOCKPT_OK;
    hipError_t e = hipHostFree(p);
    if (e != hipSuccess) {
        g_create_error = std::string("gockpt_host_free: ") + hipGetErrorString(e);
        return GOCKPT_EHIP;
    }
    return GOCKPT_OK;
}

int gockpt_replay_arena(int K, const int64_t* bounds, int64_t n, void* host_arena, size_t arena_bytes, double beta1,
                        double beta2, double eps, double weight_decay, int grad_dtype, float* master_out,
                        float* exp_avg_out, float* exp_avg_sq_out, uint16_t* w_bf16_out, gockpt_ckpt_meta* meta,
                        int nthreads) {
    std::string err;
    if (grad_dtype != GOCKPT_GRAD_BF16 && grad_dtype != GOCKPT_GRAD_FP16) {
        g_create_error = "replay_arena: unknown grad_dtype";
        return GOCKPT_EINVAL;
    }
    HParams hp{beta1, beta2, eps, weight_decay};
    int rc = replay_window(K, bounds, n, static_cast<uint8_t*>(host_arena), arena_bytes, 0, 2, hp, grad_dtype,
                           master_out, exp_avg_out, exp_avg_sq_out, w_bf16_out, meta, nthreads, 0, err);
    if (rc != GOCKPT_OK) g_create_error = err;
    return rc;
}

}  // extern "C"
