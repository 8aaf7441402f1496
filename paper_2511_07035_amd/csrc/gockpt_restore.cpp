// gockpt_restore.cpp -- CPU reconstruction of a consistent checkpoint
// (Sec. 4.3.1, Fig. update_backend).
//
// Part j of the state reached the host arena as it stood after window step j;
// steps j+1..K then moved it on the device.  Replaying those steps on the host
// with the gradients the window saved for part j (the gradient block of step s
// covers parts 1..s-1) and each step's recorded step count, learning rate and
// loss scale gives the state after step K -- the checkpoint a blocking
// snapshot after the last step would hold.  Skipped steps are not replayed.
//
// The replay is time-fused: a tile of elements is loaded once, all of its
// steps in the requested range are applied while it sits in L1, and it is
// stored once.  Worker threads take pieces from a shared counter (Sec. 4.3.1
// runs the update with several threads).  The same routine serves the replay
// at restore time (all steps at once) and the in-window replay of a batch of
// steps (steps a+1..b onto the parts received so far).
#include <immintrin.h>
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <chrono>
#include <string>
#include <thread>
#include <vector>

#include "gockpt_internal.h"

#pragma clang fp contract(off)

namespace gockpt {

// Move a landed staging slot into the pageable arena with streaming stores:
// the arena's lines are written whole and not read first (an ordinary copy
// would fetch each destination line before overwriting it), and they do not
// displace the replay's working set from the caches.
void copy_to_arena(void* dst, const void* src, size_t len) {
    uint8_t* d = static_cast<uint8_t*>(dst);
    const uint8_t* s = static_cast<const uint8_t*>(src);
    const size_t head = (32 - (reinterpret_cast<uintptr_t>(d) & 31)) & 31;
    if (len < head + 256) {
        memcpy(d, s, len);
        return;
    }
    memcpy(d, s, head);
    d += head;
    s += head;
    len -= head;
    const size_t body = len / 128 * 128;
    for (size_t i = 0; i < body; i += 128) {
        const __m256i a = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(s + i));
        const __m256i b = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(s + i + 32));
        const __m256i c = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(s + i + 64));
        const __m256i e = _mm256_loadu_si256(reinterpret_cast<const __m256i*>(s + i + 96));
        _mm256_stream_si256(reinterpret_cast<__m256i*>(d + i), a);
        _mm256_stream_si256(reinterpret_cast<__m256i*>(d + i + 32), b);
        _mm256_stream_si256(reinterpret_cast<__m256i*>(d + i + 64), c);
        _mm256_stream_si256(reinterpret_cast<__m256i*>(d + i + 96), e);
    }
    _mm_sfence();  // the streamed lines are visible before the slot is released
    memcpy(d + body, s + body, len - body);
}

void arena_layout(int K, const int64_t* b, int64_t n, int R, gockpt_arena_layout* lay, uint64_t* goff);
bool valid_bounds(int K, const int64_t* b, int64_t n);

namespace {

constexpr int64_t kPiece = 1 << 16;  // elements per work item
constexpr int64_t kTile = 1024;      // elements kept in L1 while replaying

struct Piece {
    int64_t begin, end;
    int first_step, last_step;  // inclusive; empty if first > last
};

bool same_bits(float a, float b) { return f32_to_bits(a) == f32_to_bits(b); }

}  // namespace

int check_records(int K, const gockpt_step_record* rec, int upto, const HParams& hp, StepScalars* sc,
                  std::string& err) {
    for (int s = 1; s <= upto; ++s) {
        const gockpt_step_record& r = rec[s - 1];
        if (r.window_step != s) {
            err = "replay: record " + std::to_string(s) + " has window_step " + std::to_string(r.window_step);
            return GOCKPT_EFAILED;
        }
        if (s > 1) {
            const int64_t expect_t = rec[s - 2].t + (r.skip ? 0 : 1);
            if (r.t != expect_t) {
                err = "replay: step count of record " + std::to_string(s) + " is inconsistent";
                return GOCKPT_EFAILED;
            }
        }
        sc[s - 1] = step_scalars(hp, r.lr, r.t, r.scale_used);
        if (!r.skip) {
            const StepScalars& c = sc[s - 1];
            if (!same_bits(c.step_size, r.step_size) || !same_bits(c.sqrt_bc2, r.sqrt_bc2) ||
                !same_bits(c.decay, r.decay) || !same_bits(c.inv_scale, r.inv_scale)) {
                err = "replay: host scalars of step " + std::to_string(s) + " differ from the device's";
                return GOCKPT_EFAILED;
            }
        }
    }
    (void)K;
    return GOCKPT_OK;
}

// Parts first_part..last_part: load from (ip, im, iv), apply steps
// max(s_lo, j+1)..s_hi of part j with the gradient block gblk[s-1] (indexed
// from element 0), store to (op, om, ov); w_out (nullable) gets bf16(p).
// Records 1..s_hi must have been checked (sc filled).  Returns the number of
// element updates applied.
namespace {

// The time-fused tile loop of one piece: load, all steps, store.
template <int kKind>
void replay_piece(const Piece& pc, const gockpt_step_record* rec, const StepScalars* sc,
                  const uint16_t* const* gblk, const float* ip, const float* im, const float* iv, float* op,
                  float* om, float* ov, uint16_t* w_out) {
    alignas(64) float tp[kTile], tm[kTile], tv[kTile];
    for (int64_t a = pc.begin; a < pc.end; a += kTile) {
        const int64_t len = a + kTile < pc.end ? kTile : pc.end - a;
        memcpy(tp, ip + a, len * sizeof(float));
        memcpy(tm, im + a, len * sizeof(float));
        memcpy(tv, iv + a, len * sizeof(float));
        for (int s = pc.first_step; s <= pc.last_step; ++s) {
            if (rec[s - 1].skip) continue;
            const StepScalars c = sc[s - 1];
            const uint16_t* g = gblk[s - 1] + a;
            for (int64_t i = 0; i < len; ++i) adamw_update<kKind>(c, g[i], tp[i], tm[i], tv[i]);
        }
        memcpy(op + a, tp, len * sizeof(float));
        memcpy(om + a, tm, len * sizeof(float));
        memcpy(ov + a, tv, len * sizeof(float));
        if (w_out != nullptr)
            for (int64_t i = 0; i < len; ++i) w_out[a + i] = f32_to_bf16_rne(tp[i]);
    }
}

}  // namespace

int64_t replay_parts(int K, const int64_t* bounds, const gockpt_step_record* rec, const StepScalars* sc,
                     const uint16_t* const* gblk, int first_part, int last_part, int s_lo, int s_hi,
                     const float* ip, const float* im, const float* iv, float* op, float* om, float* ov,
                     uint16_t* w_out, int nthreads, int grad_kind) {
    (void)K;
    std::vector<Piece> pieces;
    int64_t updates = 0;
    for (int j = first_part; j <= last_part; ++j) {
        const int fs = s_lo > j + 1 ? s_lo : j + 1;
        int live = 0;
        for (int s = fs; s <= s_hi; ++s) live += rec[s - 1].skip ? 0 : 1;
        const bool copy_needed = (ip != op) || (im != om) || (iv != ov) || w_out != nullptr;
        if (live == 0 && !copy_needed) continue;
        updates += static_cast<int64_t>(live) * (bounds[j] - bounds[j - 1]);
        for (int64_t a = bounds[j - 1]; a < bounds[j]; a += kPiece) {
            const int64_t e = a + kPiece < bounds[j] ? a + kPiece : bounds[j];
            pieces.push_back({a, e, fs, s_hi});
        }
    }
    std::atomic<size_t> next{0};
    auto worker = [&]() {
        for (;;) {
            const size_t k = next.fetch_add(1, std::memory_order_relaxed);
            if (k >= pieces.size()) break;
            if (grad_kind == kGradFP16)
                replay_piece<kGradFP16>(pieces[k], rec, sc, gblk, ip, im, iv, op, om, ov, w_out);
            else
                replay_piece<kGradBF16>(pieces[k], rec, sc, gblk, ip, im, iv, op, om, ov, w_out);
        }
    };
    if (nthreads <= 0) nthreads = 16;
    if (static_cast<size_t>(nthreads) > pieces.size()) nthreads = pieces.empty() ? 1 : static_cast<int>(pieces.size());
    std::vector<std::thread> pool;
    for (int i = 1; i < nthreads; ++i) pool.emplace_back(worker);
    worker();
    for (auto& th : pool) th.join();
    return updates;
}

// The restore: steps s_first..K (s_first = first step not yet replayed during
// the window, 2 when nothing was) onto every part, out of place or in place.
int replay_window(int K, const int64_t* bounds, int64_t n, uint8_t* arena, size_t arena_bytes, int R,
                  int s_first, const HParams& hp, int grad_kind, float* p_out, float* m_out, float* v_out,
                  uint16_t* w_out, gockpt_ckpt_meta* meta, int nthreads, int64_t earlier_updates,
                  std::string& err) {
    const auto t_start = std::chrono::steady_clock::now();
    if (!valid_bounds(K, bounds, n)) {
        err = "replay: invalid K or bounds";
        return GOCKPT_EINVAL;
    }
    gockpt_arena_layout lay;
    std::vector<uint64_t> goff(K);
    arena_layout(K, bounds, n, R, &lay, goff.data());
    if (arena == nullptr || arena_bytes < lay.total) {
        err = "replay: host arena missing or smaller than the window layout";
        return GOCKPT_ENOMEM;
    }
    const gockpt_step_record* rec = reinterpret_cast<const gockpt_step_record*>(arena + lay.records);
    std::vector<StepScalars> sc(K);
    int rc = check_records(K, rec, K, hp, sc.data(), err);
    if (rc != GOCKPT_OK) return rc;
    int skipped = 0;
    for (int s = 1; s <= K; ++s) skipped += rec[s - 1].skip ? 1 : 0;
    std::vector<const uint16_t*> gblk(K);
    for (int s = 1; s <= K; ++s) gblk[s - 1] = reinterpret_cast<const uint16_t*>(arena + goff[s - 1]);
    float* ap = reinterpret_cast<float*>(arena + lay.master);
    float* am = reinterpret_cast<float*>(arena + lay.exp_avg);
    float* av = reinterpret_cast<float*>(arena + lay.exp_avg_sq);
    if (p_out == nullptr) p_out = ap;
    if (m_out == nullptr) m_out = am;
    if (v_out == nullptr) v_out = av;
    const int64_t updates = replay_parts(K, bounds, rec, sc.data(), gblk.data(), 1, K, s_first < 2 ? 2 : s_first, K,
                                         ap, am, av, p_out, m_out, v_out, w_out, nthreads, grad_kind);
    if (meta != nullptr) {
        const gockpt_step_record& last = rec[K - 1];
        meta->t = last.t;
        meta->tracker = last.tracker;
        meta->scale = last.scale_next;
        meta->K = K;
        meta->skipped = skipped;
        meta->reserved_ = 0;
        meta->element_updates = updates + earlier_updates;
        meta->restore_ms =
            std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_start).count();
    }
    return GOCKPT_OK;
}

}  // namespace gockpt
