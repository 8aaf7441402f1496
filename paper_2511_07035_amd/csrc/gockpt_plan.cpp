// gockpt_plan.cpp -- host-only sizing and partitioning (no device calls).
//
//   gockpt_workspace_bytes  device workspace of a context
//   gockpt_arena_layout_for the pinned host arena of a K-step window
//   gockpt_plan_bounds      split [0, n) into K parts (Sec. 4.2.1)
#include <stdint.h>
#include <string.h>

#include "gockpt_internal.h"

namespace {

constexpr uint64_t kArenaAlign = 256;

uint64_t round_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

bool bounds_ok(int K, const int64_t* b, int64_t n) {
    if (K < 1 || K > GOCKPT_MAX_K || b == nullptr || n < 0) return false;
    if (b[0] != 0 || b[K] != n) return false;
    for (int j = 1; j <= K; ++j) {
        if (b[j] <= b[j - 1]) return false;
        if (j < K && (b[j] % GOCKPT_ALIGN_ELEMS) != 0) return false;
    }
    return true;
}

}  // namespace

namespace gockpt {

bool valid_bounds(int K, const int64_t* b, int64_t n) { return bounds_ok(K, b, n); }

// Arena: [records K x 64 B, padded to 4 KiB][master fp32 n][exp_avg fp32 n]
// [exp_avg_sq fp32 n][gradient store]; every piece starts on a 256-byte
// boundary.  Step s's gradient block holds the bf16 gradients of elements
// [0, bounds[s-1]) (step 1's block is empty).  With 1 <= R < K the store is R
// slots sized for the largest block, step s using slot (s-1) mod R (the
// window replays every R steps, freeing the slots); otherwise every step has
// its own block.
void arena_layout(int K, const int64_t* b, int64_t n, int R, gockpt_arena_layout* lay, uint64_t* goff) {
    uint64_t off = 0;
    lay->records = off;
    off = round_up(static_cast<uint64_t>(K) * sizeof(gockpt_step_record), 4096);
    lay->master = off;
    off = round_up(off + 4ull * static_cast<uint64_t>(n), kArenaAlign);
    lay->exp_avg = off;
    off = round_up(off + 4ull * static_cast<uint64_t>(n), kArenaAlign);
    lay->exp_avg_sq = off;
    off = round_up(off + 4ull * static_cast<uint64_t>(n), kArenaAlign);
    lay->grads = off;
    if (R >= 1 && R < K) {
        const uint64_t slot = round_up(2ull * static_cast<uint64_t>(b[K - 1]), kArenaAlign);
        for (int s = 1; s <= K; ++s)
            if (goff != nullptr) goff[s - 1] = off + static_cast<uint64_t>((s - 1) % R) * slot;
        off += static_cast<uint64_t>(R) * slot;
    } else {
        for (int s = 1; s <= K; ++s) {
            if (goff != nullptr) goff[s - 1] = off;
            off = round_up(off + 2ull * static_cast<uint64_t>(b[s - 1]), kArenaAlign);
        }
    }
    lay->total = off;
}

}  // namespace gockpt

extern "C" {

size_t gockpt_workspace_bytes(int64_t n) {
    (void)n;
    return round_up(gockpt::kWsBytes, 256);
}

int gockpt_arena_layout_for(int K, const int64_t* bounds, int64_t n, gockpt_arena_layout* out,
                            uint64_t* grad_offsets) {
    return gockpt_arena_layout_ex(K, bounds, n, 0, out, grad_offsets);
}

int gockpt_arena_layout_ex(int K, const int64_t* bounds, int64_t n, int replay_every, gockpt_arena_layout* out,
                           uint64_t* grad_offsets) {
    if (out == nullptr || !bounds_ok(K, bounds, n) || replay_every < 0) return GOCKPT_EINVAL;
    gockpt::arena_layout(K, bounds, n, replay_every, out, grad_offsets);
    return GOCKPT_OK;
}

int gockpt_plan_bounds(int K, int64_t n, const int64_t* tensor_ends, int n_tensors, int64_t align,
                       int64_t* bounds_out) {
    if (bounds_out == nullptr || K < 1 || K > GOCKPT_MAX_K || n < K) return GOCKPT_EINVAL;
    bounds_out[0] = 0;
    bounds_out[K] = n;
    if (tensor_ends == nullptr) {
        if (align <= 0 || align % GOCKPT_ALIGN_ELEMS != 0) return GOCKPT_EINVAL;
        for (int j = 1; j < K; ++j) {
            // j*n/K without overflow for n < 2^62 / K
            const int64_t target = static_cast<int64_t>((static_cast<__int128>(n) * j) / K);
            bounds_out[j] = target / align * align;
        }
    } else {
        if (n_tensors < K || tensor_ends[n_tensors - 1] != n) return GOCKPT_EINVAL;
        for (int t = 1; t < n_tensors; ++t)
            if (tensor_ends[t] <= tensor_ends[t - 1]) return GOCKPT_EINVAL;
        // Interior bounds are tensor ends other than the last one; pick, for
        // each j, the candidate nearest j*n/K that keeps the sequence strictly
        // increasing and leaves enough candidates for the remaining bounds.
        int prev = -1;  // index into tensor_ends of the previous bound
        const int last_cand = n_tensors - 2;
        for (int j = 1; j < K; ++j) {
            const int64_t target = static_cast<int64_t>((static_cast<__int128>(n) * j) / K);
            const int lo = prev + 1;
            const int hi = last_cand - (K - 1 - j);  // leave K-1-j candidates
            if (lo > hi) return GOCKPT_EINVAL;
            int best = lo;
            int64_t best_d = INT64_MAX;
            for (int c = lo; c <= hi; ++c) {
                const int64_t d = tensor_ends[c] > target ? tensor_ends[c] - target : target - tensor_ends[c];
                if (d < best_d) {
                    best_d = d;
                    best = c;
                }
                if (tensor_ends[c] > target) break;  // later candidates only move away
            }
            bounds_out[j] = tensor_ends[best];
            prev = best;
        }
    }
    return bounds_ok(K, bounds_out, n) ? GOCKPT_OK : GOCKPT_EINVAL;
}

}  // extern "C"
