// gockpt_planner.cpp -- window planner (Sec. 4.2.3 "Checkpoint Stall
// Analysis"): an event model of a window on two streams, and a search over
// the window length K and the part bounds that minimises the predicted stall.
//
// The model follows what gockpt_step does (host-only, no device calls):
//   compute stream, per step: forward (t_fwd) -> [lazy rule: wait for the
//   previous step's gradient copies that came straight from the gradient
//   buffer] -> backward (t_bwd) -> [wait for the previous step's direct state
//   copies] -> ring plan -> update (t_upd + pack stores) -> [GRADS: wait for
//   this step's gradient copies; ALL: for all of its copies].
//   copy stream: the step's gradients that did not fit the ring, straight
//   from the gradient buffer, as soon as the update starts; after the update,
//   the ring's gradients and state, then the rest of the state; in pieces of
//   copy_bytes at link_gbs, one after another and after the previous step's.
//   ring: a byte stream; a step uses the space whose copies have finished by
//   the time its update starts (QUERY / HOST_WAIT), or the whole ring with the
//   update waiting for the copies of the bytes it overwrites (DEVICE_WAIT);
//   whole segments first, then the largest multiple of 8 elements that fits,
//   and everything after that goes straight from the live buffers.  Space is
//   freed per pack segment, when the segment's last copy has finished.
//   staging (pageable arena): copy q lands in slot q mod nslots, starts only
//   once the host has emptied the slot (copy q - nslots), and the host
//   empties landed slots in copy order at host_gbs.  Each step's record takes
//   a slot of its own (its bytes are negligible and not counted).
// The stall is the compute-stream time of the window's K steps and the step
// after it (which carries the last lazy waits) minus K + 1 plain steps.
//
// With the paper's own accounting (14 B of state and 2 B of gradient per
// element, one part's transfer taking one step, no ring) the model gives the
// stall formulas of Sec. 4.2.3: (N-1) T_step for Async-O and N(N-1)/14 T_step
// for GoCkpt with its explicit gradient wait.
#include <math.h>
#include <stdint.h>
#include <string.h>

#include <deque>
#include <vector>

#include "gockpt_internal.h"

namespace {

struct Params {
    int64_t n;
    const int64_t* tensor_ends;
    int n_tensors;
    int policy;
    int64_t align;
    double t_fwd, t_bwd, t_upd;
    double pack_rate;  // bytes per ms (0: the pack is free)
    double link;       // bytes per ms
    uint64_t ring;
    uint64_t chunk;
    double S, G;  // bytes per element: state of a part, one gradient
    int max_K;
    int ring_plan;
    uint64_t nslots;   // staging slots (0: pinned arena)
    double host_rate;  // bytes per ms (0: instant)
};

bool load_params(const gockpt_plan_params* p, Params* q) {
    if (p == nullptr || p->n < 1 || !(p->link_gbs > 0.0) || !(p->t_fwd_ms >= 0.0) || !(p->t_bwd_ms >= 0.0) ||
        !(p->t_upd_ms >= 0.0) || !isfinite(p->t_fwd_ms + p->t_bwd_ms + p->t_upd_ms) || !isfinite(p->link_gbs))
        return false;
    if (p->wait_policy < GOCKPT_WAIT_LAZY || p->wait_policy > GOCKPT_WAIT_ALL) return false;
    if (p->ring_bytes % 256 != 0) return false;
    if (p->copy_bytes % 256 != 0) return false;
    if (p->max_K > GOCKPT_MAX_K) return false;
    if (p->ring_plan < GOCKPT_RING_QUERY || p->ring_plan > GOCKPT_RING_DEVICE_WAIT) return false;
    if (!isfinite(p->host_gbs)) return false;
    q->n = p->n;
    q->tensor_ends = p->tensor_ends;
    q->n_tensors = p->n_tensors;
    if (q->tensor_ends != nullptr) {
        if (q->n_tensors < 1 || q->tensor_ends[q->n_tensors - 1] != p->n) return false;
        for (int t = 0; t < q->n_tensors; ++t)
            if (q->tensor_ends[t] <= (t ? q->tensor_ends[t - 1] : 0)) return false;
    }
    q->policy = p->wait_policy;
    q->align = p->align > 0 ? p->align : 256;
    if (q->align % GOCKPT_ALIGN_ELEMS != 0) return false;
    q->t_fwd = p->t_fwd_ms;
    q->t_bwd = p->t_bwd_ms;
    q->t_upd = p->t_upd_ms;
    q->pack_rate = p->pack_gbs > 0.0 ? p->pack_gbs * 1e6 : 0.0;
    q->link = p->link_gbs * 1e6;
    q->ring = p->ring_bytes;
    q->chunk = p->copy_bytes ? p->copy_bytes : GOCKPT_DEFAULT_COPY_BYTES;
    q->S = p->state_bytes > 0.0 ? p->state_bytes : 12.0;
    q->G = p->grad_bytes > 0.0 ? p->grad_bytes : 2.0;
    q->max_K = p->max_K > 0 ? p->max_K : 7;
    q->ring_plan = p->ring_plan;
    if (p->staging_bytes != 0 && p->staging_bytes < q->chunk) return false;
    q->nslots = p->staging_bytes / q->chunk;
    q->host_rate = p->host_gbs > 0.0 ? p->host_gbs * 1e6 : 0.0;
    return true;
}

uint64_t up256(double x) {
    const uint64_t b = static_cast<uint64_t>(ceil(x));
    return (b + 255) / 256 * 256;
}

struct SimOut {
    double stall = 0, latency = 0, d2h = 0, spilled = 0;
};

// One window with bounds b[0..K]; per_step (nullable, K+1 entries) gets each
// step's delay over a plain step.
SimOut simulate(const Params& P, int K, const int64_t* b, double* per_step) {
    struct Segment {
        uint64_t lbeg, lend;
        double done;  // the segment's last copy has finished
    };
    std::deque<Segment> inflight;
    uint64_t head = 0;
    const double T = P.t_fwd + P.t_bwd + P.t_upd;
    double t = 0.0, copy_free = 0.0;
    double grad_spill_done = -1.0, state_spill_done = -1.0;
    // staging: when the host has emptied each copy's slot, in copy order
    std::vector<double> emptied;
    double host_free = 0.0;
    const bool device_wait = P.ring_plan == GOCKPT_RING_DEVICE_WAIT;
    SimOut o;
    for (int s = 1; s <= K + 1; ++s) {
        const double t0 = t;
        t += P.t_fwd;
        if (grad_spill_done >= 0.0) t = t > grad_spill_done ? t : grad_spill_done;
        grad_spill_done = -1.0;
        t += P.t_bwd;
        if (state_spill_done >= 0.0) t = t > state_spill_done ? t : state_spill_done;
        state_spill_done = -1.0;
        if (s == K + 1) {  // the first step after the window: plain update
            t += P.t_upd;
            if (per_step != nullptr) per_step[s - 1] = t - t0 - T;
            break;
        }
        // ring plan at the start of the update
        double avail = 0.0;
        if (P.ring) {
            if (device_wait) {
                avail = static_cast<double>(P.ring);
            } else {
                while (!inflight.empty() && inflight.front().done <= t) inflight.pop_front();
                const uint64_t drained = inflight.empty() ? head : inflight.front().lbeg;
                avail = static_cast<double>(P.ring) - static_cast<double>(head - drained);
            }
        }
        if (avail < 0.0) avail = 0.0;
        const double len[2] = {static_cast<double>(b[s - 1]), static_cast<double>(b[s] - b[s - 1])};
        const double esz[2] = {P.G, P.S};
        double ring_b[2] = {0, 0}, spill_b[2] = {0, 0};
        uint64_t lstart[2] = {0, 0};
        uint64_t lpos = head;
        bool full = false;
        for (int k = 0; k < 2; ++k) {
            lstart[k] = lpos;
            const double bytes = len[k] * esz[k];
            const double need = static_cast<double>(up256(bytes));
            if (!full && need <= avail) {
                ring_b[k] = bytes;
                avail -= need;
                lpos += static_cast<uint64_t>(need);
            } else {
                double fit = full ? 0.0 : floor(avail / (esz[k] * GOCKPT_ALIGN_ELEMS)) * GOCKPT_ALIGN_ELEMS;
                if (fit > len[k]) fit = len[k];
                ring_b[k] = fit * esz[k];
                lpos += static_cast<uint64_t>(ring_b[k]);
                avail = 0.0;
                full = true;
            }
            spill_b[k] = bytes - ring_b[k];
        }
        head = (lpos + 255) / 256 * 256;
        if (device_wait && P.ring && head > P.ring) {
            // the update overwrites logical bytes below head - ring: it waits
            // for the segments there (their copies finish in order)
            const uint64_t reuse_end = head - P.ring;
            while (!inflight.empty() && inflight.front().lbeg < reuse_end) {
                t = t > inflight.front().done ? t : inflight.front().done;
                inflight.pop_front();
            }
        }
        const double pack = ring_b[0] + ring_b[1];
        const double t_start = t;
        t += P.t_upd + (P.pack_rate > 0.0 ? pack / P.pack_rate : 0.0);
        // copies of the step, in the library's order: the gradients from the
        // gradient buffer need only the gradients, the rest the update
        double c = t_start > copy_free ? t_start : copy_free;
        auto piece_copy = [&](double bytes) {
            if (P.nslots) {
                const size_t q = emptied.size();
                if (q >= P.nslots && emptied[q - P.nslots] > c) c = emptied[q - P.nslots];
                c += bytes / P.link;
                host_free = (host_free > c ? host_free : c) + (P.host_rate > 0.0 ? bytes / P.host_rate : 0.0);
                emptied.push_back(host_free);
            } else {
                c += bytes / P.link;
            }
        };
        auto run = [&](double bytes, bool from_ring, uint64_t l0) {
            double done = 0.0;
            while (done < bytes) {
                const double piece = bytes - done < static_cast<double>(P.chunk) ? bytes - done
                                                                                  : static_cast<double>(P.chunk);
                piece_copy(piece);
                done += piece;
            }
            if (from_ring && bytes > 0.0) inflight.push_back({l0, l0 + static_cast<uint64_t>(bytes), c});
        };
        run(spill_b[0], false, 0);
        if (spill_b[0] > 0.0) grad_spill_done = c;
        if (c < t) c = t;
        if (P.nslots) piece_copy(0.0);  // the step record's slot
        run(ring_b[0], true, lstart[0]);
        const double grads_done = c;
        run(ring_b[1], true, lstart[1]);
        run(spill_b[1], false, 0);
        if (spill_b[1] > 0.0) state_spill_done = c;
        copy_free = c;
        o.d2h += ring_b[0] + ring_b[1] + spill_b[0] + spill_b[1];
        o.spilled += spill_b[0] + spill_b[1];
        if (P.policy == GOCKPT_WAIT_GRADS) t = t > grads_done ? t : grads_done;
        if (P.policy == GOCKPT_WAIT_ALL) t = t > c ? t : c;
        if (per_step != nullptr) per_step[s - 1] = t - t0 - T;
    }
    o.stall = t - (K + 1) * T;
    o.latency = copy_free > host_free ? copy_free : host_free;
    return o;
}

bool bounds_valid(int K, const int64_t* b, int64_t n) {
    if (b[0] != 0 || b[K] != n) return false;
    for (int j = 1; j <= K; ++j) {
        if (b[j] <= b[j - 1]) return false;
        if (j < K && b[j] % GOCKPT_ALIGN_ELEMS != 0) return false;
    }
    return true;
}

// Interior bound positions the planner may use, in increasing order: the
// multiples of align below n, or the tensor ends below n that are multiples
// of 8.  Element mode is kept implicit (pos(i) = (i + 1) * align).
struct Positions {
    const Params* P;
    std::vector<int64_t> list;  // tensor mode
    int64_t m = 0;              // number of positions
    void init(const Params& p) {
        P = &p;
        if (p.tensor_ends != nullptr) {
            for (int t = 0; t < p.n_tensors; ++t)
                if (p.tensor_ends[t] < p.n && p.tensor_ends[t] % GOCKPT_ALIGN_ELEMS == 0) list.push_back(p.tensor_ends[t]);
            m = static_cast<int64_t>(list.size());
        } else {
            m = (p.n - 1) / p.align;
        }
    }
    int64_t pos(int64_t i) const { return P->tensor_ends != nullptr ? list[i] : (i + 1) * P->align; }
    // index of the position nearest to x
    int64_t nearest(double x) const {
        if (m == 0) return 0;
        if (P->tensor_ends == nullptr) {
            int64_t i = llround(x / static_cast<double>(P->align)) - 1;
            return i < 0 ? 0 : (i >= m ? m - 1 : i);
        }
        int64_t lo = 0, hi = m - 1;
        while (lo < hi) {
            const int64_t mid = (lo + hi) / 2;
            if (static_cast<double>(list[mid]) < x) lo = mid + 1; else hi = mid;
        }
        if (lo > 0 && fabs(static_cast<double>(list[lo - 1]) - x) <= fabs(static_cast<double>(list[lo]) - x)) --lo;
        return lo;
    }
};

// Better plan: lower stall, then fewer bytes to the host, then an earlier
// last copy, then a shorter window; differences within eps (stall, latency)
// and rel (bytes) count as ties.
struct Order {
    double eps;      // ms
    double rel = 0;  // relative tolerance on bytes
    bool operator()(const SimOut& a, int ka, const SimOut& b, int kb) const {
        if (a.stall < b.stall - eps) return true;
        if (a.stall > b.stall + eps) return false;
        if (a.d2h < b.d2h * (1.0 - rel)) return true;
        if (a.d2h > b.d2h * (1.0 + rel)) return false;
        if (a.latency < b.latency - eps) return true;
        if (a.latency > b.latency + eps) return false;
        return ka < kb;
    }
};

struct Search {
    const Params& P;
    Positions pos;
    Order better;  // across window lengths: near-equal stalls are ties
    Order finer;   // within one window length: any lower stall wins
    int64_t budget = 40000;  // simulations
    std::vector<int64_t> b;

    explicit Search(const Params& p) : P(p) {
        pos.init(p);
        // stalls closer than 1 us or 1e-4 of a step are ties
        const double T = p.t_fwd + p.t_bwd + p.t_upd;
        better.eps = 1e-4 * T > 1e-3 ? 1e-4 * T : 1e-3;
        better.rel = 1e-4;
        finer.eps = 1e-12 * (T > 1.0 ? T : 1.0);
        finer.rel = 1e-15;
    }
    SimOut eval(int K, const std::vector<int64_t>& idx) {
        b.assign(K + 1, 0);
        b[K] = P.n;
        for (int j = 1; j < K; ++j) b[j] = pos.pos(idx[j]);
        --budget;
        return simulate(P, K, b.data(), nullptr);
    }
    // idx[1..K-1] strictly increasing in [0, m); idx[0], idx[K] unused.
    bool fix(int K, std::vector<int64_t>& idx) {
        if (pos.m < K - 1) return false;
        for (int j = 1; j < K; ++j) {
            const int64_t lo = j > 1 ? idx[j - 1] + 1 : 0;
            if (idx[j] < lo) idx[j] = lo;
        }
        for (int j = K - 1; j >= 1; --j) {
            const int64_t hi = pos.m - 1 - (K - 1 - j);
            const int64_t cap = j < K - 1 ? idx[j + 1] - 1 : hi;
            if (idx[j] > (hi < cap ? hi : cap)) idx[j] = hi < cap ? hi : cap;
        }
        for (int j = 1; j < K; ++j)
            if (idx[j] < 0 || (j > 1 && idx[j] <= idx[j - 1])) return false;
        return true;
    }
    static double binom(int64_t m, int k) {
        double c = 1.0;
        for (int i = 0; i < k; ++i) c = c * static_cast<double>(m - i) / (i + 1);
        return c;
    }
    // every choice of K - 1 interior positions
    void exhaustive(int K, std::vector<int64_t>& idx, int j, std::vector<int64_t>& best_idx, SimOut& best,
                    bool& have) {
        if (j == K) {
            const SimOut o = eval(K, idx);
            if (!have || finer(o, K, best, K)) {
                best = o;
                best_idx = idx;
                have = true;
            }
            return;
        }
        const int64_t lo = j > 1 ? idx[j - 1] + 1 : 0;
        for (int64_t i = lo; i <= pos.m - 1 - (K - 1 - j); ++i) {
            idx[j] = i;
            exhaustive(K, idx, j + 1, best_idx, best, have);
        }
    }
    // one bound at a time by +-step positions, halving the step when no move helps
    void refine(int K, std::vector<int64_t>& idx, SimOut& cur) {
        if (K < 2) return;
        int64_t step = pos.m / (2 * K);
        if (step < 1) step = 1;
        std::vector<int64_t> trial;
        while (step >= 1 && budget > 0) {
            bool moved = false;
            for (int j = 1; j < K && budget > 0; ++j) {
                for (int dir = -1; dir <= 1; dir += 2) {
                    trial = idx;
                    trial[j] += dir * step;
                    const int64_t lo = j > 1 ? idx[j - 1] + 1 : 0;
                    const int64_t hi = j < K - 1 ? idx[j + 1] - 1 : pos.m - 1;
                    if (trial[j] < lo || trial[j] > hi) continue;
                    const SimOut o = eval(K, trial);
                    if (finer(o, K, cur, K)) {
                        idx = trial;
                        cur = o;
                        moved = true;
                        break;
                    }
                }
            }
            if (!moved) step /= 2;
        }
    }
    // best bounds for one K
    bool best_for(int K, std::vector<int64_t>& out_idx, SimOut& out) {
        std::vector<int64_t> idx(K + 1, 0);
        bool have = false;
        if (K == 1) {
            out = eval(1, idx);
            out_idx = idx;
            return true;
        }
        if (pos.m < K - 1) return false;
        if (binom(pos.m, K - 1) <= 20000.0) {
            exhaustive(K, idx, 1, out_idx, out, have);
            return have;
        }
        // starting layouts: equal parts, parts that keep every step's copy
        // volume equal, and front- or back-loaded variants; the best three are
        // refined
        const double q = 1.0 - P.G / P.S;
        struct Start {
            std::vector<int64_t> idx;
            SimOut o;
        };
        std::vector<Start> starts;
        const double gammas[] = {1.0, 0.0, 0.6, 0.8, 1.25, 1.6};
        for (double g : gammas) {
            for (int j = 1; j < K; ++j) {
                double f;
                if (g == 0.0)
                    f = (q > 0.0 && q < 1.0) ? (1.0 - pow(q, j)) / (1.0 - pow(q, K)) : static_cast<double>(j) / K;
                else
                    f = pow(static_cast<double>(j) / K, g);
                idx[j] = pos.nearest(f * static_cast<double>(P.n));
            }
            if (!fix(K, idx)) continue;
            starts.push_back({idx, eval(K, idx)});
        }
        if (starts.empty()) return false;
        for (size_t a = 0; a < starts.size(); ++a)
            for (size_t c = a + 1; c < starts.size(); ++c)
                if (finer(starts[c].o, K, starts[a].o, K)) std::swap(starts[a], starts[c]);
        for (size_t a = 0; a < starts.size() && a < 3; ++a) {
            refine(K, starts[a].idx, starts[a].o);
            if (!have || finer(starts[a].o, K, out, K)) {
                out = starts[a].o;
                out_idx = starts[a].idx;
                have = true;
            }
        }
        return have;
    }
};

void fill(gockpt_plan_result* out, int K, const SimOut& o) {
    out->K = K;
    out->reserved_ = 0;
    out->stall_ms = o.stall;
    out->latency_ms = o.latency;
    out->d2h_bytes = o.d2h;
    out->spilled_bytes = o.spilled;
}

}  // namespace

extern "C" {

int gockpt_simulate_window(const gockpt_plan_params* params, int K, const int64_t* bounds, gockpt_plan_result* out,
                           double* step_stall_ms) {
    Params P;
    if (!load_params(params, &P) || out == nullptr || bounds == nullptr || K < 1 || K > GOCKPT_MAX_K ||
        !bounds_valid(K, bounds, P.n))
        return GOCKPT_EINVAL;
    fill(out, K, simulate(P, K, bounds, step_stall_ms));
    return GOCKPT_OK;
}

int gockpt_plan_window(const gockpt_plan_params* params, int64_t* bounds_out, gockpt_plan_result* out) {
    Params P;
    if (!load_params(params, &P) || out == nullptr || bounds_out == nullptr) return GOCKPT_EINVAL;
    Search S(P);
    std::vector<int64_t> best_idx;
    SimOut best;
    int best_K = 0;
    for (int K = 1; K <= P.max_K; ++K) {
        std::vector<int64_t> idx;
        SimOut o;
        if (!S.best_for(K, idx, o)) continue;
        if (best_K == 0 || S.better(o, K, best, best_K)) {
            best = o;
            best_K = K;
            best_idx = idx;
        }
    }
    if (best_K == 0) return GOCKPT_EINVAL;
    bounds_out[0] = 0;
    bounds_out[best_K] = P.n;
    for (int j = 1; j < best_K; ++j) bounds_out[j] = S.pos.pos(best_idx[j]);
    fill(out, best_K, best);
    return GOCKPT_OK;
}

}  // extern "C"
