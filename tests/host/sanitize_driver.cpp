// Host-only driver for the sanitizer builds of the library's CPU code: the
// window planner, part bounds and arena layout, the checkpoint writer and
// reader, and the multithreaded replay.  Built with g++ against the .cpp
// sources (no HIP runtime); exits non-zero on any inconsistency, and the
// sanitizers abort on memory or threading errors.
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#include <string>
#include <vector>

#include "gockpt_internal.h"

namespace gockpt {
void set_host_error(const std::string& msg) { fprintf(stderr, "host error: %s\n", msg.c_str()); }
int replay_window(int K, const int64_t* bounds, int64_t n, uint8_t* arena, size_t arena_bytes, int R,
                  int s_first, const HParams& hp, int grad_kind, float* p_out, float* m_out, float* v_out,
                  uint16_t* w_out, gockpt_ckpt_meta* meta, int nthreads, int64_t earlier_updates,
                  std::string& err);
void arena_layout(int K, const int64_t* b, int64_t n, int R, gockpt_arena_layout* lay, uint64_t* goff);
void copy_to_arena(void* dst, const void* src, size_t len);
}  // namespace gockpt

#define CHECK(x)                                                  \
    do {                                                          \
        if (!(x)) {                                               \
            fprintf(stderr, "%s:%d check failed: %s\n", __FILE__, __LINE__, #x); \
            exit(1);                                              \
        }                                                         \
    } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t rnd() {
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    return static_cast<uint32_t>(rng_state >> 11);
}

static void planner() {
    gockpt_plan_params p;
    memset(&p, 0, sizeof p);
    p.n = 1 << 22;
    p.t_fwd_ms = 3;
    p.t_bwd_ms = 6;
    p.t_upd_ms = 0.5;
    p.link_gbs = 2;
    p.ring_bytes = 1 << 20;
    p.copy_bytes = 1 << 18;
    p.max_K = 9;
    for (int pol = 0; pol < 3; ++pol) {
        p.wait_policy = pol;
        std::vector<int64_t> b(p.max_K + 1);
        gockpt_plan_result r;
        CHECK(gockpt_plan_window(&p, b.data(), &r) == GOCKPT_OK);
        CHECK(r.K >= 1 && r.K <= p.max_K && b[0] == 0 && b[r.K] == p.n);
        std::vector<double> per(r.K + 1);
        gockpt_plan_result r2;
        CHECK(gockpt_simulate_window(&p, r.K, b.data(), &r2, per.data()) == GOCKPT_OK);
        CHECK(r2.stall_ms == r.stall_ms);
    }
    std::vector<int64_t> ends;
    int64_t e = 0;
    for (int t = 0; t < 300; ++t) ends.push_back(e += 8 * (1 + rnd() % 4096));
    p.n = e;
    p.tensor_ends = ends.data();
    p.n_tensors = static_cast<int32_t>(ends.size());
    std::vector<int64_t> b(p.max_K + 1);
    gockpt_plan_result r;
    CHECK(gockpt_plan_window(&p, b.data(), &r) == GOCKPT_OK);
    std::vector<int64_t> pb(9);
    CHECK(gockpt_plan_bounds(8, e, ends.data(), static_cast<int>(ends.size()), 0, pb.data()) == GOCKPT_OK);
    CHECK(gockpt_plan_bounds(8, e, nullptr, 0, 256, pb.data()) == GOCKPT_OK);
}

static void persistence(const char* dir) {
    const int64_t n = 300007;
    std::vector<float> p(n), m(n), v(n), q(n), r(n), s(n);
    for (int64_t i = 0; i < n; ++i) {
        p[i] = static_cast<float>(rnd()) * 1e-9f;
        m[i] = -p[i];
        v[i] = p[i] * p[i];
    }
    gockpt_ckpt_info info;
    memset(&info, 0, sizeof info);
    info.n = n;
    info.t = 77;
    info.scale = 1024.0f;
    info.beta1 = 0.9;
    info.beta2 = 0.999;
    info.eps = 1e-8;
    info.weight_decay = 0.01;
    info.piece_bytes = 1 << 16;
    gockpt_io_stats st;
    CHECK(gockpt_write_checkpoint(dir, p.data(), m.data(), v.data(), &info, "user text\n", 6, &st) == GOCKPT_OK);
    gockpt_ckpt_info got;
    CHECK(gockpt_read_checkpoint(dir, n, q.data(), r.data(), s.data(), &got, 5, &st) == GOCKPT_OK);
    CHECK(memcmp(p.data(), q.data(), n * 4) == 0 && memcmp(m.data(), r.data(), n * 4) == 0 &&
          memcmp(v.data(), s.data(), n * 4) == 0);
    CHECK(got.t == 77 && got.scale == 1024.0f && got.has_user == 1);
    char buf[64];
    size_t len = 0;
    CHECK(gockpt_read_checkpoint_user(dir, buf, sizeof buf, &len) == GOCKPT_OK && len == 10);
    CHECK(gockpt_read_checkpoint(dir, n + 8, q.data(), r.data(), s.data(), &got, 2, &st) == GOCKPT_EINVAL);
}

// A drained arena built here: records whose scalars follow the contract, the
// state of each part, and the gradient blocks; replayed with 1 and 4 threads,
// which must give the same bits.
static void replay() {
    const int K = 6;
    const int64_t n = 200003;
    const int64_t bounds[K + 1] = {0, 8, 40000, 80000, 120000, 199992, n};
    gockpt::HParams hp{0.9, 0.999, 1e-8, 0.01};
    for (int kind = 0; kind < 2; ++kind) {
        gockpt_arena_layout lay;
        std::vector<uint64_t> goff(K);
        gockpt::arena_layout(K, bounds, n, 0, &lay, goff.data());
        std::vector<uint8_t> arena(lay.total + 256);
        uint8_t* base = arena.data() + ((256 - reinterpret_cast<uintptr_t>(arena.data()) % 256) % 256);
        auto* rec = reinterpret_cast<gockpt_step_record*>(base + lay.records);
        for (int s = 1; s <= K; ++s) {
            gockpt_step_record& r = rec[s - 1];
            memset(&r, 0, sizeof r);
            r.window_step = s;
            r.skip = s == 3;
            r.t = s == 1 ? 1 : rec[s - 2].t + (r.skip ? 0 : 1);
            r.scale_used = 1.0f;
            r.lr = 1e-3f;
            const gockpt::StepScalars c = gockpt::step_scalars(hp, r.lr, r.t, r.scale_used);
            r.step_size = c.step_size;
            r.sqrt_bc2 = c.sqrt_bc2;
            r.decay = c.decay;
            r.inv_scale = c.inv_scale;
        }
        float* ap = reinterpret_cast<float*>(base + lay.master);
        float* am = reinterpret_cast<float*>(base + lay.exp_avg);
        float* av = reinterpret_cast<float*>(base + lay.exp_avg_sq);
        for (int64_t i = 0; i < n; ++i) {
            ap[i] = static_cast<float>(rnd() % 20000) * 1e-6f - 0.01f;
            am[i] = 1e-4f;
            av[i] = 1e-8f;
        }
        for (int s = 1; s <= K; ++s) {
            auto* g = reinterpret_cast<uint16_t*>(base + goff[s - 1]);
            for (int64_t i = 0; i < bounds[s - 1]; ++i) g[i] = static_cast<uint16_t>(0x3A00 + rnd() % 0x300);
        }
        std::vector<float> p1(n), m1(n), v1(n), p4(n), m4(n), v4(n);
        std::vector<uint16_t> w1(n), w4(n);
        std::string err;
        gockpt_ckpt_meta meta;
        CHECK(gockpt::replay_window(K, bounds, n, base, lay.total, 0, 2, hp, kind, p1.data(), m1.data(), v1.data(),
                                    w1.data(), &meta, 1, 0, err) == GOCKPT_OK);
        CHECK(gockpt::replay_window(K, bounds, n, base, lay.total, 0, 2, hp, kind, p4.data(), m4.data(), v4.data(),
                                    w4.data(), &meta, 4, 0, err) == GOCKPT_OK);
        CHECK(memcmp(p1.data(), p4.data(), n * 4) == 0 && memcmp(v1.data(), v4.data(), n * 4) == 0);
        CHECK(memcmp(w1.data(), w4.data(), n * 2) == 0 && meta.skipped == 1);
        CHECK(gockpt::replay_window(K, bounds, n, base, lay.total - 256, 0, 2, hp, kind, p4.data(), m4.data(),
                                    v4.data(), w4.data(), &meta, 2, 0, err) == GOCKPT_ENOMEM);
    }
}

// The streaming copy of landed staging slots: every destination alignment
// and a spread of lengths (below, at and above the streaming threshold, with
// ragged tails) give exactly memcpy's bytes and touch nothing around them.
static void arena_copy() {
    std::vector<uint8_t> src(70000), a(70100), b(70100);
    for (auto& x : src) x = static_cast<uint8_t>(rnd());
    const size_t lens[] = {0, 1, 31, 255, 256, 287, 300, 4096, 4097, 65536 + 77, 69000};
    for (size_t off = 0; off < 40; ++off)
        for (size_t len : lens) {
            memset(a.data(), 0xA5, a.size());
            memset(b.data(), 0xA5, b.size());
            gockpt::copy_to_arena(a.data() + off, src.data() + (off * 7) % 64, len);
            memcpy(b.data() + off, src.data() + (off * 7) % 64, len);
            CHECK(memcmp(a.data(), b.data(), a.size()) == 0);
        }
}

int main(int argc, char** argv) {
    if (argc != 2) return 2;
    arena_copy();
    planner();
    persistence(argv[1]);
    replay();
    printf("host sanitizer driver: ok\n");
    return 0;
}
