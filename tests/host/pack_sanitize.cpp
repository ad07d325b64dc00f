// Memory-safety check of the host planning code (pp_plan_bounds, pp_pack, pp_pack_padded),
// built with AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_pack_sanitized.py.
//
// Every plan array is its own heap allocation of exactly the size pp_plan_bounds reports (the
// contract in prepack.h), so a write one element past any of them stops the run.  Random
// batches (seeded, several length mixes, k up to 400) go through pp_pack with capacity 0, the
// maximum length and larger capacities, and through pp_pack_padded; each call is repeated with
// one capacity one element too small (it must fail with PP_ERR_BUFFER_TOO_SMALL and write
// nothing out of bounds) and with invalid arguments.  Light invariants of the results are
// checked too; the exact plans are compared with the oracle by the Python tests.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <memory>
#include <vector>

#include "prepack.h"

namespace {

// splitmix64 (Steele, Lea, Flood 2014)
struct Rng {
    uint64_t s;
    uint64_t next() {
        uint64_t z = (s += 0x9E3779B97F4A7C15ull);
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        return z ^ (z >> 31);
    }
    int32_t uniform(int32_t lo, int32_t hi) { return lo + static_cast<int32_t>(next() % uint64_t(hi - lo + 1)); }
};

int g_fail = 0;
#define CHECK(cond, ...)                                        \
    do {                                                        \
        if (!(cond)) {                                          \
            std::fprintf(stderr, "check failed: %s: ", #cond);  \
            std::fprintf(stderr, __VA_ARGS__);                  \
            std::fprintf(stderr, "\n");                         \
            ++g_fail;                                           \
        }                                                       \
    } while (0)

// One allocation per array, sized exactly; caps as given.
struct Buffers {
    std::vector<std::unique_ptr<int32_t[]>> owned;
    pp_plan plan{};
    int32_t* make(int64_t n) {
        owned.emplace_back(new int32_t[n > 0 ? n : 1]);   // n == 0: a 1-element block nothing may touch
        return owned.back().get();
    }
    Buffers(int32_t k, int64_t slot_cap, int64_t qtile_cap, int64_t mtile_cap) {
        plan.slot_cap = slot_cap;
        plan.qtile_cap = qtile_cap;
        plan.mtile_cap = mtile_cap;
        plan.row_seg_ptr = make(int64_t(k) + 1);
        plan.seg_prompt = make(k);
        plan.seg_start = make(k);
        plan.seg_len = make(k);
        plan.prompt_kv_off = make(int64_t(k) + 1);
        plan.slot_seg = make(slot_cap);
        plan.slot_pos = make(slot_cap);
        plan.slot_kv = make(slot_cap);
        plan.qtile_seg = make(qtile_cap);
        plan.qtile_q0 = make(qtile_cap);
        plan.mtile_m0 = make(mtile_cap);
    }
};

std::vector<int32_t> draw_lengths(Rng& rng, int32_t k) {
    std::vector<int32_t> l(k);
    const int mix = rng.uniform(0, 4);
    const int32_t hi = rng.uniform(1, 3000);
    for (int32_t i = 0; i < k; ++i) {
        switch (mix) {
            case 0: l[i] = rng.uniform(1, hi); break;                                  // uniform
            case 1: l[i] = hi; break;                                                  // all equal
            case 2: l[i] = rng.uniform(0, 9) == 0 ? rng.uniform(1, hi) : 1; break;      // mostly 1
            case 3: l[i] = rng.uniform(0, 4) == 0 ? rng.uniform(hi / 2 + 1, hi) : rng.uniform(1, 16); break;  // bimodal
            default: {                                                                 // heavy tail
                int32_t v = 1;
                while (v < hi && rng.uniform(0, 2) != 0) v = v * 2 + rng.uniform(0, 1);
                l[i] = v < hi ? v : hi;
            }
        }
    }
    return l;
}

// Invariants that hold for every plan (packed or padded) with row capacity C.
void check_plan(const pp_plan& p, const std::vector<int32_t>& l, int32_t C, bool padded) {
    const int32_t k = static_cast<int32_t>(l.size());
    CHECK(p.k == k, "k %d vs %d", p.k, k);
    CHECK(p.capacity == C, "capacity %d vs %d", p.capacity, C);
    CHECK(p.n_rows >= (k > 0) && p.n_rows <= k, "n_rows %d", p.n_rows);
    int64_t total = 0;
    for (int32_t i = 0; i < k; ++i) total += l[i];
    CHECK(p.total_len == total, "total_len");
    CHECK(p.prompt_kv_off[0] == 0 && p.prompt_kv_off[k] == total, "prompt_kv_off ends");
    for (int32_t i = 0; i < k; ++i) CHECK(p.prompt_kv_off[i + 1] - p.prompt_kv_off[i] == l[i], "kv span %d", i);
    const int64_t slots = int64_t(p.n_rows) * C;
    int64_t real = 0;
    for (int64_t s = 0; s < slots; ++s) {
        const int32_t seg = p.slot_seg[s];
        CHECK(seg >= -1 && seg < k, "slot_seg[%lld] = %d", (long long)s, seg);
        CHECK(p.slot_kv[s] >= -1 && p.slot_kv[s] < total, "slot_kv[%lld] = %d", (long long)s, p.slot_kv[s]);
        if (p.slot_kv[s] >= 0) ++real;
    }
    CHECK(real == total, "real slots %lld vs %lld", (long long)real, (long long)total);
    for (int32_t j = 0; j < p.n_qtiles; ++j)
        CHECK(p.qtile_seg[j] >= 0 && p.qtile_seg[j] < k && p.qtile_q0[j] >= 0 &&
                  p.qtile_q0[j] < p.seg_len[p.qtile_seg[j]] && p.qtile_q0[j] % PP_QTILE == 0,
              "qtile %d", j);
    for (int32_t j = 0; j < p.n_mtiles; ++j)
        CHECK(p.mtile_m0[j] >= 0 && p.mtile_m0[j] < slots && p.mtile_m0[j] % PP_MTILE == 0 &&
                  (j == 0 || p.mtile_m0[j] > p.mtile_m0[j - 1]),
              "mtile %d", j);
    if (padded) CHECK(p.n_rows == k, "padded rows");
}

// pp_pack (capacity >= 0) or pp_pack_padded (capacity < 0) with exact buffers, then with each
// cap one short.
void run_case(const std::vector<int32_t>& l, int32_t capacity) {
    const int32_t k = static_cast<int32_t>(l.size());
    const bool padded = capacity < 0;
    int32_t m = 0;
    for (int32_t v : l) m = v > m ? v : m;
    const int32_t C = padded || capacity == 0 ? m : capacity;
    int64_t sc = 0, qc = 0, mc = 0;
    CHECK(pp_plan_bounds(k, C, &sc, &qc, &mc) == PP_OK, "bounds: %s", pp_last_error());
    auto call = [&](Buffers& b) {
        return padded ? pp_pack_padded(l.data(), k, &b.plan) : pp_pack(l.data(), k, capacity, &b.plan);
    };
    {
        Buffers b(k, sc, qc, mc);
        const pp_status st = call(b);
        if (!padded && capacity > 0 && m > capacity) {
            CHECK(st == PP_ERR_TOO_LONG, "too long: %d", st);
            return;
        }
        CHECK(st == PP_OK, "pack k=%d capacity=%d: %s", k, capacity, pp_last_error());
        if (st == PP_OK) check_plan(b.plan, l, C, padded);
    }
    const int64_t caps[3] = {sc, qc, mc};
    for (int which = 0; which < 3; ++which) {
        if (caps[which] == 0) continue;
        Buffers b(k, sc - (which == 0), qc - (which == 1), mc - (which == 2));
        const pp_status st = call(b);
        CHECK(st == PP_ERR_BUFFER_TOO_SMALL, "cap %d one short: status %d", which, st);
    }
}

}  // namespace

int main(int argc, char** argv) {
    const int iters = argc > 1 ? std::atoi(argv[1]) : 2000;
    Rng rng{20240409};
    long calls = 0;
    for (int it = 0; it < iters; ++it) {
        const int32_t k = rng.uniform(0, 9) == 0 ? 0 : rng.uniform(1, rng.uniform(0, 3) == 0 ? 400 : 40);
        const std::vector<int32_t> l = draw_lengths(rng, k);
        int32_t m = 0;
        for (int32_t v : l) m = v > m ? v : m;
        const int32_t caps[4] = {0, m > 0 ? m : 1, m + rng.uniform(1, 5000), m > 1 ? rng.uniform(1, m - 1) : 1};
        for (int32_t c : caps) {
            run_case(l, c);
            ++calls;
        }
        run_case(l, -1);
        ++calls;
    }
    // invalid arguments: rejected without touching the plan arrays
    {
        Buffers b(4, 64, 8, 8);
        const int32_t bad[4] = {3, 0, 5, 2};
        CHECK(pp_pack(bad, 4, 0, &b.plan) == PP_ERR_INVALID_ARG, "zero length");
        const int32_t neg[2] = {4, -7};
        CHECK(pp_pack(neg, 2, 0, &b.plan) == PP_ERR_INVALID_ARG, "negative length");
        CHECK(pp_pack(nullptr, 3, 0, &b.plan) == PP_ERR_INVALID_ARG, "NULL lengths");
        CHECK(pp_pack(bad, -1, 0, &b.plan) == PP_ERR_INVALID_ARG, "negative k");
        const int32_t ok[2] = {4, 7};
        CHECK(pp_pack(ok, 2, -3, &b.plan) == PP_ERR_INVALID_ARG, "negative capacity");
        CHECK(pp_pack(ok, 2, 0, nullptr) == PP_ERR_INVALID_ARG, "NULL plan");
        CHECK(pp_pack_padded(neg, 2, &b.plan) == PP_ERR_INVALID_ARG, "padded negative length");
        int64_t s = 0, q = 0, t = 0;
        CHECK(pp_plan_bounds(-1, 4, &s, &q, &t) == PP_ERR_INVALID_ARG, "bounds k < 0");
        CHECK(pp_plan_bounds(4, -1, &s, &q, &t) == PP_ERR_INVALID_ARG, "bounds C < 0");
        CHECK(pp_plan_bounds(4, 4, nullptr, &q, &t) == PP_ERR_INVALID_ARG, "bounds NULL");
        calls += 10;
    }
    std::printf("pack_sanitize: %d batches, %ld calls, %d failed checks\n", iters, calls, g_fail);
    return g_fail == 0 ? 0 : 1;
}
