// Host-only driver of the planner and the auto-wrapping planner, built with
// AddressSanitizer and UndefinedBehaviorSanitizer (no HIP runtime, no GPU).
// It runs seeded random inputs, including invalid ones, through every host
// entry point and checks the planner's invariants; any memory error, undefined
// behaviour or broken invariant ends the process with a non-zero status.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "fsdp_bucket.h"

#define CHECK(c)                                                   \
    do {                                                           \
        if (!(c)) {                                                \
            std::fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
            std::exit(1);                                          \
        }                                                          \
    } while (0)

static void planner_round(std::mt19937_64& rng) {
    std::uniform_int_distribution<int> wdist(-2, 130), pdist(-1, 66), adist(0, 5);
    const int W = wdist(rng), P = pdist(rng);
    const int A = adist(rng) == 5 ? 3 : (1 << adist(rng));   // some invalid alignments
    std::vector<int64_t> dim0(P > 0 ? P : 1), inner(P > 0 ? P : 1);
    std::uniform_int_distribution<int64_t> ndist(-1, 5000), kdist(0, 70);
    for (int p = 0; p < P; ++p) {
        dim0[p] = ndist(rng);
        inner[p] = kdist(rng) == 70 ? (int64_t(1) << 40) : kdist(rng);   // some overflow
    }
    fsdp_plan* plan = nullptr;
    const fsdp_status st = fsdp_bucket_plan(W, P, dim0.data(), inner.data(), A, &plan);
    CHECK(fsdp_status_str(st) != nullptr && fsdp_last_error() != nullptr);
    if (st != FSDP_OK) {
        CHECK(plan == nullptr);
        return;
    }
    CHECK(W >= 1 && P >= 1 && P <= FSDP_MAX_PARAMS);
    const int64_t S = fsdp_plan_chunk_elems(plan);
    CHECK(S >= 0 && S % A == 0);
    CHECK(fsdp_plan_world_size(plan) == W && fsdp_plan_num_params(plan) == P);
    int64_t end = 0;
    for (int p = 0; p < P; ++p) {
        int64_t c = -1, off = -1, L = -1;
        CHECK(fsdp_plan_param(plan, p, &c, &off, &L) == FSDP_OK);
        CHECK(c == (dim0[p] + W - 1) / W && L == c * inner[p]);
        CHECK(off % A == 0 && off >= end && off - end < A);
        end = off + L;
        int64_t rows = 0;
        for (int r = 0; r < W; ++r) {
            const int64_t n = fsdp_plan_local_rows(plan, p, r);
            CHECK(n >= 0 && n <= c);
            rows += n;
        }
        CHECK(rows == dim0[p]);
        CHECK(fsdp_plan_local_rows(plan, p, W) < 0 && fsdp_plan_local_rows(plan, p, -1) < 0);
    }
    CHECK(S >= end && S - end < A);
    CHECK(fsdp_plan_param(plan, P, nullptr, nullptr, nullptr) != FSDP_OK);
    fsdp_plan_free(plan);
    fsdp_plan_free(plan);   // a freed handle is ignored
    CHECK(fsdp_plan_chunk_elems(plan) < 0);
}

static void wrap_round(std::mt19937_64& rng) {
    std::uniform_int_distribution<int> ndist(-1, 300), small(0, 9);
    const int n = ndist(rng);
    const int m = n > 0 ? n : 1;
    std::vector<int64_t> ag(m), rs(m), mem(m);
    std::vector<double> t(m);
    std::vector<int32_t> of(m, -7);
    for (int i = 0; i < n; ++i) {
        ag[i] = small(rng) == 9 ? -1 : small(rng);
        rs[i] = small(rng);
        t[i] = small(rng) * 0.1;
        mem[i] = small(rng);
    }
    const int backward = small(rng) % 2;
    int32_t nb = -1;
    const fsdp_status st = fsdp_auto_wrap(n, backward, ag.data(), rs.data(), t.data(), mem.data(),
                                          small(rng) * 0.1, small(rng) * 0.05, 0.2, 0.1, small(rng) * 3,
                                          of.data(), &nb);
    if (st != FSDP_OK) {
        CHECK(nb == -1);
        for (int i = 0; i < m; ++i) CHECK(of[i] == -7);
        return;
    }
    CHECK(nb >= (n > 0 ? 1 : 0) && nb <= n);
    for (int i = 0; i < n; ++i) {
        CHECK(of[i] >= 0 && of[i] < nb);
        if (i == 0) CHECK(of[i] == 0);
        else CHECK(of[i] == of[i - 1] || of[i] == of[i - 1] + 1);
    }
    if (n > 0) CHECK(of[n - 1] == nb - 1);
}

int main(int argc, char** argv) {
    const int rounds = argc > 1 ? std::atoi(argv[1]) : 3000;
    std::mt19937_64 rng(20241101);
    for (int i = 0; i < rounds; ++i) {
        planner_round(rng);
        wrap_round(rng);
    }
    std::printf("ok %d rounds\n", rounds);
    return 0;
}
