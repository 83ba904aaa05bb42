// kvio_schedule_round under AddressSanitizer and UndefinedBehaviorSanitizer:
// built with g++ from kvio_sched.cpp alone (host code), driven with seeded
// random queues including huge token counts, and checked for the invariants
// every round must keep: batch and next queue partition the input, the
// deferred requests lead the next queue in order, the rest keep queue order,
// and the first eligible request is always batched.
#include <stdio.h>
#include <stdlib.h>

#include <algorithm>
#include <vector>

#include "kvio.h"

// kvio_api.cpp (which needs the HIP runtime) provides this in the library.
kvio_status kvio_sched_fail(kvio_status st, const char *) { return st; }

#define CHECK(x)                                                             \
    do {                                                                     \
        if (!(x)) {                                                          \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #x); \
            return 1;                                                        \
        }                                                                    \
    } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint64_t next_u64() {   // splitmix64
    uint64_t z = (rng_state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

int main() {
    for (int iter = 0; iter < 3000; ++iter) {
        const int32_t n = int32_t(next_u64() % 200);
        const bool huge = next_u64() % 4 == 0;
        std::vector<kvio_request> q(static_cast<size_t>(n));
        for (auto &r : q) {
            r.load_tokens = huge ? int64_t(next_u64() >> 1) : int64_t(next_u64() % 200000);
            r.compute_tokens = huge ? int64_t(next_u64() >> 1) : int64_t(next_u64() % 5000);
            r.context = next_u64() % 3 == 0 ? -1 : int64_t(next_u64() % 8);
            r.transient_matches = next_u64() % 5 == 0 ? int64_t(next_u64() % 300) : 0;
        }
        kvio_batch_policy pol = {int64_t(1 + next_u64() % 20000), int32_t(1 + next_u64() % 32), 0,
                                 double(next_u64() % 4) * 50.0, int64_t(next_u64() % 3) * 100 - 1};
        std::vector<int32_t> batch(size_t(std::max(n, 1))), nxt(size_t(std::max(n, 1)));
        int32_t nb = -1, nn = -1;
        CHECK(kvio_schedule_round(q.data(), n, &pol, batch.data(), &nb, nxt.data(), &nn) == KVIO_OK);
        CHECK(nb >= 0 && nn >= 0 && nb + nn == n);
        std::vector<int> seen(size_t(n), 0);
        for (int32_t k = 0; k < nb; ++k) CHECK(batch[size_t(k)] >= 0 && batch[size_t(k)] < n && !seen[size_t(batch[size_t(k)])]++);
        for (int32_t k = 0; k < nn; ++k) CHECK(nxt[size_t(k)] >= 0 && nxt[size_t(k)] < n && !seen[size_t(nxt[size_t(k)])]++);
        const int64_t thr = pol.delay_hit_threshold >= 0 ? pol.delay_hit_threshold : 100;
        int32_t k = 0, last = -1, first_eligible = -1;
        for (int32_t i = 0; i < n; ++i)
            if (q[size_t(i)].transient_matches > thr) { CHECK(nxt[size_t(k)] == i); ++k; }
            else if (first_eligible < 0) first_eligible = i;
        for (; k < nn; ++k) { CHECK(nxt[size_t(k)] > last && q[size_t(nxt[size_t(k)])].transient_matches <= thr); last = nxt[size_t(k)]; }
        if (first_eligible >= 0) CHECK(nb > 0 && batch[0] == first_eligible);
    }
    printf("scheduler fuzz checks passed\n");
    return 0;
}
