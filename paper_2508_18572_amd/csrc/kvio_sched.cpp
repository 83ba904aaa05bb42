// kvio_sched.cpp -- cache-aware batch formation (Strata Sec. 4.3): deferral
// on delay hit and Balanced Batch Formation (Algorithm 1), host code behind
// the C ABI.  Bundle hits are found through a per-context index of the
// queue, so a round costs O(n) expected instead of a queue scan per join.
#include <math.h>
#include <stdint.h>

#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "kvio.h"

namespace {

// Token sums are kept in 128 bits: n requests of up to 2^63 tokens each
// cannot overflow them, and the loading-bound test converts them to double
// (rounding to nearest) as the definition does.
struct Batch {
    __int128 load = 0;
    __int128 compute = 0;
    int32_t count = 0;
    std::unordered_set<int64_t> contexts;
};

}  // namespace

kvio_status kvio_sched_fail(kvio_status st, const char *msg);   // kvio_api.cpp

extern "C" kvio_status kvio_schedule_round(const kvio_request *queue, int32_t n, const kvio_batch_policy *policy,
                                           int32_t *batch, int32_t *n_batch, int32_t *next_queue,
                                           int32_t *n_next) {
    if (policy == nullptr || n_batch == nullptr || n_next == nullptr || n < 0)
        return kvio_sched_fail(KVIO_EINVAL, "kvio_schedule_round: null argument or n < 0");
    if (n > 0 && (queue == nullptr || batch == nullptr || next_queue == nullptr))
        return kvio_sched_fail(KVIO_EINVAL, "kvio_schedule_round: null array");
    if (policy->max_tokens < 1 || policy->max_requests < 1 || policy->reserved != 0 ||
        policy->loading_bound_ratio < 0 || isnan(policy->loading_bound_ratio))
        return kvio_sched_fail(KVIO_EINVAL, "kvio_schedule_round: bad policy");
    for (int32_t i = 0; i < n; ++i)
        if (queue[i].load_tokens < 0 || queue[i].compute_tokens < 0 || queue[i].transient_matches < 0)
            return kvio_sched_fail(KVIO_EINVAL, "kvio_schedule_round: negative token count");
    const double ratio = policy->loading_bound_ratio > 0 ? policy->loading_bound_ratio : 100.0;
    const int64_t threshold = policy->delay_hit_threshold >= 0 ? policy->delay_hit_threshold : 100;

    // 1. deferral on delay hit
    std::vector<int32_t> deferred, eligible;
    deferred.reserve(size_t(n));
    eligible.reserve(size_t(n));
    for (int32_t i = 0; i < n; ++i)
        (queue[i].transient_matches > threshold ? deferred : eligible).push_back(i);

    // 2. balanced batch formation over the eligible requests
    std::vector<char> queued(size_t(n), 0);
    std::unordered_map<int64_t, std::vector<int32_t>> by_context;
    for (int32_t i : eligible) {
        queued[size_t(i)] = 1;
        if (queue[i].context >= 0) by_context[queue[i].context].push_back(i);
    }
    Batch B;
    int32_t nb = 0;
    auto is_bundle_hit = [&](int32_t i) {
        return queue[i].context >= 0 && B.contexts.count(queue[i].context) != 0;
    };
    auto is_full = [&]() { return B.compute >= policy->max_tokens || B.count >= policy->max_requests; };
    auto loading_bound = [&](int32_t i) {
        const __int128 load = B.load + (is_bundle_hit(i) ? 0 : queue[i].load_tokens);
        const __int128 compute = B.compute + queue[i].compute_tokens;
        return double(load) > ratio * double(compute);
    };
    auto add = [&](int32_t i) {
        if (!is_bundle_hit(i)) B.load += queue[i].load_tokens;
        B.compute += queue[i].compute_tokens;
        B.count += 1;
        if (queue[i].context >= 0) B.contexts.insert(queue[i].context);
        queued[size_t(i)] = 0;
        batch[nb++] = i;
    };
    auto add_bundle_hits = [&](int32_t i) {     // every queued request sharing i's context
        if (queue[i].context < 0) return;
        for (int32_t j : by_context[queue[i].context])
            if (queued[size_t(j)]) add(j);
    };
    std::vector<int32_t> deprioritized;
    size_t pos = 0;
    auto pop_front = [&]() -> int32_t {
        while (pos < eligible.size() && !queued[size_t(eligible[pos])]) ++pos;
        if (pos == eligible.size()) return -1;
        const int32_t i = eligible[pos++];
        queued[size_t(i)] = 0;
        return i;
    };
    const int32_t head = pop_front();
    if (head >= 0) {
        add(head);
        add_bundle_hits(head);
        while (!is_full()) {
            const int32_t r = pop_front();
            if (r < 0) break;
            if (loading_bound(r)) {
                deprioritized.push_back(r);
            } else {
                add(r);
                add_bundle_hits(r);
            }
        }
        for (int32_t r : deprioritized) {
            if (is_full()) break;
            add(r);
        }
    }
    // 3. the next round's queue: deferred first, then everything not batched
    std::vector<char> taken(size_t(n), 0);
    for (int32_t k = 0; k < nb; ++k) taken[size_t(batch[k])] = 1;
    int32_t nn = 0;
    for (int32_t i : deferred) next_queue[nn++] = i;
    for (int32_t i : eligible)
        if (!taken[size_t(i)]) next_queue[nn++] = i;
    *n_batch = nb;
    *n_next = nn;
    return KVIO_OK;
}
