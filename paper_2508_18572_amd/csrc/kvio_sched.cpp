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

// Token sums are kept in 128 bits: n < 2^31 requests of fewer than 2^63 tokens
// each sum to less than 2^94, so they cannot overflow.
struct Batch {
    unsigned __int128 load = 0;
    unsigned __int128 compute = 0;
    int32_t count = 0;
    std::unordered_set<int64_t> contexts;
};

// Unsigned 256-bit integer, four 64-bit limbs, least significant first: wide
// enough for a token sum (< 2^94) times the 53-bit significand of the ratio.
struct U256 {
    uint64_t w[4] = {0, 0, 0, 0};
};

U256 from_u128(unsigned __int128 v) {
    U256 r;
    r.w[0] = uint64_t(v);
    r.w[1] = uint64_t(v >> 64);
    return r;
}

U256 mul_u128_u64(unsigned __int128 a, uint64_t b) {
    const unsigned __int128 lo = (unsigned __int128)uint64_t(a) * b;
    const unsigned __int128 hi = (unsigned __int128)uint64_t(a >> 64) * b + (lo >> 64);
    U256 r;
    r.w[0] = uint64_t(lo);
    r.w[1] = uint64_t(hi);
    r.w[2] = uint64_t(hi >> 64);
    return r;
}

int bit_length(const U256 &v) {
    for (int i = 3; i >= 0; --i)
        if (v.w[i] != 0) return 64 * i + 64 - __builtin_clzll(v.w[i]);
    return 0;
}

// v * 2^s; the caller keeps the result below 2^256.
U256 shl(const U256 &v, int s) {
    U256 r;
    const int limbs = s / 64, bits = s % 64;
    for (int i = 3; i >= limbs; --i) {
        uint64_t x = v.w[i - limbs] << bits;
        if (bits != 0 && i - limbs - 1 >= 0) x |= v.w[i - limbs - 1] >> (64 - bits);
        r.w[i] = x;
    }
    return r;
}

int compare(const U256 &a, const U256 &b) {
    for (int i = 3; i >= 0; --i)
        if (a.w[i] != b.w[i]) return a.w[i] < b.w[i] ? -1 : 1;
    return 0;
}

// Sec. 4.3.2: the batch is loading-bound when the ratio of its aggregated load
// to its aggregated compute exceeds the threshold.  Decided exactly as
// load > ratio * compute on the integer sums and the ratio's exact binary
// value (ratio = m * 2^k with an integer significand m < 2^53), so the
// outcome never depends on rounding: no compute and some load is
// loading-bound; an infinite ratio never is.
bool exceeds_ratio(unsigned __int128 load, unsigned __int128 compute, double ratio) {
    if (isinf(ratio)) return false;
    if (compute == 0) return load != 0;
    if (load == 0) return false;
    int e = 0;
    const double f = frexp(ratio, &e);                  // ratio = f * 2^e, f in [0.5, 1)
    const uint64_t m = uint64_t(ldexp(f, 53));          // exact: ratio = m * 2^(e - 53)
    const int k = e - 53;
    // compare A * 2^a with B * 2^b: A = load, B = m * compute
    const U256 A = from_u128(load), B = mul_u128_u64(compute, m);
    const int a = k < 0 ? -k : 0, b = k > 0 ? k : 0;
    const int la = bit_length(A) + a, lb = bit_length(B) + b;
    if (la != lb) return la > lb;
    // equal bit lengths: the shift that aligns them keeps both below 2^256
    return a >= b ? compare(shl(A, a - b), B) > 0 : compare(A, shl(B, b - a)) > 0;
}

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
    auto is_full = [&]() {
        return B.compute >= uint64_t(policy->max_tokens) || B.count >= policy->max_requests;
    };
    auto loading_bound = [&](int32_t i) {
        const unsigned __int128 load = B.load + uint64_t(is_bundle_hit(i) ? 0 : queue[i].load_tokens);
        const unsigned __int128 compute = B.compute + uint64_t(queue[i].compute_tokens);
        return exceeds_ratio(load, compute, ratio);
    };
    auto add = [&](int32_t i) {
        if (!is_bundle_hit(i)) B.load += uint64_t(queue[i].load_tokens);
        B.compute += uint64_t(queue[i].compute_tokens);
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
