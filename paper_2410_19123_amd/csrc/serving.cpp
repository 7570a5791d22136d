// Serving-side scheduling of the pre-gated MoE (Sec. 4), host code: the
// expert-aware batching of Alg. 1 and expert-cache replacement (the
// Belady-inspired rule of Sec. 4.1, with LRU, FIFO and random replacement as
// baselines).  Pre-gating makes every token's expert known before the
// layers run, so a batch can be formed around few experts and the cache can
// look at the exact future references.
#include <stdint.h>

#include <algorithm>
#include <limits>
#include <set>
#include <unordered_map>
#include <utility>
#include <vector>

#include "readme.h"

namespace {

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): one step.
inline uint64_t splitmix64(uint64_t& state) {
    state += 0x9E3779B97F4A7C15ull;
    uint64_t z = state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

}  // namespace

extern "C" {

readme_status readme_expert_batch(int32_t E, const int32_t* queue_offsets,
                                  const int32_t* queue_items, int64_t max_tokens, int32_t* batch,
                                  int64_t* batch_len, int32_t* taken, int32_t* visited,
                                  int32_t* n_visited) {
    if (E < 1 || !queue_offsets || !batch_len || !taken || !visited || !n_visited)
        return README_ERR_ARG;
    if (max_tokens < 0) return README_ERR_ARG;
    std::vector<int64_t> len(E);
    for (int32_t e = 0; e < E; ++e) {
        len[e] = (int64_t)queue_offsets[e + 1] - queue_offsets[e];
        if (len[e] < 0) return README_ERR_ARG;
        taken[e] = 0;
    }
    if (queue_offsets[E] > 0 && !queue_items) return README_ERR_ARG;
    if (max_tokens > 0 && !batch) return README_ERR_ARG;
    int64_t n = 0;
    int32_t nv = 0;
    for (;;) {
        int32_t e = 0;  // longest queue, lowest index on ties
        for (int32_t j = 1; j < E; ++j)
            if (len[j] > len[e]) e = j;
        if (len[e] == 0) break;                // every queue empty
        const int64_t room = max_tokens - n;
        if (room <= 0) break;                  // batch full
        const int32_t* q = queue_items + queue_offsets[e] + taken[e];
        visited[nv++] = e;
        const int64_t m = len[e] < room ? len[e] : room;
        std::copy(q, q + m, batch + n);
        n += m;
        taken[e] += (int32_t)m;
        len[e] -= m;
        if (m == room) break;                  // the batch is full: a queue split or an exact fit
    }
    *batch_len = n;
    *n_visited = nv;
    return README_OK;
}

readme_status readme_cache_simulate(int32_t policy, int64_t capacity, int64_t n,
                                    const int32_t* refs, uint64_t seed, uint8_t* hits,
                                    int32_t* evicted, int64_t* n_hits) {
    if (capacity < 1 || n < 0 || !n_hits) return README_ERR_ARG;
    if (policy < README_CACHE_BELADY || policy > README_CACHE_RANDOM) return README_ERR_ARG;
    if (n > 0 && (!refs || !hits || !evicted)) return README_ERR_ARG;
    for (int64_t t = 0; t < n; ++t)
        if (refs[t] < 0) return README_ERR_ARG;
    const int64_t NEVER = std::numeric_limits<int64_t>::max();
    // Next reference of the same key after each position (Belady's future).
    std::vector<int64_t> next(n);
    {
        std::unordered_map<int32_t, int64_t> seen;
        for (int64_t t = n - 1; t >= 0; --t) {
            auto it = seen.find(refs[t]);
            next[t] = it == seen.end() ? NEVER : it->second;
            seen[refs[t]] = t;
        }
    }
    // Per cached key its ordering value: next use (Belady), last use (LRU),
    // insertion time (FIFO); the ordered set gives the victim in O(log C).
    std::unordered_map<int32_t, int64_t> val;
    std::set<std::pair<int64_t, int32_t>> order;  // (value, key) or (value, -key)
    std::set<int32_t> keys;                        // cached keys, ascending
    uint64_t state = seed;
    int64_t nh = 0;
    auto entry = [&](int32_t key, int64_t v) {
        return policy == README_CACHE_BELADY ? std::make_pair(v, -key) : std::make_pair(v, key);
    };
    for (int64_t t = 0; t < n; ++t) {
        const int32_t key = refs[t];
        auto it = val.find(key);
        if (it != val.end()) {
            hits[t] = 1;
            evicted[t] = -1;
            ++nh;
            if (policy == README_CACHE_BELADY || policy == README_CACHE_LRU) {
                order.erase(entry(key, it->second));
                it->second = policy == README_CACHE_BELADY ? next[t] : t;
                order.insert(entry(key, it->second));
            }
            continue;
        }
        hits[t] = 0;
        int32_t victim = -1;
        if ((int64_t)keys.size() == capacity) {
            if (policy == README_CACHE_BELADY) {
                // Farthest next use; among equals the lowest key (largest -key).
                victim = -std::prev(order.end())->second;
            } else if (policy == README_CACHE_RANDOM) {
                const uint64_t r = splitmix64(state);
                auto k = keys.begin();
                std::advance(k, (int64_t)(r % keys.size()));
                victim = *k;
            } else {
                victim = order.begin()->second;  // oldest use / oldest insertion
            }
            order.erase(entry(victim, val[victim]));
            val.erase(victim);
            keys.erase(victim);
        }
        const int64_t v = policy == README_CACHE_BELADY ? next[t] : t;
        val[key] = v;
        order.insert(entry(key, v));
        keys.insert(key);
        evicted[t] = victim;
    }
    *n_hits = nh;
    return README_OK;
}

}  // extern "C"
