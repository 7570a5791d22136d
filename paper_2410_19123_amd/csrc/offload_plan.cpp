// Placement planner of the expert-offload executor (Sec. 4.1), host code;
// the rules are stated in offload_plan.hpp.  Used by the executor
// (offload.hip) and exported on its own as readme_offload_plan, so the
// decisions can be checked on a machine without a GPU.
#include "offload_plan.hpp"

#include <algorithm>
#include <limits>

namespace readme {

void OffloadCache::init(int E_, int L_, int slots_, int policy_) {
    E = E_;
    L = L_;
    slots = slots_;
    policy = policy_;
    clock = 0;
    step = 0;
    clear();
}

void OffloadCache::clear() {
    slot_key.assign(slots, -1);
    slot_layer.assign(slots, -1);
    slot_step.assign(slots, -1);
    where.clear();
    last_ref.clear();
}

readme_status offload_plan_step(OffloadCache& cache, const int32_t* counts,
                                const int32_t* next_counts, std::vector<OffloadRef>& out) {
    const int E = cache.E, L = cache.L;
    out.clear();
    if (!counts) return README_ERR_ARG;
    std::vector<int32_t> active, next_active;
    for (int e = 0; e < E; ++e) {
        if (counts[e] < 0 || (next_counts && next_counts[e] < 0)) return README_ERR_ARG;
        if (counts[e] > 0) active.push_back(e);
        if (next_counts && next_counts[e] > 0) next_active.push_back(e);
    }
    const int A = (int)active.size();
    if (2 * A > cache.slots) return README_ERR_UNSUPPORTED;

    // The step's references, then the look-ahead; per key its positions.
    std::vector<int32_t> refs;
    for (int l = 0; l < L; ++l)
        for (int e : active) refs.push_back(l * E + e);
    for (int l = 0; l < L; ++l)
        for (int e : next_active) refs.push_back(l * E + e);
    const int64_t NEVER = std::numeric_limits<int64_t>::max();
    std::unordered_map<int32_t, std::vector<int64_t>> uses;
    for (int64_t t = 0; t < (int64_t)refs.size(); ++t) uses[refs[t]].push_back(t);
    auto next_use = [&](int32_t key, int64_t after) {
        auto it = uses.find(key);
        if (it == uses.end()) return NEVER;
        auto p = std::upper_bound(it->second.begin(), it->second.end(), after);
        return p == it->second.end() ? NEVER : *p;
    };

    OffloadCache c = cache;  // planned on a copy, committed at the end
    const int64_t step = c.step;
    int64_t pos = 0;
    for (int l = 0; l < L; ++l) {
        for (int e : active) {
            const int32_t key = l * E + e;
            ++c.clock;
            OffloadRef r{l, e, -1, -1, -1, false};
            auto it = c.where.find(key);
            if (it != c.where.end()) {
                r.slot = it->second;
                r.hit = true;
            } else {
                for (int32_t q = 0; q < c.slots && r.slot < 0; ++q)
                    if (c.slot_key[q] < 0) r.slot = q;
                if (r.slot < 0) {
                    int64_t best = -1;
                    int32_t best_key = 0;
                    for (int32_t q = 0; q < c.slots; ++q) {
                        if (c.slot_step[q] == step &&
                            (c.slot_layer[q] == l || c.slot_layer[q] == l - 1))
                            continue;  // read by a layer whose kernels are not enqueued yet
                        const int32_t k = c.slot_key[q];
                        const int64_t v = c.policy == README_CACHE_BELADY
                                              ? next_use(k, pos)         // farthest ahead
                                              : NEVER - c.last_ref[k];   // least recent
                        if (v > best || (v == best && k < best_key)) {
                            best = v;
                            best_key = k;
                            r.slot = q;
                        }
                    }
                    // Unreachable with 2 * A <= slots (see the header); kept
                    // so that a broken invariant fails without a state change.
                    if (r.slot < 0) return README_ERR_UNSUPPORTED;
                    r.evicted = c.slot_key[r.slot];
                    c.where.erase(r.evicted);
                    c.last_ref.erase(r.evicted);
                }
                r.wait_layer = c.slot_layer[r.slot];
                c.slot_key[r.slot] = key;
                c.where[key] = r.slot;
            }
            c.slot_layer[r.slot] = l;
            c.slot_step[r.slot] = step;
            c.last_ref[key] = c.clock;
            out.push_back(r);
            ++pos;
        }
    }
    ++c.step;
    cache = std::move(c);
    return README_OK;
}

}  // namespace readme

extern "C" {

readme_status readme_offload_plan(int32_t E, int32_t L, int32_t slots, int32_t policy,
                                  int32_t n_steps, const int32_t* counts, int32_t lookahead,
                                  int64_t max_refs, uint8_t* hits, int32_t* slot,
                                  int32_t* evicted, int64_t* n_refs) {
    using namespace readme;
    if (E < 1 || E > README_MAX_EXPERTS || L < 1 || slots < 1 || n_steps < 0 || max_refs < 0 ||
        !n_refs)
        return README_ERR_ARG;
    if (policy != README_CACHE_BELADY && policy != README_CACHE_LRU) return README_ERR_ARG;
    if (n_steps > 0 && !counts) return README_ERR_ARG;
    if (max_refs > 0 && (!hits || !slot || !evicted)) return README_ERR_ARG;
    *n_refs = 0;
    OffloadCache cache;
    cache.init(E, L, slots, policy);
    std::vector<OffloadRef> plan;
    int64_t n = 0;
    for (int32_t s = 0; s < n_steps; ++s) {
        const int32_t* cur = counts + (int64_t)s * E;
        const int32_t* nxt = lookahead && s + 1 < n_steps ? cur + E : nullptr;
        const readme_status st = offload_plan_step(cache, cur, nxt, plan);
        if (st != README_OK) return st;
        if (n + (int64_t)plan.size() > max_refs) return README_ERR_WORKSPACE;
        for (const OffloadRef& r : plan) {
            hits[n] = r.hit ? 1 : 0;
            slot[n] = r.slot;
            evicted[n] = r.evicted;
            ++n;
        }
        *n_refs = n;
    }
    return README_OK;
}

}  // extern "C"
