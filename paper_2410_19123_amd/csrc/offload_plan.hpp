// Placement planner of the expert-offload executor (Sec. 4.1), host code.
//
// The device cache holds `slots` (layer, expert) entries, key = layer*E +
// expert.  A step references, layer by layer, the experts that have tokens
// (ascending expert index within a layer); pre-gating makes the whole
// step's references known before its first layer runs, and the caller may
// add the next step's as look-ahead.  A reference hits when its key is
// cached; a miss takes the lowest empty slot, else evicts by policy among
// the slots that may be overwritten now:
//   Belady  the key whose next reference (this step, then the look-ahead)
//           is farthest ahead, never = farthest, lowest key on ties;
//   LRU     the least recently referenced key.
// A slot may not be overwritten while placing layer l if this step used it
// at layer l (its kernels have not run yet) or at layer l-1 (the executor
// enqueues the copies of layer l before layer l-1's kernels).  With
// slots >= 2 * (experts with tokens) a candidate always exists: at most
// A-1 slots of layer l and A of layer l-1 are protected.
#pragma once

#include <stdint.h>

#include <unordered_map>
#include <vector>

#include "readme.h"

namespace readme {

struct OffloadCache {
    int E = 0, L = 0, slots = 0, policy = 0;
    std::vector<int32_t> slot_key;    // key held, -1 empty
    std::vector<int32_t> slot_layer;  // layer of the slot's last use, -1 none
    std::vector<int64_t> slot_step;   // step of that use, -1 none
    std::unordered_map<int32_t, int32_t> where;     // key -> slot
    std::unordered_map<int32_t, int64_t> last_ref;  // key -> reference clock (LRU)
    int64_t clock = 0;
    int64_t step = 0;

    void init(int E_, int L_, int slots_, int policy_);
    // Forget every cached key (the slots' contents are no longer trusted).
    void clear();
};

// One reference of a planned step, in reference order.
struct OffloadRef {
    int32_t layer, expert;
    int32_t slot;        // slot the layer reads the expert from
    int32_t evicted;     // key evicted by this reference's miss, -1 none
    int32_t wait_layer;  // layer of the overwritten slot's last use (-1 none)
    bool hit;
};

// Plans one step.  counts [E] (host): tokens per expert this step;
// next_counts [E] (host, or NULL): the next step's, for Belady's look-ahead.
// On success the cache state advances to the end of the step and `out`
// holds every reference; on any error the state is left unchanged.
// README_ERR_ARG: a negative count; README_ERR_UNSUPPORTED: fewer than
// 2 * (experts with tokens) slots.
readme_status offload_plan_step(OffloadCache& cache, const int32_t* counts,
                                const int32_t* next_counts, std::vector<OffloadRef>& out);

}  // namespace readme
