"""Plain-Python oracle of the serving-side algorithms of the pre-gated MoE
(Read-ME, arXiv 2410.19123, Sec. 4): expert-aware batching (Alg. 1) and
expert-cache replacement (the Belady-inspired policy of Sec. 4.1, with LRU,
FIFO and random replacement as the baselines it is compared with).

TEST INFRASTRUCTURE.  Only the test suite and the CPU-baseline leg of
bench.py use this module; the library never does, and nothing here calls
the library.  Plain loops over Python lists, written for checking by eye.
"""
from __future__ import annotations

INF = float("inf")


def expert_batch(queues, max_tokens: int):
    """Alg. 1: fill one batch of at most max_tokens tokens from per-expert
    FIFO queues, taking whole queues longest first.

    Readings (the listing indexes the queue with its loop variable after
    choosing E; it loops forever once every queue is empty): the queue used
    is expert E's; the loop stops when the longest queue is empty; ties in
    the argmax go to the lowest expert index; lengths count tokens.
    Returns (batch, taken, visited): the token ids in batch order, how many
    tokens were taken from the front of each queue, and the experts whose
    tokens entered the batch, in order.
    """
    lens = [len(q) for q in queues]
    taken = [0] * len(queues)
    batch, visited = [], []
    while True:
        e = 0
        for j in range(1, len(lens)):
            if lens[j] > lens[e]:
                e = j
        if not lens or lens[e] == 0:
            break
        room = max_tokens - len(batch)
        if room <= 0:
            break
        q = queues[e][taken[e]:]
        visited.append(e)
        if lens[e] < room:
            batch.extend(q)
            taken[e] += lens[e]
            lens[e] = 0
        else:
            batch.extend(q[:room])
            taken[e] += room
            lens[e] -= room
            break
    return batch, taken, visited


def splitmix64(state: int):
    """One step of SplitMix64 (Steele, Lea and Flood, OOPSLA 2014):
    returns (new state, 64-bit output)."""
    m = (1 << 64) - 1
    state = (state + 0x9E3779B97F4A7C15) & m
    z = state
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & m
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & m
    return state, z ^ (z >> 31)


def cache_simulate(refs, capacity: int, policy: str, seed: int = 0):
    """Demand cache of `capacity` entries over the reference sequence `refs`
    (integer keys, e.g. layer * E + expert).  A reference hits if its key is
    cached; a miss inserts it, first evicting one entry when the cache is
    full:
      belady  the cached key whose next reference lies farthest in the
              future (never again = infinitely far), lowest key on ties --
              the replacement rule of Sec. 4.1, exact here because pre-gating
              makes the future references known;
      lru     the least recently referenced key;
      fifo    the earliest inserted key;
      random  the cached keys in ascending order, index r mod size, r the
              next SplitMix64 output from `seed`.
    Returns (hits, evicted): per reference, hit or not, and the evicted key
    (-1 if none).
    """
    if capacity < 1:
        raise ValueError("capacity must be positive")
    n = len(refs)
    cache = []            # cached keys
    last_use = {}
    inserted = {}
    hits, evicted = [], []
    state = seed
    for t in range(n):
        key = refs[t]
        if key in cache:
            hits.append(True)
            evicted.append(-1)
            last_use[key] = t
            continue
        hits.append(False)
        victim = -1
        if len(cache) == capacity:
            if policy == "belady":
                best, best_next = None, -1
                for c in sorted(cache):
                    nxt = INF
                    for u in range(t + 1, n):
                        if refs[u] == c:
                            nxt = u
                            break
                    if nxt > best_next:
                        best, best_next = c, nxt
                victim = best
            elif policy == "lru":
                victim = min(cache, key=lambda c: last_use[c])
            elif policy == "fifo":
                victim = min(cache, key=lambda c: inserted[c])
            elif policy == "random":
                state, r = splitmix64(state)
                victim = sorted(cache)[r % len(cache)]
            else:
                raise ValueError(f"unknown policy {policy}")
            cache.remove(victim)
        cache.append(key)
        inserted[key] = t
        last_use[key] = t
        evicted.append(victim)
    return hits, evicted


def offload_plan(counts_per_step, E: int, L: int, slots: int, policy: str,
                 lookahead: bool = True):
    """Placement plan of the expert-offload executor (Sec. 4.1): a device
    cache of `slots` (layer, expert) entries, key = layer * E + expert.

    Step s references, for every layer l = 0 .. L-1 in order, the key of
    every expert with tokens that step (ascending expert index).  A hit
    reuses the key's slot.  A miss takes the lowest-numbered empty slot;
    when none is empty it evicts, among the slots that step s has NOT used
    at layer l or at layer l-1 (the executor copies layer l's experts
    before layer l-1's kernels run, so those slots are still to be read):
      belady  the key whose next reference is farthest ahead (never again
              = farthest; lowest key on ties), the references being the
              rest of step s and then, with lookahead, step s+1's;
      lru     the least recently referenced key.
    A step with more than slots / 2 experts with tokens cannot be placed
    (two layers' experts must fit at once): ValueError.

    Returns one (hit, slot, evicted key or -1) per reference, in order.
    """
    slot_key = [-1] * slots      # key held by each slot
    slot_layer = [-1] * slots    # layer of the slot's last use
    slot_step = [-1] * slots     # step of that use
    last_ref = {}                # key -> time of its last reference (lru)
    clock = 0
    out = []
    for s, counts in enumerate(counts_per_step):
        active = [e for e in range(E) if counts[e] > 0]
        if 2 * len(active) > slots:
            raise ValueError("the cache cannot hold two layers' experts")
        nxt = []
        if lookahead and s + 1 < len(counts_per_step):
            nxt = [e for e in range(E) if counts_per_step[s + 1][e] > 0]
        refs = [l * E + e for l in range(L) for e in active]
        refs += [l * E + e for l in range(L) for e in nxt]
        pos = 0
        for l in range(L):
            for e in active:
                key = l * E + e
                clock += 1
                if key in slot_key:
                    q = slot_key.index(key)
                    out.append((True, q, -1))
                else:
                    victim = -1
                    empty = [q for q in range(slots) if slot_key[q] < 0]
                    if empty:
                        q = empty[0]
                    else:
                        best = None      # (value, key, slot); larger value = better victim
                        for c in range(slots):
                            if slot_step[c] == s and slot_layer[c] in (l, l - 1):
                                continue
                            k = slot_key[c]
                            if policy == "belady":
                                value = INF
                                for u in range(pos + 1, len(refs)):
                                    if refs[u] == k:
                                        value = u
                                        break
                            elif policy == "lru":
                                value = -last_ref[k]
                            else:
                                raise ValueError(f"unknown policy {policy}")
                            if best is None or value > best[0] or (value == best[0] and k < best[1]):
                                best = (value, k, c)
                        q = best[2]
                        victim = slot_key[q]
                    slot_key[q] = key
                    out.append((False, q, victim))
                slot_layer[q] = l
                slot_step[q] = s
                last_ref[key] = clock
                pos += 1
    return out
