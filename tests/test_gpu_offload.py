"""The expert-offload executor (Sec. 4.1) through the C ABI: the layer stack
computed with weights fetched into a small device cache of (layer, expert)
slots equals the resident stack bit for bit and the oracle's layer chain
within tolerance, step after step, under both replacement policies; every
step's placement equals the oracle's plan; its counters add up."""
import numpy as np
import pytest
import torch

from oracle import serving as S
from paper_2410_19123_amd import workloads as wl

from . import _util as U

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2410_19123_amd import _lib
    _lib.load()
    return _lib


def _say(*a):
    print(*a, flush=True)


def _oracle_chain(oracle_mod, x0, offsets, host_layers, eps=1e-5):
    """x <- x + F_l(RMSNorm(x)) layer by layer in the oracle, the residual
    rounded to fp32 after each layer as the stack keeps it."""
    x = x0.astype(np.float32)
    for wts in host_layers:
        x = (x.astype(np.float64) + np.pad(oracle_mod.layer(x, offsets, *wts, eps=eps),
                                           ((0, x.shape[0] - int(offsets[-1])), (0, 0))))
        x = x.astype(np.float32)
    return x


@pytest.mark.parametrize("policy", ["belady", "lru"])
def test_offload_stack_equals_resident(L, oracle_mod, policy):
    w = wl.Workload("t", T=48, d=256, E=6, I=160, dtype="bf16", layers=4)
    _say("offload", policy)
    host = [wl.make_experts(w, 50, layer=l) for l in range(w.layers)]
    layers = [L.readme_pack_experts(*U.weights_to_dev(*h)) for h in host]
    slots = 8
    ex = L.Offload(layers, w.E, w.d, w.I, slots, policy)
    rng = np.random.default_rng(50)
    steps = 7
    # each step routes the tokens to 1..4 experts
    plans = []
    for _ in range(steps):
        k = int(rng.integers(1, 5))
        experts = rng.choice(w.E, size=k, replace=False)
        plans.append(rng.choice(experts, size=w.T).astype(np.int32))
    slot_bytes = 3 * L.readme_padded_intermediate(w.I) * w.d * 2
    all_counts = [np.bincount(p, minlength=w.E).tolist() for p in plans]
    want = S.offload_plan(all_counts, w.E, w.layers, slots, policy)
    refs = 0
    x0 = np.random.default_rng(51).standard_normal((w.T, w.d)).astype(np.float32)
    try:
        for st in range(steps):
            ids = U.to_dev(plans[st])
            counts, offs, perm, inv, xg = L.readme_group_by_expert(ids, w.E, x=U.to_dev(x0))
            c = np.bincount(plans[st], minlength=w.E)
            nxt = np.bincount(plans[st + 1], minlength=w.E) if st + 1 < steps else None
            xa, xb = xg.clone(), xg.clone()
            L.readme_moe_ffn_stack(xa, offs, layers, w.E, w.I)
            ex.stack(xb, offs, c, nxt)
            torch.cuda.synchronize()
            assert (U.from_dev(xa) == U.from_dev(xb)).all(), st
            n = w.layers * int((c > 0).sum())
            assert ex.last_plan() == want[refs:refs + n], st
            refs += n
            if st in (0, steps - 1):
                offsets = U.from_dev(offs)
                x_in = U.from_dev(xg)
                ref = _oracle_chain(oracle_mod, x_in, offsets, host)
                U.close(U.from_dev(xb).astype(np.float64) - x_in, ref.astype(np.float64) - x_in,
                        f"offload chain step {st}")
        hits, misses, nbytes = ex.stats()
        assert hits + misses == refs
        assert nbytes == misses * slot_bytes
        assert misses >= min(refs, slots)  # every key is loaded once at least
    finally:
        ex.close()


def test_offload_needs_two_layers_of_slots(L):
    w = wl.Workload("t", T=32, d=128, E=4, I=64, dtype="bf16", layers=2)
    layers = [L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w, 60, layer=l)))
              for l in range(w.layers)]
    ex = L.Offload(layers, w.E, w.d, w.I, 5, "belady")
    try:
        ids = U.to_dev(np.arange(w.T, dtype=np.int32) % 3)       # 3 experts need 6 slots
        counts, offs, perm, inv, xg = L.readme_group_by_expert(
            ids, w.E, x=U.to_dev(np.ones((w.T, w.d), np.float32)))
        with pytest.raises(L.ReadmeError) as e:
            ex.stack(xg, offs, np.bincount(U.from_dev(ids), minlength=w.E))
        assert e.value.status == 2
    finally:
        ex.close()


@pytest.mark.parametrize("concentrated", [True, False])
def test_stack_with_counts_equals_plain_stack(L, concentrated):
    """Host counts only change the tile choice (narrower tiles for a batch on
    few experts); every tile accumulates K in the same order, so the stack
    gives the same bits."""
    w = wl.Workload("t", T=64, d=512, E=8, I=256, dtype="bf16", layers=3)
    layers = [L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w, 70, layer=l)))
              for l in range(w.layers)]
    rng = np.random.default_rng(70)
    ids_h = (np.full(w.T, 3, np.int32) if concentrated
             else rng.integers(0, w.E, size=w.T).astype(np.int32))
    x0 = rng.standard_normal((w.T, w.d)).astype(np.float32)
    counts, offs, perm, inv, xg = L.readme_group_by_expert(U.to_dev(ids_h), w.E,
                                                           x=U.to_dev(x0))
    xa, xb = xg.clone(), xg.clone()
    L.readme_moe_ffn_stack(xa, offs, layers, w.E, w.I)
    L.readme_moe_ffn_stack(xb, offs, layers, w.E, w.I,
                           counts=np.bincount(ids_h, minlength=w.E))
    torch.cuda.synchronize()
    assert (U.from_dev(xa) == U.from_dev(xb)).all()


def test_offload_layer_keys_of_other_steps_are_evictable(L):
    """Two slots, one expert per step: at step 3, layer 1 the only slot not
    used by this step's layers 0 and 1 holds a layer-1 key of an earlier
    step, which must be evicted (a rule that protected every layer-1 key
    would find no victim).  Steps {2}, {6}, {1}, {3}, {1} with look-ahead."""
    w = wl.Workload("t", T=16, d=128, E=8, I=64, dtype="bf16", layers=3)
    layers = [L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w, 80, layer=l)))
              for l in range(w.layers)]
    seq = [2, 6, 1, 3, 1]
    counts = [[w.T if e == s else 0 for e in range(w.E)] for s in seq]
    want = S.offload_plan(counts, w.E, w.layers, 2, "belady")
    ex = L.Offload(layers, w.E, w.d, w.I, 2, "belady")
    x0 = np.random.default_rng(81).standard_normal((w.T, w.d)).astype(np.float32)
    try:
        for st, e in enumerate(seq):
            ids = U.to_dev(np.full(w.T, e, np.int32))
            _, offs, _, _, xg = L.readme_group_by_expert(ids, w.E, x=U.to_dev(x0))
            xa, xb = xg.clone(), xg.clone()
            L.readme_moe_ffn_stack(xa, offs, layers, w.E, w.I)
            ex.stack(xb, offs, counts[st], counts[st + 1] if st + 1 < len(seq) else None)
            torch.cuda.synchronize()
            assert (U.from_dev(xa) == U.from_dev(xb)).all(), st
            assert ex.last_plan() == want[3 * st:3 * st + 3], st
    finally:
        ex.close()
