"""Pins of the oracle's top-K layer (Eq. 2 with K > 1: each token's K
highest-logit experts, outputs summed with gate weights).

Checked against: the top-1 router and layer (K = 1 must reproduce them bit
for bit), a sort-based selection and math.exp weights per token, numpy's
softmax when K = E, forced ties and NaN logits, a pure-Python brute force of
the whole layer on tiny inputs, and identical experts (the renormalised
weights sum to one, so the layer then equals one expert's FFN).
"""
import math

import numpy as np
import pytest

from paper_2410_19123_amd import workloads as wl


def test_k1_is_top1_layer(oracle_mod):
    w = wl.Workload("t", T=40, d=64, E=5, I=32, dtype="bf16", bias="zipf1")
    x = wl.make_x(w, 2)
    wr, b = wl.make_router(w, 2)
    wg, wu, wd = wl.make_experts(w, 2)
    one = oracle_mod.full_path(x, wr, b, wg, wu, wd)
    k1 = oracle_mod.full_path_topk(x, wr, b, wg, wu, wd, K=1)
    assert (k1["ids"][:, 0] == one["ids"]).all()
    assert (k1["weights"] == 1.0).all()
    assert (k1["perm"] == one["perm"]).all() and (k1["offsets"] == one["offsets"]).all()
    assert (k1["y"] == one["y"]).all()


def test_selection_and_weights_against_sorting(oracle_mod):
    rng = np.random.default_rng(4)
    T, E, K = 50, 7, 3
    logits = rng.standard_normal((T, E)).astype(np.float32)
    ids, wts = oracle_mod.topk(logits, K)
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-float(logits[t, e]), e))[:K]
        assert list(ids[t]) == order
        z = [math.exp(float(logits[t, e]) - float(logits[t, order[0]])) for e in order]
        for k in range(K):
            assert abs(wts[t, k] - z[k] / sum(z)) <= 1e-15
    assert np.allclose(wts.sum(axis=1), 1.0, rtol=0, atol=1e-15)


def test_k_equals_e_is_full_softmax(oracle_mod):
    rng = np.random.default_rng(5)
    logits = rng.standard_normal((20, 6)).astype(np.float32)
    ids, wts = oracle_mod.topk(logits, 6)
    for t in range(20):
        assert sorted(ids[t]) == list(range(6))
        l64 = logits[t].astype(np.float64)
        sm = np.exp(l64 - l64.max()) / np.exp(l64 - l64.max()).sum()
        assert np.allclose(wts[t], sm[ids[t]], rtol=1e-15, atol=0)


def test_ties_and_nan(oracle_mod):
    logits = np.array([[1.0, 3.0, 3.0, 2.0],       # tie at the top: index 1 first
                       [5.0, 5.0, 5.0, 5.0],       # all equal: index order
                       [np.nan, 1.0, np.nan, 0.5],  # a NaN first candidate keeps its place
                       [2.0, np.nan, 2.0, 9.0],     # a later NaN never wins
                       [0.5, np.nan, 1.0, np.nan]], np.float32)
    ids, wts = oracle_mod.topk(logits, 2)
    assert ids.tolist() == [[1, 2], [0, 1], [0, 1], [3, 0], [2, 0]]
    assert wts[0, 0] == wts[0, 1] == 0.5 and wts[1, 0] == 0.5
    # top-1 agrees with the router's own first-argmax rule
    ids1, _ = oracle_mod.topk(logits, 1)
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 4)).astype(np.float32)
    assert ids1[:, 0].tolist() == [1, 0, 0, 3, 2]
    # ... and with the router itself on real logits
    wr = rng.standard_normal((6, 4)).astype(np.float32)
    r_ids, r_logits = oracle_mod.route(x, wr, None)
    assert (oracle_mod.topk(r_logits, 1)[0][:, 0] == r_ids).all()


def test_brute_force_layer_tiny(oracle_mod):
    rng = np.random.default_rng(9)
    T, d, I, E, K = 7, 8, 5, 4, 2      # d a multiple of 4 (fp32 router chunks)
    x = rng.standard_normal((T, d)).astype(np.float32)
    wr = rng.standard_normal((E, d)).astype(np.float32)
    wg = (rng.standard_normal((E, I, d)) * 0.5).astype(np.float32)
    wu = (rng.standard_normal((E, I, d)) * 0.5).astype(np.float32)
    wd = (rng.standard_normal((E, d, I)) * 0.5).astype(np.float32)
    out = oracle_mod.full_path_topk(x, wr, None, wg, wu, wd, K=K)
    _, logits = oracle_mod.route(x, wr, None)
    for t in range(T):
        order = sorted(range(E), key=lambda e: (-float(logits[t, e]), e))[:K]
        z = [math.exp(float(logits[t, e]) - float(logits[t, order[0]])) for e in order]
        for c in range(d):
            yc = 0.0
            for k, e in enumerate(order):
                h = []
                for i in range(I):
                    g = sum(float(wg[e, i, q]) * float(x[t, q]) for q in range(d))
                    u = sum(float(wu[e, i, q]) * float(x[t, q]) for q in range(d))
                    h.append(g / (1.0 + math.exp(-g)) * u)
                yc += z[k] / sum(z) * sum(float(wd[e, c, i]) * h[i] for i in range(I))
            assert abs(out["y"][t, c] - yc) <= 1e-12 * max(1.0, abs(yc))


def test_identical_experts_give_one_expert(oracle_mod):
    w = wl.Workload("t", T=30, d=64, E=4, I=24, dtype="bf16", bias="zipf1")
    x = wl.make_x(w, 6)
    wr, b = wl.make_router(w, 6)
    wg, wu, wd = wl.make_experts(w, 6)
    wg, wu, wd = (np.repeat(a[:1], 4, axis=0) for a in (wg, wu, wd))
    y = oracle_mod.full_path_topk(x, wr, b, wg, wu, wd, K=3)["y"]
    one = oracle_mod.moe_ffn(x, np.array([0, 30, 30, 30, 30], np.int32), wg, wu, wd)
    assert np.allclose(y, one, rtol=1e-13, atol=1e-13 * np.abs(one).max())


def test_rows_subset_and_combine(oracle_mod):
    w = wl.Workload("t", T=33, d=64, E=5, I=24, dtype="bf16", bias="zipf1")
    x = wl.make_x(w, 8)
    wr, b = wl.make_router(w, 8)
    wg, wu, wd = wl.make_experts(w, 8)
    full = oracle_mod.full_path_topk(x, wr, b, wg, wu, wd, K=2)
    rows = np.array([32, 0, 17])
    part = oracle_mod.full_path_topk(x, wr, b, wg, wu, wd, K=2, rows=rows)
    assert np.allclose(part["y"], full["y"][rows], rtol=1e-15, atol=0)
    # combine() over the grouped outputs equals the path's own sum
    x_pairs = x[full["perm"] // 2]
    y_g = oracle_mod.moe_ffn(x_pairs, full["offsets"], wg, wu, wd)
    y = oracle_mod.combine(y_g, full["inv_perm"], full["weights"])
    assert np.allclose(y, full["y"], rtol=1e-14, atol=1e-14 * np.abs(y).max())
    with pytest.raises(ValueError):
        oracle_mod.topk(np.zeros((2, 3), np.float32), 4)
