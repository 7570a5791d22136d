"""Parity of the top-K layer (Eq. 2 with K > 1) on the HIP path, through the
C ABI, with the CPU oracle: expert ids and the pair grouping bit-exact, gate
weights within fp32 rounding, outputs within the tolerance of tests/_util.py,
and K = 1 equal to the top-1 layer bit for bit."""
import numpy as np
import pytest
import torch

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


def _gpu_path(L, w, K, x, wr, b, packed):
    xd = U.to_dev(x)
    ids1, logits = L.readme_route(xd, U.to_dev(wr), None if b is None else U.to_dev(b),
                                  logits=torch.empty(w.T, w.E, dtype=torch.float32,
                                                     device=U.dev()))
    ids, wts = L.readme_topk(logits, K)
    counts, offs, perm, inv, _ = L.readme_group_by_expert(ids, w.E)
    y_pairs = L.readme_moe_ffn_topk(xd, perm, offs, packed, w.E, w.I, K)
    y = L.readme_combine_topk(y_pairs, wts, K)
    torch.cuda.synchronize()
    return dict(ids=U.from_dev(ids).reshape(w.T, K), weights=U.from_dev(wts).reshape(w.T, K),
                logits=U.from_dev(logits), offsets=U.from_dev(offs), perm=U.from_dev(perm),
                y_pairs=U.from_dev(y_pairs), y=U.from_dev(y))


@pytest.mark.parametrize("name,K", [("llama7b_layer_top2", 2), ("prefill_skew16", 4)])
def test_topk_selection_bit_exact(L, oracle_mod, name, K):
    w = wl.WORKLOADS[name]
    _say("topk selection", name, K)
    x = wl.make_x(w)
    wr, b = wl.make_router(w)
    _, logits = L.readme_route(U.to_dev(x), U.to_dev(wr), U.to_dev(b),
                               logits=torch.empty(w.T, w.E, dtype=torch.float32, device=U.dev()))
    ids, wts = L.readme_topk(logits, K)
    torch.cuda.synchronize()
    ref_ids, ref_w = oracle_mod.topk(oracle_mod.route(x, wr, b)[1], K)
    assert (U.from_dev(ids).reshape(-1, K) == ref_ids).all()
    assert np.allclose(U.from_dev(wts).reshape(-1, K), ref_w, rtol=2e-6, atol=1e-7)


def test_topk_ties_and_nan(L, oracle_mod):
    logits = np.array([[1.0, 3.0, 3.0, 2.0, 0.0],
                       [5.0, 5.0, 5.0, 5.0, 5.0],
                       [np.nan, 1.0, np.nan, 0.5, 2.0],
                       [2.0, np.nan, 2.0, 9.0, -np.inf],
                       [-1e30, -1e30, 7.0, 7.0, -0.0]], np.float32)
    for K in (1, 2, 3, 5):
        ids, wts = L.readme_topk(U.to_dev(logits), K)
        torch.cuda.synchronize()
        ref_ids, ref_w = oracle_mod.topk(logits, K)
        assert (U.from_dev(ids).reshape(-1, K) == ref_ids).all(), K
        finite = np.isfinite(ref_w).all(axis=1)
        got = U.from_dev(wts).reshape(-1, K)
        assert np.allclose(got[finite], ref_w[finite], rtol=2e-6, atol=1e-7), K


def test_topk_layer_full_workload(L, oracle_mod):
    """route -> top-2 -> pair grouping -> FFN -> combine at full size, every
    token."""
    w = wl.WORKLOADS["llama7b_layer_top2"]
    _say("topk layer", w.name)
    x = wl.make_x(w)
    wr, b = wl.make_router(w)
    wg, wu, wd = wl.make_experts(w)
    packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
    got = _gpu_path(L, w, w.K, x, wr, b, packed)
    ref_ids, _ = oracle_mod.topk(oracle_mod.route(x, wr, b)[1], w.K)
    _, offsets, perm, inv = oracle_mod.group(ref_ids.reshape(-1), w.E)
    assert (got["ids"] == ref_ids).all()
    assert (got["offsets"] == offsets).all() and (got["perm"] == perm).all()
    ref = oracle_mod.full_path_topk(x, wr, b, wg, wu, wd, K=w.K)
    U.close(got["y"], ref["y"], w.name)


@pytest.mark.parametrize("tile", [0, 1, 6, 12, 15, 17, 21, 24, 27, 30, 31])
def test_topk_layer_tiles(L, oracle_mod, tile):
    """All rows of a small ragged top-3 layer, through the LDS-staged and the
    register-streamed GEMM kernels (the pair -> token gather in each)."""
    _say("topk tile", tile)
    L.readme_set_gemm_tile(tile)
    try:
        w = wl.Workload("t", T=300, d=256, E=6, I=160, K=3, dtype="bf16", bias="zipf1")
        x = wl.make_x(w, 40 + tile)
        wr, b = wl.make_router(w, 40 + tile)
        wg, wu, wd = wl.make_experts(w, 40 + tile)
        packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
        got = _gpu_path(L, w, 3, x, wr, b, packed)
        ref = oracle_mod.full_path_topk(x, wr, b, wg, wu, wd, K=3)
        assert (got["ids"] == ref["ids"]).all()
        U.close(got["y"], ref["y"], f"tile {tile}")
    finally:
        L.readme_set_gemm_tile(0)


def test_topk_fp32(L, oracle_mod):
    w = wl.Workload("t", T=256, d=512, E=4, I=512, K=2, dtype="f32")
    x = wl.make_x(w, 3)
    wr, b = wl.make_router(w, 3)
    wg, wu, wd = wl.make_experts(w, 3)
    packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
    got = _gpu_path(L, w, 2, x, wr, b, packed)
    ref = oracle_mod.full_path_topk(x, wr, b, wg, wu, wd, K=2)
    assert (got["ids"] == ref["ids"]).all()
    U.close(got["y"], ref["y"], "fp32 top-2")


def test_k1_equals_top1_layer(L):
    """K = 1: weight 1, pairs = tokens, so the top-K path gives the fused
    top-1 layer's bits."""
    w = wl.WORKLOADS["llama7b_layer"]
    x = U.to_dev(wl.make_x(w))
    wr, b = wl.make_router(w)
    packed = L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w)))
    ids1, logits = L.readme_route(x, U.to_dev(wr), U.to_dev(b),
                                  logits=torch.empty(w.T, w.E, dtype=torch.float32,
                                                     device=U.dev()))
    ids, wts = L.readme_topk(logits, 1)
    counts, offs, perm, inv, _ = L.readme_group_by_expert(ids, w.E)
    y_k = L.readme_combine_topk(L.readme_moe_ffn_topk(x, perm, offs, packed, w.E, w.I, 1), wts, 1)
    c1, o1, p1, i1, _ = L.readme_group_by_expert(ids1, w.E)
    y_1 = L.readme_moe_ffn_fused(x, p1, o1, packed, w.E, w.I)
    torch.cuda.synchronize()
    assert (U.from_dev(ids) == U.from_dev(ids1)).all()
    assert (U.from_dev(wts) == 1.0).all()
    assert (U.from_dev(y_k) == U.from_dev(y_1)).all()
