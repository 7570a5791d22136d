"""Edge cases of the HIP path against the CPU oracle: top-K with every expert
selected (K = E), top-K selection among the largest expert count with
heavy ties and NaN logits, stacks with no layers or no tokens, and a
131072-token layer over 64 experts."""
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


def test_topk_every_expert_selected(L, oracle_mod):
    """K = E: every token goes through every expert, weighted by the softmax
    of all its logits (Eq. 2 with K = E); ragged pair blocks of equal size."""
    _say("topk K = E")
    w = wl.Workload("t", T=150, d=128, E=4, I=96, dtype="bf16", bias="zipf1")
    x = wl.make_x(w, 4)
    wr, b = wl.make_router(w, 4)
    wg, wu, wd = wl.make_experts(w, 4)
    xd = U.to_dev(x)
    packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
    _, logits = L.readme_route(xd, U.to_dev(wr), U.to_dev(b),
                               logits=torch.empty(w.T, w.E, dtype=torch.float32, device=U.dev()))
    ids, wts = L.readme_topk(logits, w.E)
    counts, offs, perm, inv, _ = L.readme_group_by_expert(ids, w.E)
    y = L.readme_combine_topk(L.readme_moe_ffn_topk(xd, perm, offs, packed, w.E, w.I, w.E),
                              wts, w.E)
    torch.cuda.synchronize()
    ref = oracle_mod.full_path_topk(x, wr, b, wg, wu, wd, K=w.E)
    assert (U.from_dev(ids).reshape(w.T, w.E) == ref["ids"]).all()
    assert (U.from_dev(counts) == w.T).all()
    U.close(U.from_dev(y), ref["y"], "K = E")


@pytest.mark.parametrize("K", [1, 8])
def test_topk_selection_256_experts_ties_nan(L, oracle_mod, K):
    """E = 256 (every word of the taken-expert mask), logits drawn from five
    values so that most candidates tie, and a few NaN logits."""
    _say("topk E = 256", K)
    rng = np.random.default_rng(256 + K)
    T, E = 300, 256
    logits = rng.integers(0, 5, size=(T, E)).astype(np.float32)
    logits[rng.integers(0, T, size=40), rng.integers(0, E, size=40)] = np.nan
    ids, wts = L.readme_topk(U.to_dev(logits), K)
    torch.cuda.synchronize()
    ref_ids, ref_w = oracle_mod.topk(logits, K)
    assert (U.from_dev(ids).reshape(T, K) == ref_ids).all()
    got_w = U.from_dev(wts).reshape(T, K)
    assert np.array_equal(np.isnan(got_w), np.isnan(ref_w))
    ok = ~np.isnan(ref_w)
    assert np.allclose(got_w[ok], ref_w[ok], rtol=2e-6, atol=1e-7)


def test_stack_without_layers_or_tokens(L):
    """No layers: the residual stream is left as it was; no tokens: a valid
    call that does nothing."""
    w = wl.Workload("t", T=40, d=128, E=3, I=64, dtype="bf16")
    x = U.to_dev(wl.bf16_bits_to_f32(wl.make_x(w, 6))).float()
    before = U.from_dev(x).copy()
    offs = U.to_dev(np.array([0, 20, 20, 40], np.int32))
    L.readme_moe_ffn_stack(x, offs, [], w.E, w.I)
    empty = torch.empty(0, w.d, dtype=torch.float32, device=U.dev())
    packed = L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w, 6)))
    L.readme_moe_ffn_stack(empty, U.to_dev(np.zeros(w.E + 1, np.int32)), [packed], w.E, w.I)
    torch.cuda.synchronize()
    assert (U.from_dev(x) == before).all()


def test_large_batch_fused_layer(L, oracle_mod):
    """131072 tokens over 64 experts (d = 512, I = 320, Zipf-skewed ids): the
    many-workgroup grouping bit-exact, and the fused FFN's largest grids
    (thousands of workgroups per class of the mixed launch) on 4096 sampled
    rows spread over every expert."""
    T, d, E, I = 131072, 512, 64, 320
    _say("large batch", T, E)
    w = wl.Workload("large", T=T, d=d, E=E, I=I, dtype="bf16")
    x = wl.make_x(w, 11)
    rng = np.random.default_rng(11)
    p = 1.0 / np.arange(1, E + 1)
    ids = rng.choice(E, size=T, p=p / p.sum()).astype(np.int32)
    wg, wu, wd = wl.make_experts(w, 11)
    xd = U.to_dev(x)
    counts, offs, perm, inv, _ = L.readme_group_by_expert(U.to_dev(ids), E)
    packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
    y = L.readme_moe_ffn_fused(xd, perm, offs, packed, E, I)
    torch.cuda.synchronize()
    c_ref, o_ref, p_ref, i_ref = oracle_mod.group(ids, E)
    assert (U.from_dev(counts) == c_ref).all() and (U.from_dev(offs) == o_ref).all()
    assert (U.from_dev(perm) == p_ref).all() and (U.from_dev(inv) == i_ref).all()
    # 64 grouped rows from each expert's block (or all of a small block)
    rows = np.concatenate([np.linspace(o_ref[e], o_ref[e + 1] - 1, 64).astype(np.int64)
                           for e in range(E) if o_ref[e + 1] > o_ref[e]])
    rows = np.unique(rows)
    x_g = oracle_mod.gather(x, p_ref)
    ref = oracle_mod.moe_ffn(x_g, o_ref, wg, wu, wd, rows=rows)
    got = U.from_dev(y)[p_ref[rows]]
    U.close(got, ref, "large batch")
