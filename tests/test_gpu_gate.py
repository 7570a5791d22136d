"""The softmax-weighted top-1 variant through the C ABI: gate weights within
fp32 rounding of the oracle's fp64 softmax, the scaled ungroup bit for bit
against the oracle on the same inputs, and the weighted layer within the FFN
tolerance of the oracle's fp64 layer."""
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


@pytest.mark.parametrize("name", ["tiny_f32", "llama7b_layer", "prefill_skew16"])
def test_weighted_top1_layer(L, oracle_mod, name):
    w = wl.WORKLOADS[name]
    print("weighted top-1", name, flush=True)
    x = wl.make_x(w)
    wr, b = wl.make_router(w)
    wg, wu, wd = wl.make_experts(w)
    xd = U.to_dev(x)
    logits = torch.empty(w.T, w.E, dtype=torch.float32, device=U.dev())
    ids, _ = L.readme_route(xd, U.to_dev(wr), None if b is None else U.to_dev(b), logits=logits)
    counts, offs, perm, inv, xg = L.readme_group_by_expert(ids, w.E, x=xd)
    scale = L.readme_gate_weights(logits, ids, inv)
    packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
    yg = L.readme_moe_ffn(xg, offs, packed, w.E, w.I)
    y = L.readme_ungroup_scaled(yg, inv, scale)
    torch.cuda.synchronize()
    ids_h, inv_h, perm_h = U.from_dev(ids), U.from_dev(inv), U.from_dev(perm)
    lg = U.from_dev(logits)
    # gate weights: fp32 softmax against the fp64 one
    p_ref = oracle_mod.gate_weights(lg, ids_h)
    p_got = U.from_dev(scale)[inv_h]
    assert np.allclose(p_got, p_ref, rtol=2e-6, atol=0)
    # the scaled ungroup: bit for bit on the same y_g and weights
    got = U.from_dev(y)
    assert (got == oracle_mod.ungroup_scaled(U.from_dev(yg), inv_h, U.from_dev(scale))).all()
    # the weighted layer against the oracle's fp64 FFN times the fp64 gate
    n = int(U.from_dev(offs)[w.E])
    x_g = oracle_mod.gather(x, perm_h)
    ref_g = oracle_mod.moe_ffn(x_g, U.from_dev(offs), wg, wu, wd)
    ref = ref_g[inv_h] * p_ref[:, None]
    assert n == w.T
    U.close(got, ref, name)


def test_unrouted_rows_zero_and_scales_untouched(L, oracle_mod):
    T, d, E = 200, 64, 5
    rng = np.random.default_rng(5)
    ids_h = rng.integers(-1, E + 1, size=T).astype(np.int32)
    lg = rng.standard_normal((T, E)).astype(np.float32)
    ids = U.to_dev(ids_h)
    counts, offs, perm, inv, _ = L.readme_group_by_expert(ids, E)
    scale = torch.full((T,), 7.0, dtype=torch.float32, device=U.dev())
    L.readme_gate_weights(U.to_dev(lg), ids, inv, row_scale=scale)
    yg = U.to_dev(rng.standard_normal((T, d)).astype(np.float32))
    y = L.readme_ungroup_scaled(yg, inv, scale)
    torch.cuda.synchronize()
    routed = (ids_h >= 0) & (ids_h < E)
    inv_h = U.from_dev(inv)
    n = int(routed.sum())
    sc = U.from_dev(scale)
    assert (sc[n:] == 7.0).all()                    # grouped rows past the routed ones
    assert np.allclose(sc[inv_h[routed]], oracle_mod.gate_weights(lg, ids_h)[routed], rtol=2e-6)
    assert (U.from_dev(y)[~routed] == 0).all()
    assert (U.from_dev(y) == oracle_mod.ungroup_scaled(U.from_dev(yg), inv_h, sc)).all()
