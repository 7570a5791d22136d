"""Pins of the oracle's layer with a permanent expert (Sec. 3: neurons every
token activates, beside its routed expert of Eq. 2).

Checked against: the mask form of Sec. 3 evaluated per token (the dense FFN
restricted to the routed expert's columns plus the permanent columns, one
numpy fp64 SwiGLU over the union), torch's fp64 dense SwiGLU when one routed
expert and the permanent expert together cover the whole dense FFN, brute
force in pure Python on tiny inputs, the P = 0 reduction to the routed FFN,
and zero routed weights leaving the permanent expert alone.
"""
import math

import numpy as np
import pytest
import torch

from paper_2410_19123_amd import workloads as wl


def _f(a, dtype):
    return a if dtype == "f32" else wl.bf16_bits_to_f32(a)


def _swiglu_np(x, wg, wu, wd):
    x, wg, wu, wd = (np.asarray(a, np.float64) for a in (x, wg, wu, wd))
    g = x @ wg.T
    return (g / (1.0 + np.exp(-g)) * (x @ wu.T)) @ wd.T


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_mask_form_per_token(oracle_mod, dtype):
    """Token t sees the dense FFN's columns of its expert and the permanent
    columns, and nothing else."""
    E, I, P, d, T = 4, 24, 40, 64, 23
    w = wl.Workload("t", T=T, d=d, E=E, I=I, P=P, dtype=dtype)
    x = wl.make_x(w, 3)
    wg, wu, wd = wl.make_experts(w, 3)
    pg, pu, pd = wl.make_permanent(w, 3)
    dg, du, dd = (_f(a, dtype) for a in wl.make_dense(w, 3))
    ids = np.random.default_rng(5).integers(0, E, size=T).astype(np.int32)
    out = oracle_mod.full_path(x, None, None, wg, wu, wd, ids=ids, permanent=(pg, pu, pd))
    xf = _f(x, dtype)
    for t in range(T):
        e = int(ids[t])
        cols = np.r_[e * I:(e + 1) * I, E * I:E * I + P]
        ref = _swiglu_np(xf[t:t + 1], dg[cols], du[cols], dd[:, cols])[0]
        assert np.allclose(out["y"][t], ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max()), t


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_one_expert_plus_permanent_is_dense(oracle_mod, dtype):
    """E = 1: the routed expert and the permanent expert split the dense FFN."""
    T, d, I, P = 29, 64, 40, 24
    w = wl.Workload("t", T=T, d=d, E=1, I=I, P=P, dtype=dtype)
    x = wl.make_x(w, 8)
    wg, wu, wd = wl.make_experts(w, 8)
    pg, pu, pd = wl.make_permanent(w, 8)
    dg, du, dd = wl.make_dense(w, 8)
    y = oracle_mod.moe_ffn_permanent(x, np.array([0, T], np.int32), wg, wu, wd, pg, pu, pd)
    t = [torch.from_numpy(np.asarray(_f(a, dtype), np.float64)) for a in (x, dg, du, dd)]
    ref = ((torch.nn.functional.silu(t[0] @ t[1].T) * (t[0] @ t[2].T)) @ t[3].T).numpy()
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_brute_force_tiny(oracle_mod):
    rng = np.random.default_rng(11)
    T, d, I, P, E = 9, 5, 4, 3, 3
    x = rng.standard_normal((T, d)).astype(np.float32)
    wg = (rng.standard_normal((E, I, d)) * 0.5).astype(np.float32)
    wu = (rng.standard_normal((E, I, d)) * 0.5).astype(np.float32)
    wd = (rng.standard_normal((E, d, I)) * 0.5).astype(np.float32)
    pg = (rng.standard_normal((P, d)) * 0.5).astype(np.float32)
    pu = (rng.standard_normal((P, d)) * 0.5).astype(np.float32)
    pd = (rng.standard_normal((d, P)) * 0.5).astype(np.float32)
    ids = rng.integers(0, E, size=T).astype(np.int32)
    out = oracle_mod.full_path(x, None, None, wg, wu, wd, ids=ids, permanent=(pg, pu, pd))

    def neuron(gw, uw, t):
        g = sum(float(gw[k]) * float(x[t, k]) for k in range(d))
        u = sum(float(uw[k]) * float(x[t, k]) for k in range(d))
        return g / (1.0 + math.exp(-g)) * u

    for t in range(T):
        e = int(ids[t])
        h = [neuron(wg[e, i], wu[e, i], t) for i in range(I)]
        hp = [neuron(pg[i], pu[i], t) for i in range(P)]
        for c in range(d):
            yc = sum(float(wd[e, c, i]) * h[i] for i in range(I))
            yc += sum(float(pd[c, i]) * hp[i] for i in range(P))
            assert abs(out["y"][t, c] - yc) <= 1e-12 * max(1.0, abs(yc))


def test_zero_routed_weights_leave_permanent_only(oracle_mod):
    w = wl.Workload("t", T=17, d=32, E=3, I=16, P=32, dtype="bf16")
    x = wl.make_x(w, 9)
    wg, wu, wd = wl.make_experts(w, 9)
    pg, pu, pd = wl.make_permanent(w, 9)
    off = np.array([0, 5, 5, 17], np.int32)
    z = np.zeros_like(wd)
    y = oracle_mod.moe_ffn_permanent(x, off, wg, wu, z, pg, pu, pd)
    ref = _swiglu_np(_f(x, "bf16"), _f(pg, "bf16"), _f(pu, "bf16"), _f(pd, "bf16"))
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


def test_rows_subset_and_routed_part(oracle_mod):
    """The routed part is moe_ffn itself; a row subset equals the full rows."""
    w = wl.Workload("t", T=30, d=64, E=3, I=32, P=32, dtype="bf16")
    x = wl.make_x(w, 12)
    wg, wu, wd = wl.make_experts(w, 12)
    pg, pu, pd = wl.make_permanent(w, 12)
    off = np.array([0, 0, 18, 30], np.int32)
    y = oracle_mod.moe_ffn_permanent(x, off, wg, wu, wd, pg, pu, pd)
    rows = np.array([29, 0, 17, 18])
    assert (oracle_mod.moe_ffn_permanent(x, off, wg, wu, wd, pg, pu, pd, rows=rows)
            == y[rows]).all()
    zp = np.zeros_like(pd)
    assert (oracle_mod.moe_ffn_permanent(x, off, wg, wu, wd, pg, pu, zp)
            == oracle_mod.moe_ffn(x, off, wg, wu, wd)).all()


def test_workload_slices_cover_dense():
    w = wl.WORKLOADS["llama7b_layer_perm"]
    small = wl.Workload("t", T=4, d=64, E=w.E, I=8, P=8, dtype="bf16")
    wg, wu, wd = wl.make_experts(small, 0)
    pg, pu, pd = wl.make_permanent(small, 0)
    dg, du, dd = wl.make_dense(small, 0)
    assert (np.concatenate([wg.reshape(-1, 64), pg]) == dg).all()
    assert (np.concatenate([wu.reshape(-1, 64), pu]) == du).all()
    assert (np.concatenate([wd.transpose(1, 0, 2).reshape(64, -1), pd], axis=1) == dd).all()
    assert w.P == w.I  # the permanent expert is one routed expert wide
