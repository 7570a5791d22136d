"""Pins of the oracle's expert FFN (Eq. 2 with a fixed top-1 expert; the
expert form of Sec. 3 as the Llama SwiGLU FFN of Table 1).

Checked against: hand-derived scalar cases, torch's fp64 dense SwiGLU (E=1
with a full-width expert), the column-split identity (experts are slices of
one dense FFN, so their outputs sum to the dense output), brute force per
token on tiny inputs, and permutation equivariance.
"""
import os

import numpy as np
import pytest
import torch

from paper_2410_19123_amd import workloads as wl

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _f(a, dtype):
    return a if dtype == "f32" else wl.bf16_bits_to_f32(a)


def _torch_swiglu(x, wg, wu, wd):
    x, wg, wu, wd = (torch.from_numpy(np.asarray(a, np.float64)) for a in (x, wg, wu, wd))
    h = torch.nn.functional.silu(x @ wg.T) * (x @ wu.T)
    return (h @ wd.T).numpy()


def test_scalar_closed_forms(oracle_mod):
    for line in open(os.path.join(GOLD, "swiglu_scalar.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        x, g, u, dn, expect = map(float, line.split())
        y = oracle_mod.moe_ffn(np.array([[x]], np.float32), np.array([0, 1], np.int32),
                               np.array([[[g]]], np.float32), np.array([[[u]]], np.float32),
                               np.array([[[dn]]], np.float32))
        assert abs(y[0, 0] - expect) <= 1e-15 * max(1.0, abs(expect)), (line, y)


@pytest.mark.parametrize("dtype,T,d,I", [("f32", 33, 64, 48), ("bf16", 40, 128, 96)])
def test_single_expert_equals_dense_swiglu(oracle_mod, dtype, T, d, I):
    w = wl.Workload("t", T=T, d=d, E=1, I=I, dtype=dtype)
    x = wl.make_x(w, 1)
    wg, wu, wd = wl.make_experts(w, 1)
    y = oracle_mod.moe_ffn(x, np.array([0, T], np.int32), wg, wu, wd)
    ref = _torch_swiglu(_f(x, dtype), _f(wg[0], dtype), _f(wu[0], dtype), _f(wd[0], dtype))
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12 * np.abs(ref).max())


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_column_split_sums_to_dense(oracle_mod, dtype):
    E, I, d, T = 4, 24, 64, 9
    w = wl.Workload("t", T=T, d=d, E=E, I=I, dtype=dtype)
    x = wl.make_x(w, 2)
    wg, wu, wd = wl.make_experts(w, 2)
    dg, du, dd = wl.make_dense(w, 2)
    dense = _torch_swiglu(_f(x, dtype), _f(dg, dtype), _f(du, dtype), _f(dd, dtype))
    total = np.zeros((T, d))
    for e in range(E):
        # Put every token on expert e: one block covering all rows.
        off = np.array([0] * (e + 1) + [T] * (E - e), np.int32)
        total += oracle_mod.moe_ffn(x, off, wg, wu, wd)
    assert np.allclose(total, dense, rtol=1e-11, atol=1e-11 * np.abs(dense).max())


def test_brute_force_per_token_tiny(oracle_mod):
    import math
    rng = np.random.default_rng(7)
    T, d, I, E = 11, 6, 5, 3
    x = rng.standard_normal((T, d)).astype(np.float32)
    wg = (rng.standard_normal((E, I, d)) * 0.5).astype(np.float32)
    wu = (rng.standard_normal((E, I, d)) * 0.5).astype(np.float32)
    wd = (rng.standard_normal((E, d, I)) * 0.5).astype(np.float32)
    ids = rng.integers(0, E, size=T).astype(np.int32)
    out = oracle_mod.full_path(x, None, None, wg, wu, wd, ids=ids)
    for t in range(T):
        e = int(ids[t])
        h = []
        for i in range(I):
            g = sum(float(wg[e, i, k]) * float(x[t, k]) for k in range(d))
            u = sum(float(wu[e, i, k]) * float(x[t, k]) for k in range(d))
            h.append(g / (1.0 + math.exp(-g)) * u)
        for c in range(d):
            yc = sum(float(wd[e, c, i]) * h[i] for i in range(I))
            assert abs(out["y"][t, c] - yc) <= 1e-12 * max(1.0, abs(yc))


def test_permutation_equivariance_within_expert(oracle_mod):
    w = wl.Workload("t", T=30, d=32, E=2, I=16, dtype="bf16")
    x = wl.make_x(w, 4)
    wg, wu, wd = wl.make_experts(w, 4)
    off = np.array([0, 12, 30], np.int32)
    y = oracle_mod.moe_ffn(x, off, wg, wu, wd)
    p = np.concatenate([np.random.default_rng(0).permutation(12),
                        12 + np.random.default_rng(1).permutation(18)])
    yp = oracle_mod.moe_ffn(x[p], off, wg, wu, wd)
    assert (yp == y[p]).all()


def test_rows_subset_equals_full(oracle_mod):
    w = wl.Workload("t", T=40, d=64, E=3, I=32, dtype="bf16")
    x = wl.make_x(w, 6)
    wg, wu, wd = wl.make_experts(w, 6)
    off = np.array([0, 0, 25, 40], np.int32)       # expert 0 empty
    y = oracle_mod.moe_ffn(x, off, wg, wu, wd)
    rows = np.array([39, 0, 24, 25])
    assert (oracle_mod.moe_ffn(x, off, wg, wu, wd, rows=rows) == y[rows]).all()
    with pytest.raises(ValueError):
        oracle_mod.moe_ffn(x, np.array([0, 0, 25, 30], np.int32), wg, wu, wd,
                           rows=np.array([35]))
