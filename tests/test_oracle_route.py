"""Pins of the oracle's router (top-1 pre-gating, Sec. 2.3 Eq. 2 with K = 1).

The oracle fixes one fp32 summation order so that the GPU can match its ids
bit for bit.  These tests tie that order, and the argmax rule, to things
outside the oracle: hand-derived values, an fp64 library product with the
recursive-summation error bound, numpy's argmax and forced ties.
"""
import os

import numpy as np
import pytest

from paper_2410_19123_amd import workloads as wl

GOLD = os.path.join(os.path.dirname(__file__), "golden")
U32 = 2.0 ** -24


def _gamma(n):
    return n * U32 / (1 - n * U32)


def test_canonical_order_hand_values(oracle_mod):
    rows = []
    for line in open(os.path.join(GOLD, "route_canonical_order.txt")):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        f = line.split()
        rows.append((int(f[0]), [tuple(map(float, kv.split(":"))) for kv in f[1:-1]],
                     float(f[-1])))
    d = 512
    x = np.zeros((len(rows), d), np.float32)
    for t, entries, _ in rows:
        for k, v in entries:
            x[t, int(k)] = v
    w = np.ones((1, d), np.float32)
    ids, logits = oracle_mod.route(x, w, None)
    for t, _, expect in rows:
        assert logits[t, 0] == np.float32(expect), (t, logits[t, 0], expect)
    assert (ids == 0).all()


def test_bias_added_once_after_sum(oracle_mod):
    d = 512
    x = np.zeros((1, d), np.float32)
    x[0, 0] = 1.0
    w = np.ones((2, d), np.float32)
    b = np.array([2.0 ** -30, 0.5], np.float32)
    _, logits = oracle_mod.route(x, w, b)
    # 1 + 2^-30 rounds to 1 in fp32; 1 + 0.5 is exact.
    assert logits[0, 0] == np.float32(1.0)
    assert logits[0, 1] == np.float32(1.5)


@pytest.mark.parametrize("dtype,d,E", [("f32", 512, 4), ("bf16", 4096, 8),
                                       ("bf16", 1024, 16), ("bf16", 8, 3)])
def test_logits_within_fp64_error_bound(oracle_mod, dtype, d, E):
    w = wl.Workload("t", T=97, d=d, E=E, I=8, dtype=dtype, bias="zipf1")
    x = wl.make_x(w, seed=3)
    wr, b = wl.make_router(w, seed=3)
    ids, logits = oracle_mod.route(x, wr, b)
    xf = x if dtype == "f32" else wl.bf16_bits_to_f32(x)
    wf = wr if dtype == "f32" else wl.bf16_bits_to_f32(wr)
    exact = xf.astype(np.float64) @ wf.astype(np.float64).T + b.astype(np.float64)
    mag = np.abs(xf.astype(np.float64)) @ np.abs(wf.astype(np.float64)).T + np.abs(b)
    bound = _gamma(d + 1) * mag
    assert (np.abs(logits - exact) <= bound).all()
    # Where the fp64 top-2 gap exceeds twice the bound, the id is determined.
    srt = np.sort(exact, axis=1)
    gap = srt[:, -1] - srt[:, -2]
    safe = gap > 2 * bound.max(axis=1)
    assert safe.mean() > 0.9
    assert (ids[safe] == np.argmax(exact[safe], axis=1)).all()
    # And the ids are numpy's first-occurrence argmax over the oracle logits.
    assert (ids == np.argmax(logits, axis=1)).all()


def test_ties_go_to_lowest_index(oracle_mod):
    w = wl.Workload("t", T=64, d=256, E=4, I=8, dtype="bf16")
    x = wl.make_x(w, seed=5)
    wr, _ = wl.make_router(w, seed=5)
    wr = wr.copy()
    wr[2] = wr[1]
    wr[3] = wr[1]
    bias = np.array([-100.0, 0.0, 0.0, 0.0], np.float32)
    ids, logits = oracle_mod.route(x, wr, bias)
    assert (logits[:, 1] == logits[:, 2]).all() and (logits[:, 1] == logits[:, 3]).all()
    assert (ids == 1).all()


def test_nan_never_wins(oracle_mod):
    d = 512
    x = np.zeros((3, d), np.float32)
    x[:, 0] = 1.0
    w = np.zeros((3, d), np.float32)
    w[:, 0] = [1.0, 2.0, 3.0]
    b = np.array([0.0, np.nan, 0.0], np.float32)
    ids, _ = oracle_mod.route(x, w, b)
    assert (ids == 2).all()
    b = np.array([np.nan, 5.0, 0.0], np.float32)
    ids, _ = oracle_mod.route(x, w, b)   # NaN at e = 0: nothing beats it
    assert (ids == 0).all()


def test_route_rejects_unaligned_width(oracle_mod):
    x = np.zeros((2, 12), np.uint16)
    w = np.zeros((2, 12), np.uint16)
    with pytest.raises(ValueError):
        oracle_mod.route(x, w, None)
