"""Pins of the oracle's grouping (per-expert queues of Alg. 1, Sec. 4.2).

Counts, offsets and the stable permutation are checked against numpy's
bincount, cumsum and stable argsort (special cases that reduce to library
routines) and against a brute-force loop on tiny inputs.
"""
import numpy as np
import pytest


def _brute(ids, E):
    counts = [0] * E
    for i in ids:
        if 0 <= i < E:
            counts[i] += 1
    perm = []
    for e in range(E):
        perm += [t for t, i in enumerate(ids) if i == e]
    return counts, perm


@pytest.mark.parametrize("T,E,seed", [(0, 1, 0), (1, 1, 0), (63, 4, 1), (65, 4, 2),
                                      (1000, 8, 3), (4097, 256, 4), (300, 1, 5)])
def test_group_matches_library_routines(oracle_mod, T, E, seed):
    rng = np.random.default_rng(seed)
    ids = rng.integers(0, E, size=T).astype(np.int32)
    counts, offsets, perm, inv = oracle_mod.group(ids, E)
    assert (counts == np.bincount(ids, minlength=E)).all()
    assert offsets[0] == 0 and (offsets[1:] == np.cumsum(np.bincount(ids, minlength=E))).all()
    assert (perm == np.argsort(ids, kind="stable")).all()
    assert (inv[perm] == np.arange(T)).all()
    assert sorted(perm.tolist()) == list(range(T))   # bijection
    assert counts.sum() == T
    if T:
        assert (np.diff(ids[perm]) >= 0).all()


def test_group_brute_force_tiny(oracle_mod):
    rng = np.random.default_rng(11)
    for _ in range(50):
        T = int(rng.integers(0, 20))
        E = int(rng.integers(1, 6))
        ids = rng.integers(0, E, size=T).astype(np.int32)
        counts, offsets, perm, _ = oracle_mod.group(ids, E)
        bc, bp = _brute(ids.tolist(), E)
        assert counts.tolist() == bc and perm.tolist() == bp


def test_group_empty_experts_and_single_expert(oracle_mod):
    ids = np.full(100, 2, np.int32)
    counts, offsets, perm, inv = oracle_mod.group(ids, 5)
    assert counts.tolist() == [0, 0, 100, 0, 0]
    assert offsets.tolist() == [0, 0, 0, 100, 100, 100]
    assert (perm == np.arange(100)).all() and (inv == np.arange(100)).all()


def test_group_out_of_range_ids_are_left_out(oracle_mod):
    ids = np.array([0, 5, 1, -1, 1, 0, 7], np.int32)
    counts, offsets, perm, inv = oracle_mod.group(ids, 3)
    assert counts.tolist() == [2, 2, 0]
    assert offsets.tolist() == [0, 2, 4, 4]
    assert perm.tolist() == [0, 5, 2, 4, -1, -1, -1]
    assert inv.tolist() == [0, -1, 2, -1, 3, 1, -1]


def test_gather_ungroup_roundtrip(oracle_mod):
    rng = np.random.default_rng(2)
    T, d, E = 77, 24, 5
    ids = rng.integers(0, E, size=T).astype(np.int32)
    x = rng.integers(0, 65535, size=(T, d)).astype(np.uint16)
    _, _, perm, inv = oracle_mod.group(ids, E)
    xg = oracle_mod.gather(x, perm)
    assert (xg == x[perm]).all()                 # numpy fancy indexing
    back = oracle_mod.ungroup(xg, inv)
    assert (back == x).all()
    yf = rng.standard_normal((T, d))
    assert (oracle_mod.ungroup(yf, inv) == yf[inv]).all()


def test_gather_ungroup_unrouted_rows_are_zero(oracle_mod):
    ids = np.array([1, 9, 0], np.int32)
    x = np.arange(6, dtype=np.float32).reshape(3, 2) + 1
    _, offsets, perm, inv = oracle_mod.group(ids, 2)
    xg = oracle_mod.gather(x, perm)
    assert xg.tolist() == [[5, 6], [1, 2], [0, 0]]
    y = oracle_mod.ungroup(xg, inv)
    assert y.tolist() == [[1, 2], [0, 0], [5, 6]]
