"""The softmax-weighted top-1 variant (Eq. 2's gate factor under Eq. 4's
softmax): the oracle's gate weights and scaled ungroup, pinned by hand-derived
values, the full softmax of the top-K oracle, and exact special cases."""
import numpy as np

from oracle import oracle as O


def test_gate_weights_hand_derived():
    # logits 0 and ln 3: softmax (1/4, 3/4); ids outside [0, E) give NaN
    lg = np.array([[0.0, np.log(3.0)], [np.log(3.0), 0.0]], np.float32)
    w = O.gate_weights(lg, np.array([1, 1]))
    assert abs(w[0] - 0.75) < 1e-7 and abs(w[1] - 0.25) < 1e-7
    assert np.isnan(O.gate_weights(lg, np.array([2, -1]))).all()


def test_gate_weights_sum_to_one_and_match_full_softmax():
    rng = np.random.default_rng(3)
    lg = rng.standard_normal((50, 7)).astype(np.float32) * 3
    per_e = np.stack([O.gate_weights(lg, np.full(50, e)) for e in range(7)], axis=1)
    assert np.allclose(per_e.sum(axis=1), 1.0, atol=1e-12)
    # top-K with K = E is the full softmax, slots in descending logit order
    ids, w = O.topk(lg, 7)
    for k in range(7):
        assert np.allclose(O.gate_weights(lg, ids[:, k]), w[:, k], rtol=1e-12)


def test_ungroup_scaled_special_cases():
    rng = np.random.default_rng(4)
    T, d = 40, 16
    y_g = O.f32_to_bf16(rng.standard_normal((T, d)).astype(np.float32))
    inv = rng.permutation(T).astype(np.int32)
    inv[3] = -1
    one = np.ones(T, np.float32)
    got = O.ungroup_scaled(y_g, inv, one)
    ref = O.ungroup(y_g, np.where(inv < 0, -1, inv).astype(np.int32))
    assert (got == ref).all()                                   # scale 1: the plain ungroup
    two = O.ungroup_scaled(y_g, inv, 2 * one)                   # powers of two are exact
    assert ((two.astype(np.uint32) << 16).view(np.float32)[inv >= 0] ==
            2 * (ref.astype(np.uint32) << 16).view(np.float32)[inv >= 0]).all()
    assert (got[3] == 0).all()


def test_ungroup_scaled_rounding():
    # 1.0 (bf16 0x3F80) times 1 + 2^-8 is exactly halfway between 1.0 and
    # 1.0078125: round to even keeps 0x3F80; a hair more rounds up to 0x3F81.
    y = np.array([[0x3F80] * 8], np.uint16)
    inv = np.array([0], np.int32)
    assert O.ungroup_scaled(y, inv, np.array([1 + 2**-8], np.float32))[0, 0] == 0x3F80
    assert O.ungroup_scaled(y, inv, np.array([1 + 2**-8 + 2**-20], np.float32))[0, 0] == 0x3F81
    # fp32 rows: the product rounded once
    yf = np.array([[1.0, 3.0, -0.5, 0.0]], np.float32)
    got = O.ungroup_scaled(yf, inv, np.array([0.1], np.float32))
    assert (got == (yf * np.float32(0.1))).all()
