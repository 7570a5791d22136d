"""The seeded input generator: determinism, shapes, bf16 casting and the
dense-to-expert column split."""
import hashlib

import numpy as np

from paper_2410_19123_amd import workloads as wl


def _h(a):
    return hashlib.sha256(np.ascontiguousarray(a).tobytes()).hexdigest()


def test_same_seed_same_bytes():
    w = wl.WORKLOADS["tiny_f32"]
    assert _h(wl.make_x(w, 0)) == _h(wl.make_x(w, 0))
    assert _h(wl.make_x(w, 0)) != _h(wl.make_x(w, 1))
    a = wl.make_experts(w, 0)
    b = wl.make_experts(w, 0)
    assert all(_h(p) == _h(q) for p, q in zip(a, b))


def test_shapes_and_dtypes():
    for w in wl.WORKLOADS.values():
        ws = w.with_T(min(w.T, 64))
        x = wl.make_x(ws)
        assert x.shape == (ws.T, w.d)
        assert x.dtype == (np.float32 if w.dtype == "f32" else np.uint16)
        wr, b = wl.make_router(ws)
        if w.router:
            assert wr.shape == (w.E, w.d)
        b_expected = w.bias != "none" and w.router
        assert (b is not None) == b_expected


def test_bf16_cast_is_round_to_nearest_even():
    a = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -2.5], np.float32)
    got = wl.bf16_bits_to_f32(wl.to_bf16_bits(a))
    assert got.tolist() == [1.0, 1 + 2 ** -6, 1 + 2 ** -7, -2.5]


def test_experts_are_column_slices_of_dense():
    w = wl.Workload("t", T=4, d=32, E=3, I=8, dtype="f32")
    wg, wu, wd = wl.make_experts(w, 5)
    dg, du, dd = wl.make_dense(w, 5)
    for e in range(3):
        assert (wg[e] == dg[8 * e:8 * e + 8]).all()
        assert (wu[e] == du[8 * e:8 * e + 8]).all()
        assert (wd[e] == dd[:, 8 * e:8 * e + 8]).all()


def test_request_ids_are_per_request():
    w = wl.WORKLOADS["wide_requests"]
    ids = wl.make_request_ids(w)
    assert ids.shape == (8192,)
    r = ids.reshape(256, 32)
    assert (r == r[:, :1]).all()
    assert ids.min() >= 0 and ids.max() < 8


def test_layers_draw_independent_weights():
    w = wl.Workload("t", T=4, d=16, E=2, I=8, dtype="bf16", layers=3)
    a = wl.make_experts(w, 0, layer=0)[0]
    b = wl.make_experts(w, 0, layer=1)[0]
    assert _h(a) != _h(b)
