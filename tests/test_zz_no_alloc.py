"""readme_moe_ffn_fused_noalloc (h in the library's fixed device array, no
workspace) through the C ABI: two calls in a row, the second smaller, each
equal bit for bit to readme_moe_ffn_fused on the same inputs."""
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


def _case(L, w, seed):
    x = U.to_dev(wl.make_x(w, seed))
    wr, b = wl.make_router(w, seed)
    ids, _ = L.readme_route(x, U.to_dev(wr), None if b is None else U.to_dev(b))
    counts, offs, perm, inv, _ = L.readme_group_by_expert(ids, w.E)
    packed = L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w, seed)))
    return x, perm, offs, packed


def test_noalloc_equals_fused_two_calls(L):
    big = wl.WORKLOADS["llama7b_layer"]                     # h: 2048 x 1408 bf16
    small = wl.Workload("t", T=300, d=512, E=5, I=200, dtype="bf16", bias="zipf1")
    cases = [(big, 0), (small, 3)]
    prepared = [_case(L, w, s) for w, s in cases]
    outs = []
    for (w, _), (x, perm, offs, packed) in zip(cases, prepared):
        print("noalloc", w.name, w.T, w.d, w.E, w.I, flush=True)
        y = torch.full_like(x, 3.0)
        L.readme_moe_ffn_fused_noalloc(x, perm, offs, packed, w.E, w.I, y)
        outs.append(y)
    torch.cuda.synchronize()
    for (w, _), (x, perm, offs, packed), y in zip(cases, prepared, outs):
        y_ref = L.readme_moe_ffn_fused(x, perm, offs, packed, w.E, w.I)
        torch.cuda.synchronize()
        assert (U.from_dev(y) == U.from_dev(y_ref)).all(), w.name


def test_noalloc_f32_after_bf16(L):
    w = wl.WORKLOADS["tiny_f32"]
    x, perm, offs, packed = _case(L, w, 0)
    y = torch.empty_like(x)
    L.readme_moe_ffn_fused_noalloc(x, perm, offs, packed, w.E, w.I, y)
    y_ref = L.readme_moe_ffn_fused(x, perm, offs, packed, w.E, w.I)
    torch.cuda.synchronize()
    assert (U.from_dev(y) == U.from_dev(y_ref)).all()
