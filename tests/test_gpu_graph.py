"""HIP graph capture of the path.  The calls only enqueue kernels on the
caller's stream (no allocation, synchronisation, memset or host read of
device data), so a step captured once replays on new inputs.  Each replay,
with eager work and a synchronisation between replays, must equal the eager
call on the same input bit for bit."""
import numpy as np
import pytest

from paper_2410_19123_amd import workloads as wl
from tests._util import to_dev

pytestmark = pytest.mark.gpu


def _lib():
    from paper_2410_19123_amd import _lib
    return _lib


def _capture(step):
    """Warm up on a side stream, then capture step() into a graph."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    return g


def _replays_match(load_input, step, outputs, n_inputs=3):
    """Eager results for each input, then graph replays on the same inputs
    (loaded eagerly between replays) compared bit for bit."""
    import torch
    refs = []
    for i in range(n_inputs):
        load_input(i)
        step()
        torch.cuda.synchronize()
        refs.append([o.clone() for o in outputs])
    g = _capture(step)
    for rep in range(2):
        for i in range(n_inputs):
            load_input(i)
            g.replay()
            torch.cuda.synchronize()
            for o, r in zip(outputs, refs[i]):
                assert torch.equal(o, r), f"replay {rep}, input {i} differs"


def test_fused_step_replays():
    """route -> group -> gate/up (gathered) -> down (scattered)."""
    import torch
    L = _lib()
    w = wl.WORKLOADS["llama7b_layer"].with_T(512)
    wr, b = wl.make_router(w)
    wg, wu, wd = wl.make_experts(w)
    xs = [to_dev(wl.make_x(w, seed)) for seed in (1, 2, 3)]
    dev = xs[0].device
    x = torch.empty_like(xs[0])
    wr_d, b_d = to_dev(wr), to_dev(b)
    packed = L.readme_pack_experts(to_dev(wg), to_dev(wu), to_dev(wd))
    T, E, I = w.T, w.E, w.I
    ids = torch.empty(T, dtype=torch.int32, device=dev)
    counts = torch.empty(E, dtype=torch.int32, device=dev)
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev)
    perm = torch.empty(T, dtype=torch.int32, device=dev)
    inv = torch.empty(T, dtype=torch.int32, device=dev)
    y = torch.empty_like(x)
    ws = torch.empty(max(L.readme_moe_ffn_workspace_bytes(x.dtype, T, I), 1), dtype=torch.uint8,
                     device=dev)

    def step():
        L.readme_route(x, wr_d, b_d, expert_ids=ids)
        L.readme_group_by_expert(ids, E, counts=counts, offsets=offsets, perm=perm, inv_perm=inv)
        L.readme_moe_ffn_fused(x, perm, offsets, packed, E, I, y=y, workspace=ws)

    _replays_match(lambda i: x.copy_(xs[i]), step, [ids, perm, y])


def test_many_workgroup_grouping_replays():
    """The three-launch grouping of 8192+ tokens (per-chunk histograms,
    scan and ranks, inverse) inside a graph."""
    import torch
    L = _lib()
    T, E = 12000, 16
    rng = np.random.default_rng(5)
    id_sets = [to_dev(rng.integers(0, E, T).astype(np.int32)) for _ in range(3)]
    dev = id_sets[0].device
    ids = torch.empty(T, dtype=torch.int32, device=dev)
    counts = torch.empty(E, dtype=torch.int32, device=dev)
    offsets = torch.empty(E + 1, dtype=torch.int32, device=dev)
    perm = torch.empty(T, dtype=torch.int32, device=dev)
    inv = torch.empty(T, dtype=torch.int32, device=dev)

    def step():
        L.readme_group_by_expert(ids, E, counts=counts, offsets=offsets, perm=perm, inv_perm=inv)

    _replays_match(lambda i: ids.copy_(id_sets[i]), step, [counts, offsets, perm, inv])


def test_decode_stack_replays():
    """Two stacked layers updating the fp32 residual in place."""
    import torch
    L = _lib()
    w = wl.WORKLOADS["llama7b_decode32"]
    T, E, I, d = w.T, w.E, w.I, w.d
    packs = []
    for layer in range(2):
        wg, wu, wd = wl.make_experts(w, layer=layer)
        packs.append(L.readme_pack_experts(to_dev(wg), to_dev(wu), to_dev(wd)))
    rng = np.random.default_rng(6)
    x0s = [to_dev(rng.standard_normal((T, d)).astype(np.float32)) for _ in range(3)]
    counts = np.bincount(rng.integers(0, E, T), minlength=E)
    offsets = to_dev(np.concatenate([[0], np.cumsum(counts)]).astype(np.int32))
    x = torch.empty_like(x0s[0])
    ws = torch.empty(L.readme_moe_ffn_stack_workspace_bytes(T, d, I), dtype=torch.uint8,
                     device=x.device)

    def step():
        L.readme_moe_ffn_stack(x, offsets, packs, E, I, workspace=ws)

    _replays_match(lambda i: x.copy_(x0s[i]), step, [x])


def test_router_tf_replays():
    """The pre-gating router block (nine launches) inside a graph."""
    import torch
    L = _lib()
    shape = wl.RouterShape(D=256, F=192, V=1000, E=5)
    wts = wl.make_router_tf(shape, 4)
    lengths = [40, 0, 7, 150]
    tok_sets = [to_dev(wl.make_router_requests(lengths, shape.V, seed)[0]) for seed in (1, 2, 3)]
    ro = to_dev(wl.make_router_requests(lengths, shape.V, 1)[1])
    dev = ro.device
    dw = {n: to_dev(wts[n]) for n in ("emb", "wq", "wk", "wv", "wo", "w1", "w3", "w2",
                                       "w_router")}
    packed = L.readme_router_tf_pack(dw["wq"], dw["wk"], dw["wv"], dw["wo"], dw["w1"], dw["w3"],
                                     dw["w2"])
    T = int(sum(lengths))
    tokens = torch.empty(T, dtype=torch.int32, device=dev)
    ids = torch.empty(T, dtype=torch.int32, device=dev)
    logits = torch.empty(T, shape.E, dtype=torch.float32, device=dev)
    ws = torch.empty(L.readme_router_tf_workspace_bytes(T, shape.D, shape.F), dtype=torch.uint8,
                     device=dev)
    feat = L.router_tf_region(ws, T, shape.D, shape.F, "FEAT")

    def step():
        L.readme_router_tf(tokens, ro, dw["emb"], packed, shape.F, dw["w_router"], None, 1e-5,
                           expert_ids=ids, logits=logits, workspace=ws)

    _replays_match(lambda i: tokens.copy_(tok_sets[i]), step, [ids, logits, feat])
