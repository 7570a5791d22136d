"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Integer results (expert ids, counts, offsets, perm, inv_perm, moved rows) and
the router's fp32 logits must be bit-exact; FFN outputs must meet the
tolerance in tests/_util.py on every row, at full size too.
"""
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


# ------------------------------------------------------------------ route
@pytest.mark.parametrize("name", ["tiny_f32", "llama7b_layer", "llama7b_decode32",
                                  "prefill_skew16"])
def test_route_bit_exact(L, oracle_mod, name):
    w = wl.WORKLOADS[name]
    _say("route", name)
    x = wl.make_x(w)
    wr, b = wl.make_router(w)
    ids_ref, lg_ref = oracle_mod.route(x, wr, b)
    logits = torch.empty(w.T, w.E, dtype=torch.float32, device=U.dev())
    ids, _ = L.readme_route(U.to_dev(x), U.to_dev(wr), None if b is None else U.to_dev(b),
                            logits=logits)
    torch.cuda.synchronize()
    assert (U.from_dev(ids) == ids_ref).all()
    assert (U.from_dev(logits).view(np.uint32) == lg_ref.view(np.uint32)).all()


@pytest.mark.parametrize("T,d,E,dtype", [(1, 8, 1, "bf16"), (5, 24, 3, "bf16"),
                                         (70, 4, 2, "f32"), (300, 520, 37, "bf16"),
                                         (9000, 256, 16, "bf16"), (130, 1032, 256, "bf16"),
                                         (33, 4096, 4, "bf16"), (4096, 2048, 16, "bf16"),
                                         (8197, 1024, 11, "bf16"), (8192, 4096, 16, "bf16"),
                                         (8200, 2048, 9, "bf16")])
def test_route_odd_shapes_and_ties(L, oracle_mod, T, d, E, dtype):
    w = wl.Workload("t", T=T, d=d, E=E, I=8, dtype=dtype, bias="zipf1")
    _say("route shape", T, d, E, dtype)
    x = wl.make_x(w, 2)
    wr, b = wl.make_router(w, 2)
    if E >= 3:
        wr = wr.copy()
        wr[E - 1] = wr[1]          # exact tie between e=1 and e=E-1
        b = b.copy()
        b[E - 1] = b[1]
    if T > 100 and dtype == "bf16":
        # rows whose logits are NaN (inf - inf inside one chunk) or +-inf
        x = x.copy()
        x[7, 0], x[7, 1] = 0x7F80, 0xFF80        # +inf, -inf: logits +inf or NaN
        x[T - 2, 3] = 0x7F80                      # one +inf: logits +-inf
    ids_ref, lg_ref = oracle_mod.route(x, wr, b)
    logits = torch.empty(T, E, dtype=torch.float32, device=U.dev())
    ids, _ = L.readme_route(U.to_dev(x), U.to_dev(wr), U.to_dev(b), logits=logits)
    torch.cuda.synchronize()
    assert (U.from_dev(ids) == ids_ref).all()
    # Bit-exact logits; a NaN is any NaN (its payload is the hardware's).
    got = U.from_dev(logits)
    nan = np.isnan(lg_ref)
    assert (np.isnan(got) == nan).all()
    assert (got.view(np.uint32)[~nan] == lg_ref.view(np.uint32)[~nan]).all()


# ------------------------------------------------------------------ group
def _ids_case(kind, T, E, seed):
    rng = np.random.default_rng(seed)
    if kind == "uniform":
        return rng.integers(0, E, size=T).astype(np.int32)
    if kind == "one_expert":
        return np.full(T, E - 1, np.int32)
    if kind == "empty_ends":          # first and last experts empty
        return rng.integers(1, max(E - 1, 2), size=T).astype(np.int32) % E
    if kind == "invalid":             # some ids outside [0, E)
        ids = rng.integers(-2, E + 2, size=T).astype(np.int32)
        return ids
    if kind == "local":               # each token repeats its predecessor w.p. 0.713
        ids = np.empty(T, np.int32)
        cur = 0
        for t in range(T):
            if t == 0 or rng.random() >= 0.713:
                cur = int(rng.integers(0, E))
            ids[t] = cur
        return ids
    raise ValueError(kind)


@pytest.mark.parametrize("kind,T,E", [
    ("uniform", 1, 1), ("uniform", 63, 4), ("uniform", 65, 4), ("uniform", 1024, 8),
    ("uniform", 1025, 8), ("uniform", 16384, 16), ("uniform", 5000, 256),
    ("one_expert", 3000, 8), ("empty_ends", 2048, 8), ("invalid", 2500, 7),
    ("local", 4096, 8), ("uniform", 40000, 3), ("uniform", 0, 4),
    # many 1024-id rounds with many experts, invalid ids among 200 experts,
    # and sizes on both sides of 16 rounds
    ("uniform", 16384, 256), ("invalid", 9000, 200), ("local", 16384, 8),
    ("uniform", 16385, 8), ("empty_ends", 16383, 64),
    # the many-workgroup sort (8192 <= T <= 2^20) at its edges: one expert at
    # the threshold, one token below it, the largest size with 256 experts,
    # and one token past it (back on one workgroup) with invalid ids
    ("one_expert", 8192, 1), ("uniform", 8191, 8), ("uniform", 1 << 20, 256),
    ("invalid", (1 << 20) + 1, 16)])
def test_group_bit_exact(L, oracle_mod, kind, T, E):
    _say("group", kind, T, E)
    ids = _ids_case(kind, T, E, seed=T + E)
    d = 64
    x = np.random.default_rng(1).integers(0, 65535, size=(T, d)).astype(np.uint16)
    counts_ref, off_ref, perm_ref, inv_ref = oracle_mod.group(ids, E)
    xg_ref = oracle_mod.gather(x, perm_ref) if T else x
    xd = U.to_dev(x) if T else torch.empty(0, d, dtype=torch.bfloat16, device=U.dev())
    counts, offs, perm, inv, xg = L.readme_group_by_expert(
        U.to_dev(ids) if T else torch.empty(0, dtype=torch.int32, device=U.dev()), E, x=xd)
    torch.cuda.synchronize()
    assert (U.from_dev(counts) == counts_ref).all()
    assert (U.from_dev(offs) == off_ref).all()
    if T:
        assert (U.from_dev(perm) == perm_ref).all()
        assert (U.from_dev(inv) == inv_ref).all()
        assert (U.from_dev(xg) == xg_ref).all()
        # And back: ungroup of the grouped rows restores routed tokens.
        y = L.readme_ungroup(xg, inv)
        torch.cuda.synchronize()
        assert (U.from_dev(y) == oracle_mod.ungroup(xg_ref, inv_ref)).all()


# -------------------------------------------------------------------- ffn
def _run_ffn(L, x_g, offsets, wg, wu, wd, E, I):
    packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
    y = L.readme_moe_ffn(U.to_dev(x_g), U.to_dev(offsets), packed, E, I)
    torch.cuda.synchronize()
    return U.from_dev(y), packed


@pytest.mark.parametrize("dtype,d,I,counts", [
    ("bf16", 256, 96, [0, 1, 31, 32, 33, 0]),
    ("bf16", 128, 40, [127, 128, 129, 255, 256, 257]),
    ("bf16", 64, 688, [5, 0, 300, 1]),
    ("f32", 128, 72, [0, 17, 128, 129, 3]),
    ("bf16", 512, 64, [800, 0, 0, 770]),
    ("bf16", 192, 130, [1]),
])
def test_ffn_ragged_blocks(L, oracle_mod, dtype, d, I, counts):
    E = len(counts)
    T = sum(counts)
    _say("ffn ragged", dtype, d, I, counts)
    w = wl.Workload("t", T=T, d=d, E=E, I=I, dtype=dtype)
    x = wl.make_x(w, 3)
    wg, wu, wd = wl.make_experts(w, 3)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    y, _ = _run_ffn(L, x, offsets, wg, wu, wd, E, I)
    ref = oracle_mod.moe_ffn(x, offsets, wg, wu, wd)
    U.close(y, ref, f"ffn {counts}")


def test_gate_up_pad_columns_are_zero(L, oracle_mod):
    w = wl.Workload("t", T=100, d=128, E=2, I=40, dtype="bf16")
    x = wl.make_x(w, 4)
    wg, wu, wd = wl.make_experts(w, 4)
    offsets = np.array([0, 60, 100], np.int32)
    packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
    h = L.readme_moe_gate_up(U.to_dev(x), U.to_dev(offsets), packed, 2, 40)
    torch.cuda.synchronize()
    hh = U.from_dev(h)
    assert hh.shape == (100, 64)
    assert (hh[:, 40:] == 0).all()
    # h itself against fp64: silu(W_g x) * (W_u x).
    xf = U.as_f64(x)
    for e, (a, b) in enumerate([(0, 60), (60, 100)]):
        g = xf[a:b] @ U.as_f64(wg[e]).T
        u = xf[a:b] @ U.as_f64(wu[e]).T
        ref = g / (1 + np.exp(-g)) * u
        U.close(hh[a:b, :40], ref, "h")


# ------------------------------------------------------------- full path
def _full_path(L, w, x, wr, b, ids_given, wg, wu, wd):
    xd = U.to_dev(x)
    if ids_given is None:
        ids, _ = L.readme_route(xd, U.to_dev(wr), None if b is None else U.to_dev(b))
    else:
        ids = U.to_dev(ids_given)
    counts, offs, perm, inv, xg = L.readme_group_by_expert(ids, w.E, x=xd)
    packed = L.readme_pack_experts(*U.weights_to_dev(wg, wu, wd))
    yg = L.readme_moe_ffn(xg, offs, packed, w.E, w.I)
    y = L.readme_ungroup(yg, inv)
    torch.cuda.synchronize()
    return dict(ids=U.from_dev(ids), counts=U.from_dev(counts), offsets=U.from_dev(offs),
                perm=U.from_dev(perm), inv=U.from_dev(inv), x_g=U.from_dev(xg),
                y_g=U.from_dev(yg), y=U.from_dev(y))


# The oracle's fp64 FFN over all 8192 rows of the request batch (1.44
# TFLOP) takes tens of seconds on the host: a longer limit for that case.
@pytest.mark.parametrize("name", ["tiny_f32", "llama7b_layer", "prefill_skew16",
                                  pytest.param("wide_requests", marks=pytest.mark.timeout(900))])
def test_full_path_workloads(L, oracle_mod, name):
    w = wl.WORKLOADS[name]
    _say("full path", name)
    x = wl.make_x(w)
    wr, b = wl.make_router(w)
    ids_given = None if w.router else wl.make_request_ids(w)
    wg, wu, wd = wl.make_experts(w)
    got = _full_path(L, w, x, wr, b, ids_given, wg, wu, wd)
    ids_ref = ids_given if ids_given is not None else oracle_mod.route(x, wr, b)[0]
    counts, offsets, perm, inv = oracle_mod.group(ids_ref, w.E)
    assert (got["ids"] == ids_ref).all()
    assert (got["counts"] == counts).all() and (got["offsets"] == offsets).all()
    assert (got["perm"] == perm).all() and (got["inv"] == inv).all()
    x_g = oracle_mod.gather(x, perm)
    assert (got["x_g"] == x_g).all()
    # Every routed row, in the launch configuration bench.py times (all M
    # tiles, the XCD-remap boundaries and each tile's full K loop).
    n = int(offsets[w.E])
    ref = oracle_mod.moe_ffn(x_g, offsets, wg, wu, wd)
    U.close(got["y_g"][:n], ref, name)
    # Ungroup is a row move: y[t] == y_g[inv[t]] bit for bit.
    assert (got["y"] == got["y_g"][inv]).all()


def test_deterministic_bitwise(L):
    w = wl.WORKLOADS["llama7b_layer"]
    x = wl.make_x(w)
    wr, b = wl.make_router(w)
    wg, wu, wd = wl.make_experts(w)
    a = _full_path(L, w, x, wr, b, None, wg, wu, wd)
    c = _full_path(L, w, x, wr, b, None, wg, wu, wd)
    for k in a:
        assert (a[k] == c[k]).all(), k


def test_single_expert_equals_dense_ffn(L, oracle_mod):
    # E = 1 with the full dense width: the MoE layer is the dense SwiGLU FFN.
    w = wl.Workload("t", T=300, d=512, E=1, I=1376, dtype="bf16")
    x = wl.make_x(w, 8)
    wg, wu, wd = wl.make_experts(w, 8)
    offsets = np.array([0, 300], np.int32)
    y, _ = _run_ffn(L, x, offsets, wg, wu, wd, 1, 1376)
    dg, du, dd = wl.make_dense(w, 8)
    xf = U.as_f64(x)
    g = xf @ U.as_f64(dg).T
    u = xf @ U.as_f64(du).T
    ref = (g / (1 + np.exp(-g)) * u) @ U.as_f64(dd).T
    U.close(y, ref, "dense")


# ------------------------------------------------------------ decode stack
def test_decode_stack_teacher_forced(L, oracle_mod):
    w = wl.WORKLOADS["llama7b_decode32"]
    _say("decode stack")
    x = wl.make_x(w)
    wr, b = wl.make_router(w)
    ids, _ = L.readme_route(U.to_dev(x), U.to_dev(wr), U.to_dev(b))
    counts, offs, perm, inv, xg = L.readme_group_by_expert(ids, w.E, x=U.to_dev(x))
    offsets = U.from_dev(offs)
    layers = [0, 1, 2, 31]
    packed, host = {}, {}
    for l in layers:
        host[l] = wl.make_experts(w, 0, layer=l)
        packed[l] = L.readme_pack_experts(*U.weights_to_dev(*host[l]))
    xr = xg.float()
    for l in layers:
        x_in = xr.clone()
        L.readme_moe_ffn_stack(xr, offs, [packed[l]], w.E, w.I)
        torch.cuda.synchronize()
        xin = U.from_dev(x_in)
        delta = U.from_dev(xr).astype(np.float64) - xin.astype(np.float64)
        ref = oracle_mod.layer(xin, offsets, *host[l], eps=1e-5)
        U.close(delta, ref, f"layer {l}")
    # One call over several layers equals the chain of single-layer calls.
    xa = xg.float()
    L.readme_moe_ffn_stack(xa, offs, [packed[l] for l in layers], w.E, w.I)
    torch.cuda.synchronize()
    assert (U.from_dev(xa) == U.from_dev(xr)).all()
    # Ungroup of the fp32 residual stream back to token order.
    y = L.readme_ungroup(xa, inv)
    torch.cuda.synchronize()
    assert (U.from_dev(y) == U.from_dev(xa)[U.from_dev(inv)]).all()


def test_decode_stack_end_to_end_error(L, oracle_mod):
    """The 32-layer decode stack from one input against the oracle's own
    32-layer chain from the same input.  Per-layer parity is gated above
    (teacher-forced); the end-to-end drift is reported, with a loose
    sanity bound only (bf16 rounding of each layer's input and output
    compounds over the layers)."""
    w = wl.WORKLOADS["llama7b_decode32"]
    _say("decode stack end to end")
    x = wl.make_x(w)
    wr, b = wl.make_router(w)
    ids, _ = L.readme_route(U.to_dev(x), U.to_dev(wr), U.to_dev(b))
    counts, offs, perm, inv, xg = L.readme_group_by_expert(ids, w.E, x=U.to_dev(x))
    offsets = U.from_dev(offs)
    host = [wl.make_experts(w, 0, layer=l) for l in range(w.layers)]
    packed = [L.readme_pack_experts(*U.weights_to_dev(*h)) for h in host]
    x0 = U.from_dev(xg.float())
    xr = xg.float()
    L.readme_moe_ffn_stack(xr, offs, packed, w.E, w.I)
    torch.cuda.synchronize()
    got = U.from_dev(xr).astype(np.float64)
    ref = x0.astype(np.float32)
    n = int(offsets[w.E])
    for l in range(w.layers):
        delta = oracle_mod.layer(ref, offsets, *host[l], eps=1e-5)
        ref = ref.copy()
        ref[:n] = (ref[:n].astype(np.float64) + delta).astype(np.float32)
    ref = ref.astype(np.float64)
    err = np.abs(got - ref)
    max_rel = float(err.max() / np.abs(ref).max())
    l1 = float(err.sum() / np.abs(ref).sum())
    dref = ref - x0
    l1_delta = float(np.abs(got - x0 - dref).sum() / np.abs(dref).sum())
    _say(f"decode stack, 32 layers end to end vs oracle chain: max rel {max_rel:.3e}, "
         f"normalized L1 {l1:.3e} (of the residual), {l1_delta:.3e} (of the 32-layer update)")
    assert np.isfinite(got).all()
    assert l1_delta < 0.1


@pytest.mark.parametrize("d", [320, 4160, 8256])
def test_stack_layer_norm_widths(L, oracle_mod, d):
    """One stacked layer at model widths where the pre-norm holds a row in
    registers as up to 4 (d = 320) or 8 (d = 4160) vectors per thread, or
    reads it twice (d = 8256); ragged experts, one of them empty."""
    _say("stack width", d)
    w = wl.Workload("t", T=70, d=d, E=4, I=96, dtype="bf16")
    x = wl.make_x(w, d)
    counts = np.array([33, 0, 30, 7], np.int32)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    host = wl.make_experts(w, d)
    packed = L.readme_pack_experts(*U.weights_to_dev(*host))
    xr = U.to_dev(wl.bf16_bits_to_f32(x)).float()
    x_in = U.from_dev(xr).copy()
    L.readme_moe_ffn_stack(xr, U.to_dev(offsets), [packed], w.E, w.I)
    torch.cuda.synchronize()
    delta = U.from_dev(xr).astype(np.float64) - x_in.astype(np.float64)
    U.close(delta, oracle_mod.layer(x_in, offsets, *host, eps=1e-5), f"d {d}")


@pytest.mark.parametrize("tile", [0, 12, 22, 24, 25, 26, 27, 30, 31])
def test_stack_tiles_match_oracle(L, oracle_mod, tile):
    """Two stacked layers (pre-norm, expert FFN, residual added in the down
    projection's epilogue) with one forced tile, on ragged blocks that put
    rows in every height class of the mixed launches; 16 K-steps in the
    gate/up GEMM."""
    _say("stack tile", tile)
    counts = np.array([300, 0, 97, 31, 513], np.int32)
    w = wl.Workload("t", T=int(counts.sum()), d=1024, E=5, I=320, dtype="bf16", layers=2)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    host = [wl.make_experts(w, 90 + tile, layer=l) for l in range(w.layers)]
    packed = [L.readme_pack_experts(*U.weights_to_dev(*h)) for h in host]
    x0 = wl.bf16_bits_to_f32(wl.make_x(w, 90 + tile)).astype(np.float32)
    xr = U.to_dev(x0)
    L.readme_set_gemm_tile(tile)
    try:
        L.readme_moe_ffn_stack(xr, U.to_dev(offsets), packed, w.E, w.I)
        torch.cuda.synchronize()
    finally:
        L.readme_set_gemm_tile(0)
    got = U.from_dev(xr).astype(np.float64)
    ref = x0.copy()
    for l in range(w.layers):
        ref = (ref.astype(np.float64) + oracle_mod.layer(ref, offsets, *host[l], eps=1e-5))
        ref = ref.astype(np.float32)
    U.close(got - x0, ref.astype(np.float64) - x0, f"stack tile {tile}")


# ------------------------------------------------------ every tile config
@pytest.mark.parametrize("tile", list(range(1, 32)))
def test_every_gemm_tile_matches_oracle(L, oracle_mod, tile):
    """Each workgroup tile of the grouped GEMM, on ragged blocks (empty,
    single-row, tile +- 1 and multi-tile experts) in bf16 and fp32."""
    _say("tile", tile)
    L.readme_set_gemm_tile(tile)
    try:
        # The last case has 16 K-steps in both GEMMs, more than any tile
        # keeps in flight, so every tile's steady-state loop runs.
        for dtype, d, I, counts in [("bf16", 256, 200, [0, 1, 255, 257, 33, 520]),
                                    ("f32", 128, 96, [3, 0, 129, 64]),
                                    ("bf16", 1024, 1000, [97, 0, 300, 31])]:
            E, T = len(counts), sum(counts)
            w = wl.Workload("t", T=T, d=d, E=E, I=I, dtype=dtype)
            x = wl.make_x(w, 10 + tile)
            wg, wu, wd = wl.make_experts(w, 10 + tile)
            offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
            y, _ = _run_ffn(L, x, offsets, wg, wu, wd, E, I)
            U.close(y, oracle_mod.moe_ffn(x, offsets, wg, wu, wd), f"tile {tile} {dtype}")
    finally:
        L.readme_set_gemm_tile(0)


# ------------------------------------------------------------ guard bands
GUARD = 4096  # bytes of canary before and after each buffer


def _guarded(n_elems, dtype):
    """A device buffer of n_elems inside canary bands (every byte 0xA5)."""
    esz = torch.empty(0, dtype=dtype).element_size()
    g = GUARD // esz
    raw = torch.full((GUARD * 2 + n_elems * esz,), 0xA5, dtype=torch.uint8, device=U.dev())
    inner = raw[GUARD:GUARD + n_elems * esz].view(dtype)
    return raw, inner, g


def _bands_intact(raw, name):
    head = U.from_dev(raw[:GUARD])
    tail = U.from_dev(raw[-GUARD:])
    assert (head == 0xA5).all() and (tail == 0xA5).all(), f"{name}: canary overwritten"


@pytest.mark.parametrize("name", ["llama7b_layer", "prefill_skew16", "wide_requests"])
def test_guard_bands_untouched(L, name):
    """Grouping, the row gather, the unfused FFN (h in the workspace) and the
    fused FFN (rows gathered and scattered through perm) write nothing outside
    their buffers; the fused output equals the unfused one bit for bit."""
    w = wl.WORKLOADS[name]
    _say("guards", name)
    x = U.to_dev(wl.make_x(w))
    wr, b = wl.make_router(w)
    if w.router:
        ids, _ = L.readme_route(x, U.to_dev(wr), None if b is None else U.to_dev(b))
    else:
        ids = U.to_dev(wl.make_request_ids(w))
    T, d = w.T, w.d
    bufs = {}
    for nm, n, dt in [("counts", w.E, torch.int32), ("offsets", w.E + 1, torch.int32),
                      ("perm", T, torch.int32), ("inv", T, torch.int32),
                      ("x_g", T * d, x.dtype), ("y_g", T * d, x.dtype), ("y", T * d, x.dtype),
                      ("h_unfused", L.readme_moe_ffn_workspace_bytes(x.dtype, T, w.I),
                       torch.uint8),
                      ("h_fused", L.readme_moe_ffn_workspace_bytes(x.dtype, T, w.I),
                       torch.uint8)]:
        bufs[nm] = _guarded(n, dt)
    inner = {k: v[1] for k, v in bufs.items()}
    L.readme_group_by_expert(ids, w.E, x=x, counts=inner["counts"], offsets=inner["offsets"],
                             perm=inner["perm"], inv_perm=inner["inv"],
                             x_grouped=inner["x_g"].view(T, d))
    packed = L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w)))
    L.readme_moe_ffn(inner["x_g"].view(T, d), inner["offsets"], packed, w.E, w.I,
                     y_grouped=inner["y_g"].view(T, d), workspace=inner["h_unfused"])
    y_ref = L.readme_ungroup(inner["y_g"].view(T, d), inner["inv"])
    L.readme_moe_ffn_fused(x, inner["perm"], inner["offsets"], packed, w.E, w.I,
                           y=inner["y"].view(T, d), workspace=inner["h_fused"])
    torch.cuda.synchronize()
    for nm, (raw, _, _) in bufs.items():
        _bands_intact(raw, f"{name} {nm}")
    assert (U.from_dev(inner["y"].view(T, d)) == U.from_dev(y_ref)).all()


# ------------------------------------------------------------ fused moves
@pytest.mark.parametrize("name", ["tiny_f32", "llama7b_layer", "prefill_skew16",
                                  "wide_requests"])
def test_fused_row_moves_equal_unfused(L, name):
    """Gather in the gate/up loads and scatter in the down epilogue give the
    same bits as the separate gather, FFN and ungroup calls."""
    w = wl.WORKLOADS[name]
    _say("fused", name)
    x = U.to_dev(wl.make_x(w))
    wr, b = wl.make_router(w)
    if w.router:
        ids, _ = L.readme_route(x, U.to_dev(wr), None if b is None else U.to_dev(b))
    else:
        ids = U.to_dev(wl.make_request_ids(w))
    counts, offs, perm, inv, xg = L.readme_group_by_expert(ids, w.E, x=x)
    packed = L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w)))
    y_ref = L.readme_ungroup(L.readme_moe_ffn(xg, offs, packed, w.E, w.I), inv)
    y = L.readme_moe_ffn_fused(x, perm, offs, packed, w.E, w.I)
    torch.cuda.synchronize()
    assert (U.from_dev(y) == U.from_dev(y_ref)).all()


def test_fused_leaves_unrouted_rows_untouched(L):
    T, d, E, I = 300, 128, 5, 96
    w = wl.Workload("t", T=T, d=d, E=E, I=I, dtype="bf16")
    x = U.to_dev(wl.make_x(w, 12))
    rng = np.random.default_rng(12)
    ids_h = rng.integers(-1, E + 1, size=T).astype(np.int32)
    counts, offs, perm, inv, xg = L.readme_group_by_expert(U.to_dev(ids_h), E, x=x)
    packed = L.readme_pack_experts(*U.weights_to_dev(*wl.make_experts(w, 12)))
    y = torch.full((T, d), 7.0, dtype=torch.bfloat16, device=U.dev())
    L.readme_moe_ffn_fused(x, perm, offs, packed, E, I, y=y)
    y_ref = L.readme_ungroup(L.readme_moe_ffn(xg, offs, packed, E, I), inv)
    torch.cuda.synchronize()
    yh, rh = U.from_dev(y), U.from_dev(y_ref)
    routed = (ids_h >= 0) & (ids_h < E)
    assert (yh[routed] == rh[routed]).all()
    assert (wl.bf16_bits_to_f32(yh[~routed]) == 7.0).all()


