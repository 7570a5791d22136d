"""Parity of the pre-gating router G (Sec. 2.3, Table 1) on the GPU against
the oracle (oracle/router_tf.py), through the C ABI.

Each stage is checked teacher-forced: the oracle stage is fed the GPU's own
input of that stage (read from the forward's workspace), so the rounding of
one stage does not blur the check of the next.  Bars:
  positions, offsets, the gate's ids and logits     bit-exact;
  RoPE on given bf16 input                          bit-exact;
  norms of exact inputs (a) and of the GPU's own     at most one bf16 ulp off,
  residual (f)                                      on at most 1% of elements
                                                     (fp32 sums in another order);
  the MLP's norm m (of x1 = x0 + o Wo^T)            as a GEMM output, x1's
                                                     accumulation bound scaled by r;
  GEMM outputs (v, h)                               output rounding + 2^-16 of
                                                     sum |a_k w_k|, 98% bit-identical;
  rotated q, k                                      the same, with one ulp of each
                                                     pair's norm;
  attention                                         |o - o_exact| <= 2^-8 |o_exact|
                                                     + 2^-12 max|v| of the request
                                                     (bf16 output rounding; the
                                                     weights carry ~16 bits);
  the residual x                                    fp32 accumulation bound.
End to end, the ids must agree wherever the oracle's top-two logit gap
exceeds 0.05.
"""
import numpy as np
import pytest

from oracle import router_tf as R
from paper_2410_19123_amd import workloads as wl
from tests._util import from_dev, to_dev

pytestmark = pytest.mark.gpu

HD = 128


def _lib():
    from paper_2410_19123_amd import _lib
    return _lib


def _ord(bits):
    b = np.asarray(bits, dtype=np.uint16).astype(np.int64)
    return np.where(b & 0x8000, -(b & 0x7FFF), b)


def _ulps(a, b):
    return np.abs(_ord(a) - _ord(b))


def _near(got, ref, what, frac=0.01):
    """bf16 patterns equal up to one ulp, on at most `frac` of elements."""
    d = _ulps(got, ref)
    assert d.max() <= 1, f"{what}: {int(d.max())} ulps apart"
    off = float((d > 0).mean())
    assert off <= frac, f"{what}: {off:.3%} of elements one ulp off"
    return off


def _abs_sum(a_bits, w_bits):
    """sum_k |a_k| |w_k| per output: the scale of a GEMM output's fp32
    accumulation error (an output that cancels to near zero is many of its own
    ulps off, but never more than a small part of this)."""
    return np.abs(R._f(a_bits)) @ np.abs(R._f(w_bits)).T


def _gemm_near(got_bits, ref, scale, what):
    """bf16 GEMM outputs: within the output rounding (2^-8 |ref|) plus 2^-16
    of the accumulation scale; 98% bit-identical to bf16(ref)."""
    err = np.abs(R._f(got_bits) - ref)
    tol = 2.0 ** -8 * np.abs(ref) + 2.0 ** -16 * scale
    assert np.all(err <= tol), f"{what}: worst {float((err - tol).max()):.3e} over"
    same = float((got_bits == R.bf16(ref)).mean())
    assert same >= 0.98, f"{what}: only {same:.4f} bit-identical"


def _attention_ok(got_bits, q, k, v, ro, what):
    """got vs the exact (fp64) attention of the given bf16 q, k, v."""
    ref = R.attention_f64(R._f(q), R._f(k), R._f(v), ro)
    got = R._f(got_bits)
    vf = np.abs(R._f(v))
    T, HDt = ref.shape
    vmax = np.zeros((T, HDt // HD))
    for r in range(len(ro) - 1):
        a, b = int(ro[r]), int(ro[r + 1])
        if b > a:
            vmax[a:b] = vf[a:b].reshape(b - a, -1, HD).max(axis=(0, 2))
    tol = 2.0 ** -8 * np.abs(ref) + 2.0 ** -12 * np.repeat(vmax, HD, axis=1)
    err = np.abs(got - ref)
    bad = err > tol
    assert not bad.any(), (f"{what}: {int(bad.sum())} outside tolerance, worst "
                           f"{float((err - tol).max()):.3e}")
    # bit-identical to the oracle's rounded output on nearly every element
    same = float((got_bits == R.bf16(ref)).mean())
    assert same >= 0.95, f"{what}: only {same:.3f} bit-identical"


@pytest.mark.parametrize("offsets", [
    [0, 5], [0, 0, 5], [0, 5, 5], [0, 1, 2, 3], [0, 3, 3, 7, 200, 200, 333],
])
def test_request_positions(offsets):
    L = _lib()
    ro = np.array(offsets, np.int32)
    T = int(ro[-1])
    pos = from_dev(L.readme_request_positions(to_dev(ro), T))
    assert np.array_equal(pos, R.positions(ro, T))


@pytest.mark.parametrize("T,H,ld,maxpos", [(1, 1, 128, 1), (333, 2, 256, 9000),
                                           (1000, 3, 400, 70000)])
def test_rope_bit_exact(T, H, ld, maxpos):
    L = _lib()
    rng = np.random.default_rng(T)
    x = wl.to_bf16_bits(rng.standard_normal((T, ld)).astype(np.float32) * 3)
    pos = rng.integers(0, maxpos, size=T).astype(np.int32)
    got = from_dev(L.readme_rope(to_dev(x), to_dev(pos), H))
    ref = x.copy()
    ref[:, :H * HD] = R.rope(x[:, :H * HD], pos.astype(np.int64))
    assert np.array_equal(got, ref), f"{int((got != ref).sum())} elements differ"


ATTN_CASES = [
    ([1], 1, 1.0),
    ([37], 2, 1.0),
    ([32, 32, 32, 32, 32], 1, 2.0),
    ([0, 1, 31, 33, 0, 127, 128, 129, 5], 2, 1.5),
    ([600], 1, 3.0),
    ([300, 45, 0, 211, 1, 1], 4, 1.0),
    ([1000, 3, 700], 2, 2.0),
]


@pytest.mark.parametrize("lengths,H,scale", ATTN_CASES)
def test_attention_matches_oracle(lengths, H, scale):
    """Both launch shapes (one wave per 32 queries; eight waves per 128
    queries in two groups over alternate key blocks, merged at the end) on
    every case."""
    L = _lib()
    ro = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    T = int(ro[-1])
    rng = np.random.default_rng(sum(lengths) + H)
    q, k, v = (wl.to_bf16_bits(rng.standard_normal((T, H * HD)).astype(np.float32) * s)
               for s in (scale, scale, 1.0))
    pos = R.positions(ro, T).astype(np.int32)
    dq, dk, dv, dp = to_dev(q), to_dev(k), to_dev(v), to_dev(pos)
    short = from_dev(L.readme_attention_causal(dq, dk, dv, dp, H, R=max(T, 1)))
    long_ = from_dev(L.readme_attention_causal(dq, dk, dv, dp, H, R=1))
    _attention_ok(short, q, k, v, ro, f"attention {lengths} H={H}, one wave")
    _attention_ok(long_, q, k, v, ro, f"attention {lengths} H={H}, split keys")


def _forward(shape, lengths, seed, bad_tokens=False):
    """Run the GPU router; returns (inputs, outputs, workspace regions).
    bad_tokens: a few ids outside the vocabulary (they embed as zeros)."""
    L = _lib()
    import torch
    w = wl.make_router_tf(shape, seed)
    tokens, ro = wl.make_router_requests(lengths, shape.V, seed)
    if bad_tokens and len(tokens) >= 3:
        tokens[0], tokens[len(tokens) // 2], tokens[-1] = -1, shape.V, 2 ** 31 - 1
    T = len(tokens)
    dw = {n: to_dev(w[n]) for n in ("wq", "wk", "wv", "wo", "w1", "w3", "w2")}
    packed = L.readme_router_tf_pack(dw["wq"], dw["wk"], dw["wv"], dw["wo"], dw["w1"],
                                     dw["w3"], dw["w2"])
    logits = torch.empty(T, shape.E, dtype=torch.float32, device="cuda:0")
    ids, logits, ws = L.readme_router_tf(to_dev(tokens), to_dev(ro), to_dev(w["emb"]), packed,
                                         shape.F, to_dev(w["w_router"]), None, 1e-5,
                                         logits=logits)
    regions = {n: from_dev(L.router_tf_region(ws, T, shape.D, shape.F, n))
               for n in L.RTF_REGIONS}
    return w, tokens, ro, from_dev(ids), from_dev(logits), regions


def _stage_checks(w, tokens, ro, ids, logits, g, rows=None):
    """Teacher-forced checks of every stage on the requests in `rows`
    (a slice of whole requests; all tokens when None)."""
    T = len(tokens)
    D = w["wq"].shape[0]
    F = w["w1"].shape[0]
    sl = slice(0, T) if rows is None else rows
    ro_s = ro[(ro >= sl.start) & (ro <= sl.stop)] - sl.start
    pos = R.positions(ro, T)
    assert np.array_equal(g["POS"], pos)
    assert np.array_equal(g["OFFS"], [0, T])
    # embedding and the pre-attention norm
    x0 = R.embed(tokens[sl].astype(np.int64), w["emb"])
    _near(g["A"][sl], R.rmsnorm_bf16(x0), "a")
    # projections (from the GPU's a) and RoPE
    af = R._f(g["A"][sl])
    qkv = g["QKV"][sl]
    _gemm_near(qkv[:, 2 * D:], af @ R._f(w["wv"]).T, _abs_sum(g["A"][sl], w["wv"]), "v")
    # RoPE mixes each pair (i, i + 64): a GEMM rounding difference before it
    # moves both rotated values by up to one ulp of the pair's norm, plus the
    # accumulation scale of either input.
    for what, wn, got in (("q", "wq", qkv[:, :D]), ("k", "wk", qkv[:, D:2 * D])):
        ref = R.rope(R.bf16(af @ R._f(w[wn]).T), pos[sl])
        sc = _abs_sum(g["A"][sl], w[wn]).reshape(-1, D // HD, 2, 64)
        gf, rf = R._f(got).reshape(sc.shape), R._f(ref).reshape(sc.shape)
        norm = np.sqrt((rf ** 2).sum(axis=2, keepdims=True))
        tol = 2.0 ** -7 * norm + 2.0 ** -16 * sc.sum(axis=2, keepdims=True)
        assert np.all(np.abs(gf - rf) <= tol), what
        assert (got != ref).mean() <= 0.02, what
    # attention (from the GPU's q, k, v)
    _attention_ok(g["O"][sl], qkv[:, :D], qkv[:, D:2 * D], qkv[:, 2 * D:], ro_s, "o")
    # residual + Wo, MLP norm, MLP, residual (from the GPU's o, m, h)
    of = R._f(g["O"][sl])
    x1 = x0.astype(np.float64) + of @ R._f(w["wo"]).T
    # m = bf16(x1 r): the GPU's x1 carries its fp32 accumulation error
    # (2^-16 of |x0| + sum |o||Wo| bounds it), which r scales, and an element
    # of x1 that cancels to near zero is many of its own ulps off
    b1 = np.abs(x0) + np.abs(of) @ np.abs(R._f(w["wo"])).T
    r = 1.0 / np.sqrt((x1 ** 2).mean(axis=1, keepdims=True) + R.EPS)
    _gemm_near(g["M"][sl], x1 * r, r * b1, "m")
    # h = silu(g) u: g's accumulation error enters times |u| (silu' <= 1.1),
    # u's times |silu(g)| <= |g|
    mf = R._f(g["M"][sl])
    gt, up = mf @ R._f(w["w1"]).T, mf @ R._f(w["w3"]).T
    sc = 1.1 * np.abs(up) * _abs_sum(g["M"][sl], w["w1"]) + \
        np.abs(gt) * _abs_sum(g["M"][sl], w["w3"])
    Fp = g["H"].shape[1]
    _gemm_near(g["H"][sl][:, :F], R.mlp_hidden(g["M"][sl], w["w1"], w["w3"]), sc, "h")
    assert np.all(g["H"][sl][:, F:Fp] == 0)
    hf = R._f(g["H"][sl][:, :F])
    x2 = x1 + hf @ R._f(w["w2"]).T
    bound = (np.abs(x0) + np.abs(of) @ np.abs(R._f(w["wo"])).T
             + np.abs(hf) @ np.abs(R._f(w["w2"])).T)
    err = np.abs(g["X"][sl].astype(np.float64) - x2)
    assert np.all(err <= 2.0 ** -16 * bound), float((err / bound).max())
    # final norm and the gate (from the GPU's x and f)
    _near(g["FEAT"][sl], R.rmsnorm_bf16(g["X"][sl]), "f")
    from oracle import oracle as O
    ids_ref, logits_ref = O.route(g["FEAT"][sl], w["w_router"], None)
    assert np.array_equal(ids[sl], ids_ref)
    assert np.array_equal(logits[sl], logits_ref)


def _end_to_end(w, tokens, ro, ids, logits, rows=None):
    sl = slice(0, len(tokens)) if rows is None else rows
    ro_s = ro[(ro >= sl.start) & (ro <= sl.stop)] - sl.start
    out = R.router_tf(tokens[sl].astype(np.int64), ro_s, w["emb"], w["wq"], w["wk"], w["wv"],
                      w["wo"], w["w1"], w["w3"], w["w2"], w["w_router"], None)
    if out["logits"].shape[1] == 1:
        clear = np.ones(len(out["ids"]), bool)
    else:
        top2 = np.sort(out["logits"], axis=1)[:, -2:]
        clear = (top2[:, 1] - top2[:, 0]) > 0.05
    assert np.array_equal(ids[sl][clear], out["ids"][clear])
    assert np.abs(logits[sl] - out["logits"]).max() <= 0.02
    return float((ids[sl] == out["ids"]).mean())


@pytest.mark.parametrize("lengths", [
    [1],
    [5, 0, 130, 33, 1],
    list(wl.ragged_lengths(700, 9, 0)),
])
def test_router_tf_small(oracle_mod, lengths):
    shape = wl.RouterShape(D=256, F=192, V=1000, E=5)
    w, tokens, ro, ids, logits, g = _forward(shape, lengths, 1)
    _stage_checks(w, tokens, ro, ids, logits, g)
    _end_to_end(w, tokens, ro, ids, logits)


@pytest.mark.parametrize("D,F,V,E,lengths", [
    (128, 100, 50, 3, [3, 0, 40]),            # one head; F padded to 128
    (1152, 64, 300, 20, [7, 70]),             # nine heads, norm+gate with 3 chunks/lane, E = 20
    (2176, 96, 300, 1, [5, 33]),              # 17 heads: norm, then the separate gate; E = 1
])
def test_router_tf_shapes(oracle_mod, D, F, V, E, lengths):
    """Widths off Table 1: head counts 1, 9 and 17 (each path of the fused
    final norm and gate), a padded MLP width, 1 and 20 experts, and ids
    outside the vocabulary."""
    shape = wl.RouterShape(D=D, F=F, V=V, E=E)
    w, tokens, ro, ids, logits, g = _forward(shape, lengths, 2, bad_tokens=True)
    _stage_checks(w, tokens, ro, ids, logits, g)
    _end_to_end(w, tokens, ro, ids, logits)


def test_router_tf_many_requests(oracle_mod):
    """5000 requests (most of one token or empty) over 6000 tokens: the
    request offsets no longer fit the workgroup's LDS copy, so positions come
    from the search in global memory."""
    L = _lib()
    lengths = wl.ragged_lengths(6000, 5000, 7)
    ro = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    pos = from_dev(L.readme_request_positions(to_dev(ro), 6000))
    assert np.array_equal(pos, R.positions(ro, 6000))
    shape = wl.RouterShape(D=128, F=64, V=500, E=4)
    w, tokens, ro2, ids, logits, g = _forward(shape, lengths, 7)
    assert np.array_equal(ro2, ro)
    _stage_checks(w, tokens, ro, ids, logits, g)
    _end_to_end(w, tokens, ro, ids, logits)


def test_router_tf_table1_request_batch(oracle_mod):
    """Table 1's router on the request batch (256 requests x 32 tokens), the
    launch the benchmark times: every stage on every token."""
    shape = wl.ROUTER_TABLE1
    w, tokens, ro, ids, logits, g = _forward(shape, [32] * 256, 0)
    assert ids.min() >= 0 and ids.max() < shape.E
    _stage_checks(w, tokens, ro, ids, logits, g)
    _end_to_end(w, tokens, ro, ids, logits)


def test_router_tf_table1_long_prompts(oracle_mod):
    """Table 1's router on long prompts (8 x 1024 tokens, the split-key
    attention): every stage on every token."""
    shape = wl.ROUTER_TABLE1
    w, tokens, ro, ids, logits, g = _forward(shape, [1024] * 8, 1)
    _stage_checks(w, tokens, ro, ids, logits, g)
    _end_to_end(w, tokens, ro, ids, logits)


def test_router_tf_empty_batch():
    L = _lib()
    import torch
    shape = wl.RouterShape(D=128, F=64, V=10, E=2)
    w = wl.make_router_tf(shape, 0)
    dw = {n: to_dev(w[n]) for n in ("wq", "wk", "wv", "wo", "w1", "w3", "w2")}
    packed = L.readme_router_tf_pack(dw["wq"], dw["wk"], dw["wv"], dw["wo"], dw["w1"],
                                     dw["w3"], dw["w2"])
    tokens = torch.empty(0, dtype=torch.int32, device="cuda:0")
    ro = to_dev(np.zeros(1, np.int32))
    ids, _, _ = L.readme_router_tf(tokens, ro, to_dev(w["emb"]), packed, shape.F,
                                   to_dev(w["w_router"]))
    assert ids.numel() == 0
