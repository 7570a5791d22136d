"""Seeded synthetic workloads for the pre-gated expert-FFN layer.

This module only draws inputs.  It holds none of the layer's arithmetic: no
routing, grouping or FFN maths lives here, so that both the CPU oracle (under
``oracle/``) and the HIP path can be fed from it without sharing any code
with each other.

Shapes follow the paper's setting: the experts are contiguous slices of the
intermediate columns of one dense Llama-style SwiGLU FFN (Sec. 3, the expert
form F_i(x) = W_2 M_i^T sigma(M_i W_1 x) with M_i a selection matrix), and the
router is a layer-independent gate evaluated once per token ahead of all
layers (Sec. 2.3, Eq. 2).  Because the trained router and checkpoints are not
available, the router is a linear map d -> E with a fixed logit bias that
produces the load imbalance of the named workload.

Values:
  * every tensor is drawn with numpy's PCG64 from a substream keyed by
    ``[seed, tag, layer, chunk]`` (all keys have this one length); chunks of 2**22 elements are independent
    substreams, so any tensor (or any layer of a stack) can be regenerated on
    its own and in parallel;
  * N(0, 1) activations, N(0, 0.02) weights, drawn in fp32;
  * bf16 workloads round each fp32 draw to bf16 (round to nearest even) and
    keep the raw 16-bit patterns as ``uint16`` arrays.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

# Substream tags.
TAG_X, TAG_ROUTER, TAG_GATE, TAG_UP, TAG_DOWN, TAG_REQ = 1, 2, 3, 4, 5, 6
TAG_RTF = 7  # the transformer router's weights and tokens (sub-tag in the layer key)
_CHUNK = 1 << 22

# Logit bias constant for expert 0 of the prefill-scale skewed layer
# (T=16384, d=4096, E=16).  Chosen so that expert 0 receives about 40% of the
# tokens at seed 0; written by oracle/calibrate_skew_bias.py.
SKEW_BIAS0 = 0.2826


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic MoE-layer workload.

    T tokens of width d, E experts each a SwiGLU FFN of intermediate width I,
    ``layers`` stacked layers sharing one routing (the pre-gating router runs
    once per step).  ``router`` is False when expert ids are given per request
    instead of computed.  ``P`` > 0 adds a permanent expert of P intermediate
    neurons that every token passes through; ``K`` > 1 routes each token to
    its K highest-logit experts.
    """
    name: str
    T: int
    d: int
    E: int
    I: int
    dtype: str            # "f32" or "bf16"
    P: int = 0
    K: int = 1
    batching: str = ""    # "alg1" | "fifo": batches drawn from a pool of waiting requests
    pool: int = 0         # waiting decode requests the batches are drawn from
    offload_slots: int = 0  # >0: weights in host memory, a device cache of this many slots
    policy: str = ""      # the cache's replacement rule: "belady" | "lru"
    layers: int = 1
    router: bool = True
    bias: str = "none"    # "none" | "zipf1" | "skew40_zipf1.2"
    requests: int = 0     # >0: ids are per request of T // requests tokens
    description: str = ""

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    def with_T(self, T: int) -> "Workload":
        return dataclasses.replace(self, T=T)


WORKLOADS = {
    "tiny_f32": Workload(
        "tiny_f32", T=256, d=512, E=4, I=512, dtype="f32",
        description="tiny fp32 MoE layer: T=256, d=512, E=4, I=512, linear "
                    "router 512->4, top-1, no bias"),
    "llama7b_layer": Workload(
        "llama7b_layer", T=2048, d=4096, E=8, I=1376, dtype="bf16",
        bias="zipf1",
        description="Llama-7B-shaped MoE layer: T=2048, d=4096, E=8, "
                    "I=1376 (11008/8 split), Zipf(1.0) router bias"),
    "llama7b_decode32": Workload(
        "llama7b_decode32", T=64, d=4096, E=8, I=1376, dtype="bf16",
        layers=32, bias="zipf1",
        description="decode step: 64 tokens through 32 stacked Llama-7B-"
                    "shaped MoE layers, routed once"),
    "llama7b_decode32_alg1": Workload(
        "llama7b_decode32_alg1", T=64, d=4096, E=8, I=1376, dtype="bf16",
        layers=32, router=False, batching="alg1", pool=1024,
        description="serving loop: 64-token decode batches formed by expert-aware "
                    "batching (Alg. 1) from 1024 waiting requests, 32 stacked "
                    "Llama-7B-shaped MoE layers"),
    "llama7b_decode32_fifo": Workload(
        "llama7b_decode32_fifo", T=64, d=4096, E=8, I=1376, dtype="bf16",
        layers=32, router=False, batching="fifo", pool=1024,
        description="serving loop: 64-token decode batches taken first-come "
                    "first-served from 1024 waiting requests, 32 stacked "
                    "Llama-7B-shaped MoE layers"),
    "llama7b_decode8_offload_belady": Workload(
        "llama7b_decode8_offload_belady", T=64, d=4096, E=8, I=1376, dtype="bf16",
        layers=8, router=False, batching="fifo", pool=1024, offload_slots=24,
        policy="belady",
        description="serving loop with expert offload: 64-token first-come "
                    "first-served decode batches through 8 Llama-7B-shaped MoE "
                    "layers whose experts live in host memory, 24 device slots "
                    "of the 64 (layer, expert) pairs, Belady replacement"),
    "llama7b_decode8_offload_lru": Workload(
        "llama7b_decode8_offload_lru", T=64, d=4096, E=8, I=1376, dtype="bf16",
        layers=8, router=False, batching="fifo", pool=1024, offload_slots=24,
        policy="lru",
        description="as llama7b_decode8_offload_belady with LRU replacement"),
    "prefill_skew16": Workload(
        "prefill_skew16", T=16384, d=4096, E=16, I=688, dtype="bf16",
        bias="skew40_zipf1.2",
        description="prefill-scale skewed layer: T=16384, d=4096, E=16, "
                    "I=688, expert 0 ~40%, rest Zipf(1.2)"),
    "llama7b_layer_perm": Workload(
        "llama7b_layer_perm", T=2048, d=4096, E=8, I=1376, P=1376, dtype="bf16",
        bias="zipf1",
        description="Llama-7B-shaped MoE layer with a permanent expert: T=2048, "
                    "d=4096, E=8 routed experts of I=1376 plus P=1376 neurons "
                    "every token passes through, Zipf(1.0) router bias"),
    "llama7b_layer_top2": Workload(
        "llama7b_layer_top2", T=2048, d=4096, E=8, I=1376, K=2, dtype="bf16",
        bias="zipf1",
        description="Llama-7B-shaped MoE layer with top-2 routing: T=2048, "
                    "d=4096, E=8, I=1376, each token on its two highest-logit "
                    "experts with renormalised softmax weights"),
    "wide_requests": Workload(
        "wide_requests", T=8192, d=8192, E=8, I=3584, dtype="bf16",
        router=False, requests=256,
        description="expert-aware batch: 256 requests x 32 tokens, d=8192, "
                    "E=8, I=3584, one expert id per request"),
}


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def normal(shape, std: float, key) -> np.ndarray:
    """fp32 draws of N(0, std^2), chunked into independent substreams."""
    n = int(np.prod(shape))
    out = np.empty(n, np.float32)
    nchunks = (n + _CHUNK - 1) // _CHUNK

    def fill(c):
        s = c * _CHUNK
        e = min(n, s + _CHUNK)
        rng = np.random.default_rng(list(key) + [c])
        rng.standard_normal(e - s, dtype=np.float32, out=out[s:e])
        if std != 1.0:
            out[s:e] *= np.float32(std)

    if nchunks <= 1:
        for c in range(nchunks):
            fill(c)
    else:
        with ThreadPoolExecutor(min(_threads(), nchunks)) as ex:
            list(ex.map(fill, range(nchunks)))
    return out.reshape(shape)


def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest even) and return the 16-bit patterns."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to fp32 exactly."""
    return (b.astype(np.uint32) << 16).view(np.float32)


def _cast(w: Workload, a: np.ndarray) -> np.ndarray:
    return a if w.dtype == "f32" else to_bf16_bits(a)


def router_bias(w: Workload) -> np.ndarray | None:
    """Fixed per-expert logit bias giving the workload's load imbalance.

    zipf1: b_e = -ln(e+1), a Zipf(1.0) prior over experts.
    skew40_zipf1.2: b_e = -1.2 ln(e) for e >= 1 and the constant SKEW_BIAS0
    for expert 0.
    """
    if w.bias == "none" or not w.router:
        return None
    e = np.arange(w.E, dtype=np.float64)
    if w.bias == "zipf1":
        b = -np.log(e + 1.0)
    elif w.bias == "skew40_zipf1.2":
        b = np.empty(w.E)
        b[0] = SKEW_BIAS0
        b[1:] = -1.2 * np.log(e[1:])
    else:
        raise ValueError(w.bias)
    return b.astype(np.float32)


def make_x(w: Workload, seed: int = 0) -> np.ndarray:
    """Activations x[T][d] ~ N(0, 1)."""
    return _cast(w, normal((w.T, w.d), 1.0, [seed, TAG_X, 0]))


def make_router(w: Workload, seed: int = 0):
    """Router weight W_r[E][d] ~ N(0, 0.02) and bias (fp32, or None)."""
    if not w.router:
        return None, None
    return _cast(w, normal((w.E, w.d), 0.02, [seed, TAG_ROUTER, 0])), router_bias(w)


def make_request_ids(w: Workload, seed: int = 0) -> np.ndarray:
    """Given ids: one uniform expert id per request, repeated over its tokens."""
    per = w.T // w.requests
    rng = np.random.default_rng([seed, TAG_REQ, 0, 0])
    req = rng.integers(0, w.E, size=w.requests).astype(np.int32)
    return np.repeat(req, per).astype(np.int32)


def make_locality_ids(steps: int, batch: int, E: int, seed: int = 0,
                      keep: float = 2921 / 4096, zipf: float = 1.0) -> np.ndarray:
    """Expert ids [steps][batch] of decode requests with temporal locality:
    each request keeps its previous token's expert with probability `keep`
    (2921/4096, the share of tokens that follow the previous token's expert
    reported in Sec. 5.3), else draws one with probability proportional to
    (e+1)^-zipf."""
    rng = np.random.default_rng([seed, 0x5EED])
    p = 1.0 / np.arange(1, E + 1, dtype=np.float64) ** zipf
    p /= p.sum()
    ids = np.empty((steps, batch), np.int32)
    ids[0] = rng.choice(E, size=batch, p=p)
    for s in range(1, steps):
        stay = rng.random(batch) < keep
        ids[s] = np.where(stay, ids[s - 1], rng.choice(E, size=batch, p=p))
    return ids


def make_pool(w: Workload, seed: int = 0):
    """Expert id of each of the w.pool waiting requests (probability
    proportional to 1/(e+1)) and the random stream that draws their later
    tokens' experts."""
    rng = np.random.default_rng([seed, 0xB47C])
    p = 1.0 / np.arange(1, w.E + 1, dtype=np.float64)
    p /= p.sum()
    return rng.choice(w.E, size=w.pool, p=p).astype(np.int32), rng, p


def make_dense(w: Workload, seed: int = 0, layer: int = 0):
    """The dense FFN the experts are sliced from: (W_gate[D][d], W_up[D][d],
    W_down[d][D]) with D = E*I + P, in the workload's dtype."""
    D = w.E * w.I + w.P
    wg = normal((D, w.d), 0.02, [seed, TAG_GATE, layer])
    wu = normal((D, w.d), 0.02, [seed, TAG_UP, layer])
    wd = normal((w.d, D), 0.02, [seed, TAG_DOWN, layer])
    return _cast(w, wg), _cast(w, wu), _cast(w, wd)


def make_experts(w: Workload, seed: int = 0, layer: int = 0):
    """Routed expert weights of one layer, sliced from one dense SwiGLU FFN.

    The dense FFN has intermediate width D = E*I + P; expert e owns
    intermediate columns [e*I, (e+1)*I) (the permanent expert, if any, the
    last P).  Returns (w_gate[E][I][d], w_up[E][I][d], w_down[E][d][I]).
    """
    dg, du, dd = make_dense(w, seed, layer)
    n = w.E * w.I
    wg = dg[:n].reshape(w.E, w.I, w.d)
    wu = du[:n].reshape(w.E, w.I, w.d)
    wd = np.ascontiguousarray(dd[:, :n].reshape(w.d, w.E, w.I).transpose(1, 0, 2))
    return np.ascontiguousarray(wg), np.ascontiguousarray(wu), wd


def make_permanent(w: Workload, seed: int = 0, layer: int = 0):
    """The permanent expert of one layer: intermediate columns [E*I, E*I + P)
    of the same dense FFN.  Returns (p_gate[P][d], p_up[P][d], p_down[d][P])."""
    if w.P <= 0:
        raise ValueError(f"workload {w.name} has no permanent expert")
    dg, du, dd = make_dense(w, seed, layer)
    n = w.E * w.I
    return (np.ascontiguousarray(dg[n:]), np.ascontiguousarray(du[n:]),
            np.ascontiguousarray(dd[:, n:]))


def flops_per_layer(w: Workload) -> float:
    """Algorithmic FLOP of the expert FFN of one layer: 6*T*d*(I + P)."""
    return 6.0 * w.T * w.d * (w.I + w.P)


def describe(w: Workload) -> str:
    return w.description or w.name


__all__ = [
    "Workload", "WORKLOADS", "normal", "to_bf16_bits", "bf16_bits_to_f32",
    "router_bias", "make_x", "make_router", "make_request_ids",
    "make_experts", "make_permanent", "make_dense", "make_locality_ids", "make_pool", "flops_per_layer", "describe", "SKEW_BIAS0",
]


@dataclasses.dataclass(frozen=True)
class RouterShape:
    """The pre-gating router G (Table 1): one transformer block of width D
    (D / 128 heads of 128), SwiGLU MLP width F, vocabulary V, and a gate to
    E experts."""
    D: int = 512
    F: int = 512
    V: int = 32000
    E: int = 8


# Table 1's router, gating the eight experts of the request batch.
ROUTER_TABLE1 = RouterShape()


def make_router_tf(r: RouterShape, seed: int = 0) -> dict:
    """Random-init bf16 weights of G ([out][in] row-major bit patterns):
    emb [V][D] ~ N(0, 1) (rows of the norm's output scale), the projections
    wq, wk, wv, wo [D][D], w1, w3 [F][D], w2 [D][F] and the gate w_router
    [E][D] ~ N(0, 0.02).  No gate bias (the block's output sets the load)."""
    def b(sub, shape, std):
        return to_bf16_bits(normal(shape, std, [seed, TAG_RTF, sub]))
    D, F = r.D, r.F
    return dict(emb=b(1, (r.V, D), 1.0), wq=b(2, (D, D), 0.02), wk=b(3, (D, D), 0.02),
                wv=b(4, (D, D), 0.02), wo=b(5, (D, D), 0.02), w1=b(6, (F, D), 0.02),
                w3=b(7, (F, D), 0.02), w2=b(8, (D, F), 0.02), w_router=b(9, (r.E, D), 0.02),
                bias=None)


def make_router_requests(lengths, V: int, seed: int = 0):
    """Token ids uniform over [0, V) for requests of the given lengths
    (zero allowed); returns (tokens [T] int32, req_offsets [R+1] int32)."""
    lengths = np.asarray(lengths, dtype=np.int64)
    offs = np.zeros(len(lengths) + 1, np.int64)
    np.cumsum(lengths, out=offs[1:])
    rng = np.random.default_rng([seed, TAG_RTF, 100, 0])
    tokens = rng.integers(0, V, size=int(offs[-1])).astype(np.int32)
    return tokens, offs.astype(np.int32)


def ragged_lengths(T: int, R: int, seed: int = 0):
    """R request lengths summing to T, cut at R - 1 uniform points (so some
    may be zero and a few long)."""
    rng = np.random.default_rng([seed, TAG_RTF, 101, 0])
    cuts = np.sort(rng.integers(0, T + 1, size=R - 1))
    return np.diff(np.concatenate([[0], cuts, [T]])).astype(np.int64)
