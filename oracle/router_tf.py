"""CPU oracle of the pre-gating router G: one causal transformer block over
each request's token prefix, then the gate over the experts (Sec. 2.3: G
reads the current and all previous tokens of the sequence; Table 1: one
layer, four heads, embedding, feature and MLP width 512, SwiGLU, RoPE,
RMSNorm; Eq. 2: G's output picks the expert).

TEST INFRASTRUCTURE.  Only the test suite and the smoke check use this
module; the product path never does.

Reading (the paper gives the block's type and sizes, not its wiring):
  x0 = E[token]                       fp32 residual (bf16 table entries)
  a  = bf16(rmsnorm(x0))              no gain, eps 1e-5, as the FFN layers
  q, k, v = bf16(a Wq^T), bf16(a Wk^T), bf16(a Wv^T)
  q, k <- bf16(RoPE(q, k))            per head of 128 dims, rotate-half pairs
                                      (i, i + 64), angle p * 10000^(-2i/128),
                                      p = the token's position in its request
  o  = bf16(softmax(q k^T / sqrt(128), causal within the request) v)
  x1 = fp32(x0 + o Wo^T)
  x2 = fp32(x1 + W2 (silu(W1 m) * W3 m)),  m = bf16(rmsnorm(x1)), the
                                      hidden product unrounded (as in the
                                      expert layers' oracle)
  f  = bf16(rmsnorm(x2))
  logits, id = the canonical fp32 gate of ``oracle.route`` on f.
Sums and products are fp64 here; the roundings to bf16 and fp32 sit where
the GPU path stores its intermediates (its precision at those points).
Token ids outside the vocabulary embed as zero rows.

Arrays: bf16 tensors are uint16 bit patterns, fp32 tensors float32.
"""
from __future__ import annotations

import math

import numpy as np

from . import oracle as O

HEAD_DIM = 128
ROPE_BASE = 10000.0
EPS = 1e-5


def _f(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> float64."""
    u = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def bf16(a: np.ndarray) -> np.ndarray:
    """Round to bf16 through fp32 (nearest, ties to even) -> bit patterns."""
    return O.f32_to_bf16(np.asarray(a, dtype=np.float32))


def positions(req_offsets: np.ndarray, T: int) -> np.ndarray:
    """Position of each token inside its request (requests are contiguous)."""
    pos = np.empty(T, np.int64)
    ro = np.asarray(req_offsets, dtype=np.int64)
    for r in range(len(ro) - 1):
        pos[ro[r]:ro[r + 1]] = np.arange(ro[r + 1] - ro[r])
    return pos


def embed(tokens: np.ndarray, emb_bits: np.ndarray) -> np.ndarray:
    """Embedding rows as the fp32 residual; out-of-range ids give zeros."""
    V, D = emb_bits.shape
    x = np.zeros((len(tokens), D), np.float32)
    ok = (tokens >= 0) & (tokens < V)
    x[ok] = _f(emb_bits[tokens[ok]]).astype(np.float32)
    return x


def rmsnorm_bf16(x32: np.ndarray, eps: float = EPS) -> np.ndarray:
    """bf16(x * r), r = 1 / sqrt(mean x^2 + eps), formed in fp32 as the GPU's
    pre-norm stores it (the same arithmetic as the FFN layer's input)."""
    x32 = np.asarray(x32, dtype=np.float32)
    ss = np.zeros(x32.shape[0], np.float32)
    for k in range(x32.shape[1]):                 # sequential fp32 sum over k
        ss = ss + x32[:, k] * x32[:, k]
    rs = np.float32(1.0) / np.sqrt(ss / np.float32(x32.shape[1]) + np.float32(eps))
    return bf16(x32 * rs[:, None])


def rope_f64(x: np.ndarray, pos: np.ndarray) -> np.ndarray:
    """Rotate-half RoPE in fp64 on [T][H*128] values (unrounded)."""
    x = np.asarray(x, dtype=np.float64)
    T, HD = x.shape
    half = HEAD_DIM // 2
    i = np.arange(half, dtype=np.float64)
    inv = ROPE_BASE ** (-2.0 * i / HEAD_DIM)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]   # [T][64]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    for h in range(HD // HEAD_DIM):
        a = x[:, h * HEAD_DIM:h * HEAD_DIM + half]
        b = x[:, h * HEAD_DIM + half:(h + 1) * HEAD_DIM]
        out[:, h * HEAD_DIM:h * HEAD_DIM + half] = a * c - b * s
        out[:, h * HEAD_DIM + half:(h + 1) * HEAD_DIM] = b * c + a * s
    return out


def rope(x_bits: np.ndarray, pos: np.ndarray) -> np.ndarray:
    """RoPE on bf16 [T][H*128] -> bf16."""
    return bf16(rope_f64(_f(x_bits), pos))


def attention_f64(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                  req_offsets: np.ndarray) -> np.ndarray:
    """Causal multi-head attention inside each request, fp64 (unrounded):
    o_t = sum_{j <= t, same request} softmax_j(q_t . k_j / sqrt(128)) v_j."""
    q, k, v = (np.asarray(a, dtype=np.float64) for a in (q, k, v))
    T, HD = q.shape
    out = np.zeros((T, HD), np.float64)
    scale = 1.0 / math.sqrt(HEAD_DIM)
    ro = np.asarray(req_offsets, dtype=np.int64)
    for r in range(len(ro) - 1):
        a, b = int(ro[r]), int(ro[r + 1])
        n = b - a
        if n == 0:
            continue
        mask = np.tril(np.ones((n, n), dtype=bool))
        for h in range(HD // HEAD_DIM):
            sl = slice(h * HEAD_DIM, (h + 1) * HEAD_DIM)
            s = (q[a:b, sl] @ k[a:b, sl].T) * scale
            s = np.where(mask, s, -np.inf)
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p = p / p.sum(axis=1, keepdims=True)
            out[a:b, sl] = p @ v[a:b, sl]
    return out


def attention(q_bits, k_bits, v_bits, req_offsets) -> np.ndarray:
    """Causal attention on bf16 inputs -> bf16 output."""
    return bf16(attention_f64(_f(q_bits), _f(k_bits), _f(v_bits), req_offsets))


def mlp_hidden(m_bits: np.ndarray, w1: np.ndarray, w3: np.ndarray) -> np.ndarray:
    """The SwiGLU MLP's hidden activations silu(W1 m) * (W3 m), fp64
    (unrounded), silu(z) = z / (1 + exp(-z)); W2 of this is the MLP's output."""
    mf = _f(m_bits)
    g, u = mf @ _f(w1).T, mf @ _f(w3).T
    return g / (1.0 + np.exp(-g)) * u


def router_tf(tokens, req_offsets, emb, wq, wk, wv, wo, w1, w3, w2, w_router, bias,
              eps: float = EPS) -> dict:
    """The whole router; returns the ids, the logits and every intermediate."""
    tokens = np.asarray(tokens, dtype=np.int64)
    T = len(tokens)
    ro = np.asarray(req_offsets, dtype=np.int64)
    assert ro[0] == 0 and ro[-1] == T and np.all(np.diff(ro) >= 0)
    pos = positions(ro, T)
    x0 = embed(tokens, emb)
    a = rmsnorm_bf16(x0, eps)
    af = _f(a)
    q = bf16(af @ _f(wq).T)
    k = bf16(af @ _f(wk).T)
    v = bf16(af @ _f(wv).T)
    qr, kr = rope(q, pos), rope(k, pos)
    o = attention(qr, kr, v, ro)
    x1 = (x0.astype(np.float64) + _f(o) @ _f(wo).T).astype(np.float32)
    offs = np.array([0, T], np.int32)
    delta = O.layer(x1, offs, w1[None], w3[None], w2[None], eps=eps)
    x2 = (x1.astype(np.float64) + delta).astype(np.float32)
    f = rmsnorm_bf16(x2, eps)
    ids, logits = O.route(f, w_router, bias)
    return dict(ids=ids, logits=logits, x0=x0, a=a, q=qr, k=kr, v=v, o=o, x1=x1, x2=x2,
                f=f, pos=pos)
