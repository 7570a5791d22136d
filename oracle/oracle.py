"""Python face of the CPU oracle (``liboracle.so``, built from oracle.c).

TEST INFRASTRUCTURE.  Only the test suite, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` import this module.  The product path never
does, and nothing here imports the HIP library.

Arrays are numpy: bf16 tensors are ``uint16`` bit patterns, fp32 tensors are
``float32``.  Every function is a thin ctypes call into oracle.c, whose
comments give the definitions and the paper passages they follow.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "oracle.c")
F32, BF16 = 0, 1

_lib = None


def build(force: bool = True) -> str:
    """Compile oracle.c with gcc (no reassociation, no contraction)."""
    if force or not os.path.exists(LIB_PATH):
        tmp = LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
               "-ffp-contract=off", "-fno-fast-math", "-Wall", "-Wextra",
               SRC_PATH, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build(force=True)
        lib = ctypes.CDLL(LIB_PATH)
        P, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
        lib.oracle_route.argtypes = [ctypes.c_int, I64, I64, I32, P, P, P, P, P]
        lib.oracle_group.argtypes = [I64, I32, P, P, P, P, P]
        lib.oracle_gather.argtypes = [ctypes.c_int, I64, I64, P, P, P]
        lib.oracle_ungroup.argtypes = [I64, I64, P, P, P]
        lib.oracle_moe_ffn_rows.argtypes = [ctypes.c_int, I64, I64, I32, I64,
                                            P, P, P, P, P, I64, P, P]
        lib.oracle_layer_rows.argtypes = [I64, I64, I32, I64, P, P, P, P, P,
                                          ctypes.c_float, I64, P, P, P]
        lib.oracle_f32_to_bf16.argtypes = [I64, P, P]
        lib.oracle_f32_to_bf16.restype = None
        lib.oracle_threads.argtypes = []
        lib.oracle_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"unsupported element type {a.dtype}")


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"{what}: oracle returned {rc}")


def route(x: np.ndarray, w_router: np.ndarray, bias: np.ndarray | None):
    """Top-1 ids and fp32 logits (canonical summation order, see oracle.c)."""
    x = np.ascontiguousarray(x)
    w_router = np.ascontiguousarray(w_router, dtype=x.dtype)
    T, d = x.shape
    E = w_router.shape[0]
    ids = np.empty(T, np.int32)
    logits = np.empty((T, E), np.float32)
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    _check(_load().oracle_route(_dtype_code(x), T, d, E, _p(x), _p(w_router),
                                _p(b), _p(ids), _p(logits)), "route")
    return ids, logits


def group(ids: np.ndarray, E: int):
    """(counts[E], offsets[E+1], perm[T], inv_perm[T]) of a stable counting sort."""
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    T = ids.shape[0]
    counts = np.empty(E, np.int32)
    offsets = np.empty(E + 1, np.int32)
    perm = np.empty(T, np.int32)
    inv = np.empty(T, np.int32)
    _check(_load().oracle_group(T, E, _p(ids), _p(counts), _p(offsets),
                                _p(perm), _p(inv)), "group")
    return counts, offsets, perm, inv


def gather(x: np.ndarray, perm: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x)
    perm = np.ascontiguousarray(perm, dtype=np.int32)
    T, d = x.shape
    out = np.empty_like(x)
    _check(_load().oracle_gather(_dtype_code(x), T, d, _p(perm), _p(x),
                                 _p(out)), "gather")
    return out


def ungroup(y_g: np.ndarray, inv_perm: np.ndarray) -> np.ndarray:
    y_g = np.ascontiguousarray(y_g)
    inv_perm = np.ascontiguousarray(inv_perm, dtype=np.int32)
    T = y_g.shape[0]
    out = np.empty_like(y_g)
    row_bytes = y_g.strides[0] if T > 0 else 1
    _check(_load().oracle_ungroup(T, row_bytes, _p(inv_perm), _p(y_g),
                                  _p(out)), "ungroup")
    return out


def moe_ffn(x_g, offsets, w_gate, w_up, w_down, rows=None) -> np.ndarray:
    """fp64 expert FFN of the grouped rows (all rows, or the listed ones)."""
    x_g = np.ascontiguousarray(x_g)
    T, d = x_g.shape
    E, I, _ = w_gate.shape
    w_gate = np.ascontiguousarray(w_gate, dtype=x_g.dtype)
    w_up = np.ascontiguousarray(w_up, dtype=x_g.dtype)
    w_down = np.ascontiguousarray(w_down, dtype=x_g.dtype)
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    if rows is None:
        n = int(offsets[E])
        r = None
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        n = r.shape[0]
    y = np.empty((n, d), np.float64)
    _check(_load().oracle_moe_ffn_rows(_dtype_code(x_g), T, d, E, I, _p(x_g),
                                       _p(offsets), _p(w_gate), _p(w_up),
                                       _p(w_down), n, _p(r), _p(y)), "moe_ffn")
    return y


def moe_ffn_permanent(x_g, offsets, w_gate, w_up, w_down, p_gate, p_up, p_down,
                      rows=None) -> np.ndarray:
    """fp64 FFN of a layer with a permanent expert (Sec. 3: a set of neurons
    that every token activates, beside the routed expert of Eq. 2):
    y[j] = F_{e_j}(x_g[j]) + F_perm(x_g[j]), F_perm the SwiGLU FFN with
    p_gate[P][d], p_up[P][d], p_down[d][P].  Both terms are moe_ffn's fp64
    evaluation; the permanent one as a single expert whose block is every
    routed row."""
    x_g = np.ascontiguousarray(x_g)
    E = w_gate.shape[0]
    routed = moe_ffn(x_g, offsets, w_gate, w_up, w_down, rows=rows)
    n = int(offsets[E])
    if rows is None:
        rows = np.arange(n)
    everyone = np.array([0, n], np.int32)
    perm_part = moe_ffn(x_g, everyone, p_gate[None], p_up[None],
                        np.ascontiguousarray(p_down)[None], rows=rows)
    return routed + perm_part


def layer(x_res, offsets, w_gate, w_up, w_down, eps=1e-5, rows=None,
          want_xn=False):
    """One decode-stack layer's FFN output (the residual increment), fp64."""
    x_res = np.ascontiguousarray(x_res, dtype=np.float32)
    T, d = x_res.shape
    E, I, _ = w_gate.shape
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    if rows is None:
        n = int(offsets[E])
        r = None
    else:
        r = np.ascontiguousarray(rows, dtype=np.int64)
        n = r.shape[0]
    y = np.empty((n, d), np.float64)
    xn = np.empty((n, d), np.uint16) if want_xn else None
    _check(_load().oracle_layer_rows(
        T, d, E, I, _p(x_res), _p(offsets),
        _p(np.ascontiguousarray(w_gate, dtype=np.uint16)),
        _p(np.ascontiguousarray(w_up, dtype=np.uint16)),
        _p(np.ascontiguousarray(w_down, dtype=np.uint16)),
        float(eps), n, _p(r), _p(y), _p(xn)), "layer")
    return (y, xn) if want_xn else y


def topk(logits: np.ndarray, K: int):
    """Top-K experts per token and their gate weights (Eq. 2 with K > 1).

    Selection decides integers, so it runs on the fp32 logits of ``route``
    (the canonical order) and compares only: slot k takes, among the experts
    not yet taken, the first one in ascending index order unless a later one
    has a strictly larger logit -- top-1 is ``route``'s argmax, ties go to the
    lower index and a NaN logit never beats another.  The weights are the
    softmax of the selected logits (fp64), renormalised over the K slots, so
    that K = 1 gives weight 1: the unweighted top-1 layer.
    Returns ids [T][K] int32 (descending logit) and weights [T][K] float64.
    """
    logits = np.asarray(logits, np.float32)
    T, E = logits.shape
    if not 1 <= K <= E:
        raise ValueError("need 1 <= K <= E")
    taken = np.zeros((T, E), bool)
    ids = np.empty((T, K), np.int32)
    rows = np.arange(T)
    for k in range(K):
        best_id = np.full(T, -1, np.int64)
        best = np.zeros(T, np.float32)
        for e in range(E):
            free = ~taken[:, e]
            first = free & (best_id < 0)
            better = free & (best_id >= 0) & (logits[:, e] > best)
            pick = first | better
            best_id = np.where(pick, e, best_id)
            best = np.where(pick, logits[:, e], best)
        ids[:, k] = best_id
        taken[rows, best_id] = True
    sel = logits[rows[:, None], ids].astype(np.float64)
    z = np.exp(sel - sel[:, :1])
    return ids, z / z.sum(axis=1, keepdims=True)


def combine(y_g: np.ndarray, inv_perm: np.ndarray, weights: np.ndarray) -> np.ndarray:
    """y[t] = sum over slots k (ascending) of weights[t,k] * y_g[inv_perm[t*K + k]],
    fp64 (the gate-weighted sum of Eq. 2 over the K selected experts)."""
    weights = np.asarray(weights, np.float64)
    T, K = weights.shape
    rows = np.asarray(inv_perm).reshape(T, K)
    y = np.zeros((T, y_g.shape[1]), np.float64)
    for k in range(K):
        y += weights[:, k:k + 1] * np.asarray(y_g, np.float64)[rows[:, k]]
    return y


def full_path_topk(x, w_router, bias, w_gate, w_up, w_down, K: int, rows=None):
    """route -> top-K -> group the T*K (token, slot) pairs -> expert FFN of each
    pair -> gate-weighted combine.  Pair p = t*K + k carries token t's k-th
    expert.  Returns ids [T][K], weights, counts, offsets, perm (pair index
    per grouped row), inv_perm (grouped row per pair) and y (fp64; only the
    listed token rows when ``rows`` is given, else all)."""
    E = w_gate.shape[0]
    _, logits = route(x, w_router, bias)
    ids, wts = topk(logits, K)
    counts, offsets, perm, inv = group(ids.reshape(-1), E)
    T = x.shape[0]
    toks = np.arange(T) if rows is None else np.asarray(rows, np.int64)
    need = inv.reshape(T, K)[toks].reshape(-1)            # grouped rows those tokens use
    x_pairs = np.ascontiguousarray(np.asarray(x)[perm // K])  # activation row of each pair
    y_need = moe_ffn(x_pairs, offsets, w_gate, w_up, w_down, rows=need)
    y = (wts[toks][:, :, None] * y_need.reshape(len(toks), K, -1)).sum(axis=1)
    return dict(ids=ids, weights=wts, logits=logits, counts=counts, offsets=offsets,
                perm=perm, inv_perm=inv, y=y)


def threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(_load().oracle_threads())


def f32_to_bf16(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a, dtype=np.float32)
    out = np.empty(a.shape, np.uint16)
    _load().oracle_f32_to_bf16(a.size, _p(a), _p(out))
    return out


def gate_weights(logits: np.ndarray, ids: np.ndarray) -> np.ndarray:
    """Gate value of each token's expert under a softmax over the router's
    logits (Eq. 2's factor G(x)_i with Eq. 4's softmax applied to G): the
    weighted top-1 variant, p_t = softmax(logits[t])[ids[t]], in fp64 on the
    fp32 logits.  NaN for tokens whose id is outside [0, E)."""
    lg = np.asarray(logits, np.float32).astype(np.float64)
    T, E = lg.shape
    ids = np.asarray(ids, np.int64)
    out = np.full(T, np.nan)
    for t in range(T):
        e = int(ids[t])
        if 0 <= e < E:
            z = np.exp(lg[t] - lg[t].max())
            out[t] = z[e] / z.sum()
    return out


def ungroup_scaled(y_g: np.ndarray, inv_perm: np.ndarray, row_scale: np.ndarray) -> np.ndarray:
    """y[t] = y_g[j] * row_scale[j], j = inv_perm[t]: the product of the
    element (exact in fp32) and the fp32 weight, rounded to fp32 (IEEE) and
    then to the element type (bf16: round to nearest even); zero rows where
    j < 0.  bf16 arrays are uint16 bit patterns."""
    inv = np.asarray(inv_perm, np.int64)
    scale = np.asarray(row_scale, np.float32)
    bf16 = y_g.dtype == np.uint16
    vals = (y_g.astype(np.uint32) << 16).view(np.float32) if bf16 else y_g.astype(np.float32)
    out = np.zeros(y_g.shape, np.float32)
    ok = inv >= 0
    out[ok] = vals[inv[ok]] * scale[inv[ok]][:, None]
    if bf16:
        res = f32_to_bf16(out)
        res[~ok] = 0
        return res
    return out


def full_path(x, w_router, bias, w_gate, w_up, w_down, ids=None, permanent=None):
    """route -> group -> gather -> expert FFN -> ungroup, one layer.

    Returns a dict with ids, logits, counts, offsets, perm, inv_perm, x_g,
    y_g (fp64) and y (fp64, token order).  ``ids`` given skips the router;
    ``permanent`` = (p_gate, p_up, p_down) adds the permanent expert.
    """
    E = w_gate.shape[0]
    logits = None
    if ids is None:
        ids, logits = route(x, w_router, bias)
    counts, offsets, perm, inv = group(ids, E)
    x_g = gather(x, perm)
    n = int(offsets[E])
    y_g = np.zeros(x.shape, np.float64)
    if permanent is None:
        y_g[:n] = moe_ffn(x_g, offsets, w_gate, w_up, w_down, rows=np.arange(n))
    else:
        y_g[:n] = moe_ffn_permanent(x_g, offsets, w_gate, w_up, w_down, *permanent,
                                    rows=np.arange(n))
    y = ungroup(y_g, inv)
    return dict(ids=ids, logits=logits, counts=counts, offsets=offsets,
                perm=perm, inv_perm=inv, x_g=x_g, y_g=y_g, y=y)
