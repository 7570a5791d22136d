"""ctypes binding of libreadme (include/readme.h), one function per C entry.

Argument marshalling only: tensors become device pointers, the current torch
stream becomes the stream argument, and a nonzero status raises.  Outputs the
caller does not pass are allocated with torch (device memory plumbing); all
arithmetic runs in the library's HIP kernels.  There is no fallback: if the
library is missing or no GPU is present, calls fail loudly.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libreadme.so")

README_F32, README_BF16 = 0, 1
README_MAX_EXPERTS = 256
README_MAX_PERMANENT_SLICES = 16

_STATUS = {0: "ok", 1: "invalid argument", 2: "unsupported size or type",
           3: "buffer smaller than required", 4: "HIP launch failed"}

# (name, restype, argtypes) of every exported symbol of readme.h.
_P, _I64, _I32, _SZ, _F = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                           ctypes.c_size_t, ctypes.c_float)
SIGNATURES = {
    "readme_status_string": (ctypes.c_char_p, [_I32]),
    "readme_abi_version": (_I32, []),
    "readme_route": (_I32, [_I32, _I64, _I64, _I32, _P, _P, _P, _P, _P, _P]),
    "readme_group_by_expert": (_I32, [_I64, _I32, _P, _P, _P, _P, _P, _I32, _I64,
                                      _P, _P, _P]),
    "readme_packed_experts_bytes": (_SZ, [_I32, _I32, _I64, _I64]),
    "readme_pack_experts": (_I32, [_I32, _I32, _I64, _I64, _P, _P, _P, _P, _SZ, _P]),
    "readme_padded_intermediate": (_I64, [_I64]),
    "readme_set_gemm_tile": (_I32, [_I32]),
    "readme_get_gemm_tile": (_I32, []),
    "readme_moe_ffn_workspace_bytes": (_SZ, [_I32, _I64, _I64]),
    "readme_moe_ffn": (_I32, [_I32, _I64, _I64, _I32, _I64, _P, _P, _P, _P, _P, _SZ, _P]),
    "readme_moe_gate_up": (_I32, [_I32, _I64, _I64, _I32, _I64, _P, _P, _P, _P, _P]),
    "readme_moe_ffn_fused": (_I32, [_I32, _I64, _I64, _I32, _I64, _P, _P, _P, _P, _P, _P, _SZ,
                                    _P]),
    "readme_moe_ffn_fused_noalloc": (_I32, [_I32, _I64, _I64, _I32, _I64, _P, _P, _P, _P, _P,
                                            _P]),
    "readme_moe_gate_up_gather": (_I32, [_I32, _I64, _I64, _I32, _I64, _P, _P, _P, _P, _P, _P]),
    "readme_moe_down_scatter": (_I32, [_I32, _I64, _I64, _I32, _I64, _P, _P, _P, _P, _P, _P]),
    "readme_moe_down": (_I32, [_I32, _I64, _I64, _I32, _I64, _P, _P, _P, _P, _P]),
    "readme_packed_experts_permanent_bytes": (_SZ, [_I32, _I32, _I64, _I64, _I64]),
    "readme_pack_experts_permanent": (_I32, [_I32, _I32, _I64, _I64, _I64, _P, _P, _P, _P, _P,
                                             _P, _P, _SZ, _P]),
    "readme_moe_ffn_permanent_workspace_bytes": (_SZ, [_I32, _I64, _I64, _I64]),
    "readme_moe_ffn_permanent": (_I32, [_I32, _I64, _I64, _I32, _I64, _I64, _P, _P, _P, _P, _P,
                                        _SZ, _P]),
    "readme_moe_ffn_permanent_fused": (_I32, [_I32, _I64, _I64, _I32, _I64, _I64, _P, _P, _P,
                                              _P, _P, _P, _SZ, _P]),
    "readme_moe_gate_up_permanent_gather": (_I32, [_I32, _I64, _I64, _I32, _I64, _I64, _P, _P,
                                                   _P, _P, _P, _P]),
    "readme_moe_down_permanent_scatter": (_I32, [_I32, _I64, _I64, _I32, _I64, _I64, _P, _P, _P,
                                                 _P, _P, _P]),
    "readme_topk": (_I32, [_I64, _I32, _I32, _P, _P, _P, _P]),
    "readme_moe_gate_up_gather_topk": (_I32, [_I32, _I64, _I64, _I32, _I64, _I32, _P, _P, _P, _P,
                                              _P, _P]),
    "readme_moe_ffn_topk": (_I32, [_I32, _I64, _I64, _I32, _I64, _I32, _P, _P, _P, _P, _P, _P,
                                   _SZ, _P]),
    "readme_combine_topk": (_I32, [_I32, _I64, _I64, _I32, _P, _P, _P, _P]),
    "readme_expert_batch": (_I32, [_I32, _P, _P, _I64, _P, _P, _P, _P, _P]),
    "readme_cache_simulate": (_I32, [_I32, _I64, _I64, _P, ctypes.c_uint64, _P, _P, _P]),
    "readme_offload_create": (_I32, [_I32, _I64, _I64, _I32, _I32, _I32, _P, _P, _P]),
    "readme_offload_stack": (_I32, [_P, _I64, _P, _P, _P, _P, _F, _P, _SZ, _P]),
    "readme_offload_stats": (_I32, [_P, _P, _P, _P]),
    "readme_offload_destroy": (None, [_P]),
    "readme_offload_last_plan": (_I32, [_P, _I64, _P, _P, _P, _P]),
    "readme_offload_plan": (_I32, [_I32, _I32, _I32, _I32, _I32, _P, _I32, _I64, _P, _P, _P,
                                   _P]),
    "readme_ungroup": (_I32, [_I32, _I64, _I64, _P, _P, _P, _P]),
    "readme_gate_weights": (_I32, [_I64, _I32, _P, _P, _P, _P, _P]),
    "readme_ungroup_scaled": (_I32, [_I32, _I64, _I64, _P, _P, _P, _P, _P]),
    "readme_moe_ffn_stack_workspace_bytes": (_SZ, [_I64, _I64, _I64]),
    "readme_moe_ffn_stack": (_I32, [_I64, _I64, _I32, _I64, _I32, _P, _P, _P, _F, _P,
                                    _SZ, _P]),
    "readme_moe_ffn_stack_counts": (_I32, [_I64, _I64, _I32, _I64, _I32, _P, _P, _P, _P, _F,
                                           _P, _SZ, _P]),
    "readme_router_tf_packed_bytes": (_SZ, [_I64, _I64]),
    "readme_router_tf_pack": (_I32, [_I64, _I64, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "readme_router_tf_workspace_bytes": (_SZ, [_I64, _I64, _I64]),
    "readme_router_tf_workspace_offset": (_I64, [_I64, _I64, _I64, _I32]),
    "readme_router_tf": (_I32, [_I64, _I32, _I64, _I64, _I32, _I64, _P, _P, _P, _P, _P, _P, _F,
                                _P, _P, _P, _SZ, _P]),
    "readme_request_positions": (_I32, [_I64, _I32, _P, _P, _P]),
    "readme_rope": (_I32, [_I64, _I32, _P, _P, _I64, _P]),
    "readme_attention_causal": (_I32, [_I64, _I32, _I32, _P, _P, _P, _P, _I64, _P, _I64, _P]),
}

# Workspace regions of readme_router_tf (README_RTF_*).
RTF_REGIONS = ("X", "A", "QKV", "O", "M", "H", "FEAT", "POS", "OFFS")

_lib = None


class ReadmeError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn}: status {status} ({_STATUS.get(status, 'unknown')})")
        self.status = status


def load() -> ctypes.CDLL:
    """Load libreadme.so (built in-tree by paper_2410_19123_amd.build)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run "
                              "`python -m paper_2410_19123_amd.build` first")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _call(name: str, *args) -> None:
    st = getattr(load(), name)(*args)
    if st != 0:
        raise ReadmeError(name, st)


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return README_F32
    if t.dtype == torch.bfloat16:
        return README_BF16
    raise ValueError(f"unsupported dtype {t.dtype}")


def _dev(*ts):
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("libreadme takes device tensors")
        if not t.is_contiguous():
            raise ValueError("libreadme takes contiguous tensors")


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def readme_route(x, w_router, bias=None, expert_ids=None, logits=None):
    """Top-1 expert id per token; returns (expert_ids, logits or None)."""
    T, d = x.shape
    E = w_router.shape[0]
    if expert_ids is None:
        expert_ids = torch.empty(T, dtype=torch.int32, device=x.device)
    _dev(x, w_router, bias, expert_ids, logits)
    if w_router.dtype != x.dtype or w_router.shape[1] != d:
        raise ValueError("w_router must be [E][d] of x's dtype")
    if bias is not None and (bias.dtype != torch.float32 or bias.numel() != E):
        raise ValueError("bias must be fp32 [E]")
    _call("readme_route", _dt(x), T, d, E, _p(x), _p(w_router), _p(bias), _p(expert_ids),
          _p(logits), _stream(x.device))
    return expert_ids, logits


def readme_group_by_expert(expert_ids, E, x=None, counts=None, offsets=None, perm=None,
                           inv_perm=None, x_grouped=None):
    """Group tokens by expert; returns (counts, offsets, perm, inv_perm, x_grouped)."""
    T = expert_ids.shape[0]
    dev = expert_ids.device
    counts = counts if counts is not None else torch.empty(E, dtype=torch.int32, device=dev)
    offsets = offsets if offsets is not None else torch.empty(E + 1, dtype=torch.int32, device=dev)
    perm = perm if perm is not None else torch.empty(T, dtype=torch.int32, device=dev)
    inv_perm = inv_perm if inv_perm is not None else torch.empty(T, dtype=torch.int32, device=dev)
    if x is not None and x_grouped is None:
        x_grouped = torch.empty_like(x)
    _dev(expert_ids, counts, offsets, perm, inv_perm, x, x_grouped)
    dt = _dt(x) if x is not None else README_BF16
    d = x.shape[1] if x is not None else 0
    _call("readme_group_by_expert", T, E, _p(expert_ids), _p(counts), _p(offsets), _p(perm),
          _p(inv_perm), dt, d, _p(x), _p(x_grouped), _stream(dev))
    return counts, offsets, perm, inv_perm, x_grouped


def readme_padded_intermediate(I: int) -> int:
    return int(load().readme_padded_intermediate(I))


def readme_set_gemm_tile(tile: int) -> None:
    """Force a grouped-GEMM tile configuration (0 = automatic)."""
    _call("readme_set_gemm_tile", tile)


def readme_packed_experts_bytes(dtype, E, d, I) -> int:
    return int(load().readme_packed_experts_bytes(_dt(torch.empty(0, dtype=dtype)), E, d, I))


def readme_pack_experts(w_gate, w_up, w_down, packed=None):
    """Repack [E][I][d], [E][I][d], [E][d][I] expert weights; returns packed bytes."""
    E, I, d = w_gate.shape
    dt = _dt(w_gate)
    nbytes = readme_packed_experts_bytes(w_gate.dtype, E, d, I)
    if packed is None:
        packed = torch.empty(nbytes, dtype=torch.uint8, device=w_gate.device)
    _dev(w_gate, w_up, w_down, packed)
    if w_up.shape != w_gate.shape or w_down.shape != (E, d, I):
        raise ValueError("expert weight shapes disagree")
    if w_up.dtype != w_gate.dtype or w_down.dtype != w_gate.dtype:
        raise ValueError("expert weight dtypes disagree")
    _call("readme_pack_experts", dt, E, d, I, _p(w_gate), _p(w_up), _p(w_down), _p(packed),
          packed.numel() * packed.element_size(), _stream(w_gate.device))
    return packed


def readme_moe_ffn_workspace_bytes(dtype, T, I) -> int:
    return int(load().readme_moe_ffn_workspace_bytes(_dt(torch.empty(0, dtype=dtype)), T, I))


def readme_moe_ffn(x_grouped, offsets, packed, E, I, y_grouped=None, workspace=None):
    """Every expert's SwiGLU FFN on its grouped token block; returns y_grouped."""
    T, d = x_grouped.shape
    if y_grouped is None:
        y_grouped = torch.empty_like(x_grouped)
    ws = readme_moe_ffn_workspace_bytes(x_grouped.dtype, T, I)
    if workspace is None:
        workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=x_grouped.device)
    _dev(x_grouped, offsets, packed, y_grouped, workspace)
    _call("readme_moe_ffn", _dt(x_grouped), T, d, E, I, _p(x_grouped), _p(offsets), _p(packed),
          _p(y_grouped), _p(workspace), workspace.numel() * workspace.element_size(),
          _stream(x_grouped.device))
    return y_grouped


def readme_moe_ffn_fused(x, perm, offsets, packed, E, I, y=None, workspace=None):
    """Gather + expert FFN + ungroup with the row moves inside the GEMMs;
    returns y in token order (rows of unrouted tokens are not written)."""
    T, d = x.shape
    if y is None:
        y = torch.empty_like(x)
    ws = readme_moe_ffn_workspace_bytes(x.dtype, T, I)
    if workspace is None:
        workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=x.device)
    _dev(x, perm, offsets, packed, y, workspace)
    _call("readme_moe_ffn_fused", _dt(x), T, d, E, I, _p(x), _p(perm), _p(offsets), _p(packed),
          _p(y), _p(workspace), workspace.numel() * workspace.element_size(),
          _stream(x.device))
    return y


def readme_moe_ffn_fused_noalloc(x, perm, offsets, packed, E, I, y):
    """readme_moe_ffn_fused with h in the library's fixed device array (no
    workspace); y (token order) must be given."""
    T, d = x.shape
    _dev(x, perm, offsets, packed, y)
    _call("readme_moe_ffn_fused_noalloc", _dt(x), T, d, E, I, _p(x), _p(perm), _p(offsets),
          _p(packed), _p(y), _stream(x.device))
    return y


def readme_moe_gate_up_gather(x, perm, offsets, packed, E, I, h=None):
    """readme_moe_gate_up reading activation rows through perm (token order x)."""
    T, d = x.shape
    if h is None:
        h = torch.empty(T, readme_padded_intermediate(I), dtype=x.dtype, device=x.device)
    _dev(x, perm, offsets, packed, h)
    _call("readme_moe_gate_up_gather", _dt(x), T, d, E, I, _p(x), _p(perm), _p(offsets),
          _p(packed), _p(h), _stream(x.device))
    return h


def readme_moe_down_scatter(h, perm, offsets, packed, E, I, d, y):
    """readme_moe_down writing output rows through perm (token order y)."""
    T = h.shape[0]
    _dev(h, perm, offsets, packed, y)
    _call("readme_moe_down_scatter", _dt(h), T, d, E, I, _p(h), _p(perm), _p(offsets),
          _p(packed), _p(y), _stream(h.device))
    return y


def readme_moe_gate_up(x_grouped, offsets, packed, E, I, h=None):
    """h = silu(W_gate x) * (W_up x) per grouped row; returns h [T][I padded]."""
    T, d = x_grouped.shape
    if h is None:
        h = torch.empty(T, readme_padded_intermediate(I), dtype=x_grouped.dtype,
                        device=x_grouped.device)
    _dev(x_grouped, offsets, packed, h)
    _call("readme_moe_gate_up", _dt(x_grouped), T, d, E, I, _p(x_grouped), _p(offsets),
          _p(packed), _p(h), _stream(x_grouped.device))
    return h


def readme_moe_down(h, offsets, packed, E, I, d, y_grouped=None):
    """y = W_down h per grouped row; returns y_grouped [T][d]."""
    T = h.shape[0]
    if y_grouped is None:
        y_grouped = torch.empty(T, d, dtype=h.dtype, device=h.device)
    _dev(h, offsets, packed, y_grouped)
    _call("readme_moe_down", _dt(h), T, d, E, I, _p(h), _p(offsets), _p(packed),
          _p(y_grouped), _stream(h.device))
    return y_grouped


def readme_packed_experts_permanent_bytes(dtype, E, d, I, P) -> int:
    return int(load().readme_packed_experts_permanent_bytes(
        _dt(torch.empty(0, dtype=dtype)), E, d, I, P))


def readme_pack_experts_permanent(w_gate, w_up, w_down, p_gate, p_up, p_down, packed=None):
    """Repack the routed experts ([E][I][d], [E][I][d], [E][d][I]) and the
    permanent expert ([P][d], [P][d], [d][P]); returns the packed bytes."""
    E, I, d = w_gate.shape
    P = p_gate.shape[0]
    dt = _dt(w_gate)
    nbytes = readme_packed_experts_permanent_bytes(w_gate.dtype, E, d, I, P)
    if packed is None:
        packed = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=w_gate.device)
    _dev(w_gate, w_up, w_down, p_gate, p_up, p_down, packed)
    if w_up.shape != w_gate.shape or w_down.shape != (E, d, I):
        raise ValueError("expert weight shapes disagree")
    if p_gate.shape != (P, d) or p_up.shape != (P, d) or p_down.shape != (d, P):
        raise ValueError("permanent expert shapes disagree")
    if any(t.dtype != w_gate.dtype for t in (w_up, w_down, p_gate, p_up, p_down)):
        raise ValueError("weight dtypes disagree")
    _call("readme_pack_experts_permanent", dt, E, d, I, P, _p(w_gate), _p(w_up), _p(w_down),
          _p(p_gate), _p(p_up), _p(p_down), _p(packed), packed.numel() * packed.element_size(),
          _stream(w_gate.device))
    return packed


def readme_moe_ffn_permanent_workspace_bytes(dtype, T, I, P) -> int:
    return int(load().readme_moe_ffn_permanent_workspace_bytes(
        _dt(torch.empty(0, dtype=dtype)), T, I, P))


def readme_moe_ffn_permanent(x_grouped, offsets, packed, E, I, P, y_grouped=None,
                             workspace=None):
    """Routed expert + permanent expert on the grouped rows; returns y_grouped."""
    T, d = x_grouped.shape
    if y_grouped is None:
        y_grouped = torch.empty_like(x_grouped)
    ws = readme_moe_ffn_permanent_workspace_bytes(x_grouped.dtype, T, I, P)
    if workspace is None:
        workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=x_grouped.device)
    _dev(x_grouped, offsets, packed, y_grouped, workspace)
    _call("readme_moe_ffn_permanent", _dt(x_grouped), T, d, E, I, P, _p(x_grouped),
          _p(offsets), _p(packed), _p(y_grouped), _p(workspace),
          workspace.numel() * workspace.element_size(), _stream(x_grouped.device))
    return y_grouped


def readme_moe_ffn_permanent_fused(x, perm, offsets, packed, E, I, P, y=None, workspace=None):
    """readme_moe_ffn_permanent with the row moves inside the GEMMs; returns y in
    token order (rows of unrouted tokens are not written)."""
    T, d = x.shape
    if y is None:
        y = torch.empty_like(x)
    ws = readme_moe_ffn_permanent_workspace_bytes(x.dtype, T, I, P)
    if workspace is None:
        workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=x.device)
    _dev(x, perm, offsets, packed, y, workspace)
    _call("readme_moe_ffn_permanent_fused", _dt(x), T, d, E, I, P, _p(x), _p(perm), _p(offsets),
          _p(packed), _p(y), _p(workspace), workspace.numel() * workspace.element_size(),
          _stream(x.device))
    return y


def readme_moe_gate_up_permanent_gather(x, perm, offsets, packed, E, I, P, h=None):
    """Gate/up half of readme_moe_ffn_permanent_fused; returns h [T][(1+P/I)*Ip]."""
    T, d = x.shape
    if h is None:
        h = torch.empty(T, (1 + P // I) * readme_padded_intermediate(I), dtype=x.dtype,
                        device=x.device)
    _dev(x, perm, offsets, packed, h)
    _call("readme_moe_gate_up_permanent_gather", _dt(x), T, d, E, I, P, _p(x), _p(perm),
          _p(offsets), _p(packed), _p(h), _stream(x.device))
    return h


def readme_moe_down_permanent_scatter(h, perm, offsets, packed, E, I, P, d, y):
    """Down half of readme_moe_ffn_permanent_fused: writes y[perm[j]]."""
    T = h.shape[0]
    _dev(h, perm, offsets, packed, y)
    _call("readme_moe_down_permanent_scatter", _dt(h), T, d, E, I, P, _p(h), _p(perm),
          _p(offsets), _p(packed), _p(y), _stream(h.device))
    return y


def readme_topk(logits, K, ids=None, weights=None):
    """Top-K experts and renormalised gate weights from fp32 logits [T][E];
    returns (ids [T*K] int32, weights [T*K] fp32)."""
    T, E = logits.shape
    if ids is None:
        ids = torch.empty(T * K, dtype=torch.int32, device=logits.device)
    if weights is None:
        weights = torch.empty(T * K, dtype=torch.float32, device=logits.device)
    _dev(logits, ids, weights)
    if logits.dtype != torch.float32:
        raise ValueError("logits must be fp32")
    _call("readme_topk", T, E, K, _p(logits), _p(ids), _p(weights), _stream(logits.device))
    return ids, weights


def readme_moe_gate_up_gather_topk(x, perm, offsets, packed, E, I, K, h=None):
    """Gate/up over the T*K grouped pair rows (activation row perm[j] // K)."""
    T, d = x.shape
    if h is None:
        h = torch.empty(T * K, readme_padded_intermediate(I), dtype=x.dtype, device=x.device)
    _dev(x, perm, offsets, packed, h)
    _call("readme_moe_gate_up_gather_topk", _dt(x), T, d, E, I, K, _p(x), _p(perm), _p(offsets),
          _p(packed), _p(h), _stream(x.device))
    return h


def readme_moe_ffn_topk(x, perm, offsets, packed, E, I, K, y_pairs=None, workspace=None):
    """Expert FFN of every (token, slot) pair; returns y_pairs [T*K][d] in pair order."""
    T, d = x.shape
    if y_pairs is None:
        y_pairs = torch.empty(T * K, d, dtype=x.dtype, device=x.device)
    ws = readme_moe_ffn_workspace_bytes(x.dtype, T * K, I)
    if workspace is None:
        workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=x.device)
    _dev(x, perm, offsets, packed, y_pairs, workspace)
    _call("readme_moe_ffn_topk", _dt(x), T, d, E, I, K, _p(x), _p(perm), _p(offsets),
          _p(packed), _p(y_pairs), _p(workspace), workspace.numel() * workspace.element_size(),
          _stream(x.device))
    return y_pairs


def readme_combine_topk(y_pairs, weights, K, y=None):
    """y[t] = sum_k weights[t*K+k] * y_pairs[t*K+k] (fp32, slot order)."""
    TK, d = y_pairs.shape
    T = TK // K
    if y is None:
        y = torch.empty(T, d, dtype=y_pairs.dtype, device=y_pairs.device)
    _dev(y_pairs, weights, y)
    _call("readme_combine_topk", _dt(y_pairs), T, d, K, _p(y_pairs), _p(weights), _p(y),
          _stream(y_pairs.device))
    return y


README_CACHE_POLICIES = {"belady": 0, "lru": 1, "fifo": 2, "random": 3}


def to_device(a, device="cuda:0") -> torch.Tensor:
    """Host array -> device tensor (uint16 arrays hold bf16 bit patterns)."""
    import numpy as np
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def from_device(t: torch.Tensor):
    """Device tensor -> host array (bf16 as uint16 bit patterns)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        import numpy as np
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def _host_i32(a):
    import numpy as np
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.c_void_p)


def readme_expert_batch(queues, max_tokens: int):
    """Alg. 1 on host lists of per-expert token queues; returns
    (batch list, taken per expert, visited experts)."""
    import numpy as np
    E = len(queues)
    offs = np.zeros(E + 1, np.int64)
    offs[1:] = np.cumsum([len(q) for q in queues])
    offs, p_offs = _host_i32(offs)
    items, p_items = _host_i32(np.concatenate([np.asarray(q, np.int64) for q in queues])
                               if offs[-1] else np.zeros(1))
    batch = np.zeros(max(max_tokens, 1), np.int32)
    taken = np.zeros(E, np.int32)
    visited = np.zeros(E, np.int32)
    blen, nv = ctypes.c_int64(0), ctypes.c_int32(0)
    _call("readme_expert_batch", E, p_offs, p_items, max_tokens,
          batch.ctypes.data_as(ctypes.c_void_p), ctypes.byref(blen),
          taken.ctypes.data_as(ctypes.c_void_p), visited.ctypes.data_as(ctypes.c_void_p),
          ctypes.byref(nv))
    return batch[:blen.value].tolist(), taken.tolist(), visited[:nv.value].tolist()


def readme_cache_simulate(refs, capacity: int, policy: str, seed: int = 0):
    """Cache replacement over a host reference sequence; returns
    (hits [n] bool, evicted [n] int, number of hits)."""
    import numpy as np
    refs, p_refs = _host_i32(refs)
    n = refs.shape[0]
    hits = np.zeros(max(n, 1), np.uint8)
    evicted = np.zeros(max(n, 1), np.int32)
    nh = ctypes.c_int64(0)
    _call("readme_cache_simulate", README_CACHE_POLICIES[policy], capacity, n, p_refs, seed,
          hits.ctypes.data_as(ctypes.c_void_p), evicted.ctypes.data_as(ctypes.c_void_p),
          ctypes.byref(nh))
    return hits[:n].astype(bool).tolist(), evicted[:n].tolist(), nh.value


def readme_offload_plan(counts_per_step, E: int, L: int, slots: int, policy: str,
                        lookahead: bool = True):
    """The offload executor's placement planner on host counts [steps][E];
    returns one (hit, slot, evicted key or -1) per reference."""
    import numpy as np
    counts, p_counts = _host_i32(np.asarray(counts_per_step, np.int64).reshape(-1, E))
    n_steps = counts.shape[0]
    cap = max(1, int(L * (counts > 0).sum()))
    hits = np.zeros(cap, np.uint8)
    slot = np.zeros(cap, np.int32)
    evicted = np.zeros(cap, np.int32)
    n = ctypes.c_int64(0)
    _call("readme_offload_plan", E, L, slots, README_CACHE_POLICIES[policy], n_steps, p_counts,
          1 if lookahead else 0, cap, hits.ctypes.data_as(ctypes.c_void_p),
          slot.ctypes.data_as(ctypes.c_void_p), evicted.ctypes.data_as(ctypes.c_void_p),
          ctypes.byref(n))
    return [(bool(hits[i]), int(slot[i]), int(evicted[i])) for i in range(n.value)]


class Offload:
    """Expert-offload executor (readme_offload_*): packed layers in pinned host
    memory, `slots` device slots, copies one layer ahead on its own stream."""

    def __init__(self, packed_layers, E, d, I, slots, policy="belady"):
        arr = (ctypes.c_void_p * len(packed_layers))(*[p.data_ptr() for p in packed_layers])
        h = ctypes.c_void_p()
        _call("readme_offload_create", E, d, I, len(packed_layers), slots,
              README_CACHE_POLICIES[policy], arr, ctypes.byref(h),
              _stream(packed_layers[0].device))
        self.h, self.E, self.d, self.I, self.L = h, E, d, I, len(packed_layers)

    def stack(self, x_resid_grouped, offsets, counts, next_counts=None, rms_eps=1e-5,
              workspace=None):
        import numpy as np
        T = x_resid_grouped.shape[0]
        ws = readme_moe_ffn_stack_workspace_bytes(T, self.d, self.I)
        if workspace is None:
            workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=x_resid_grouped.device)
        _dev(x_resid_grouped, offsets, workspace)
        c = np.ascontiguousarray(counts, dtype=np.int32)
        nc = None if next_counts is None else np.ascontiguousarray(next_counts, dtype=np.int32)
        _call("readme_offload_stack", self.h, T, _p(offsets), c.ctypes.data_as(ctypes.c_void_p),
              None if nc is None else nc.ctypes.data_as(ctypes.c_void_p), _p(x_resid_grouped),
              rms_eps, _p(workspace), workspace.numel() * workspace.element_size(),
              _stream(x_resid_grouped.device))
        return x_resid_grouped

    def last_plan(self):
        """The last step's references: (hit, slot, evicted key or -1) each."""
        import numpy as np
        n = ctypes.c_int64(0)
        st = load().readme_offload_last_plan(self.h, 0, None, None, None, ctypes.byref(n))
        if st not in (0, 3):
            raise ReadmeError("readme_offload_last_plan", st)
        cap = max(1, n.value)
        hits = np.zeros(cap, np.uint8)
        slot = np.zeros(cap, np.int32)
        evicted = np.zeros(cap, np.int32)
        _call("readme_offload_last_plan", self.h, cap, hits.ctypes.data_as(ctypes.c_void_p),
              slot.ctypes.data_as(ctypes.c_void_p), evicted.ctypes.data_as(ctypes.c_void_p),
              ctypes.byref(n))
        return [(bool(hits[i]), int(slot[i]), int(evicted[i])) for i in range(n.value)]

    def stats(self):
        h, m, b = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _call("readme_offload_stats", self.h, ctypes.byref(h), ctypes.byref(m), ctypes.byref(b))
        return h.value, m.value, b.value

    def close(self):
        if self.h:
            load().readme_offload_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def readme_gate_weights(logits, expert_ids, inv_perm, row_scale=None):
    """Softmax gate of each routed token at its expert, in grouped order."""
    T, E = logits.shape
    if row_scale is None:
        row_scale = torch.zeros(T, dtype=torch.float32, device=logits.device)
    _dev(logits, expert_ids, inv_perm, row_scale)
    _call("readme_gate_weights", T, E, _p(logits), _p(expert_ids), _p(inv_perm), _p(row_scale),
          _stream(logits.device))
    return row_scale


def readme_ungroup_scaled(y_grouped, inv_perm, row_scale, y=None):
    """Rows back to token order, each scaled by its grouped row's weight."""
    T, d = y_grouped.shape
    if y is None:
        y = torch.empty_like(y_grouped)
    _dev(y_grouped, inv_perm, row_scale, y)
    _call("readme_ungroup_scaled", _dt(y_grouped), T, d, _p(y_grouped), _p(inv_perm),
          _p(row_scale), _p(y), _stream(y_grouped.device))
    return y


def readme_ungroup(y_grouped, inv_perm, y=None):
    """Rows back to token order; returns y."""
    T, d = y_grouped.shape
    if y is None:
        y = torch.empty_like(y_grouped)
    _dev(y_grouped, inv_perm, y)
    _call("readme_ungroup", _dt(y_grouped), T, d, _p(y_grouped), _p(inv_perm), _p(y),
          _stream(y_grouped.device))
    return y


def readme_moe_ffn_stack_workspace_bytes(T, d, I) -> int:
    return int(load().readme_moe_ffn_stack_workspace_bytes(T, d, I))


def readme_moe_ffn_stack(x_resid_grouped, offsets, packed_layers, E, I, rms_eps=1e-5,
                         workspace=None, counts=None):
    """Run len(packed_layers) pre-norm residual MoE layers in place on x (fp32).
    counts (host, [E]): the batch's token counts, for the tile choice."""
    T, d = x_resid_grouped.shape
    if x_resid_grouped.dtype != torch.float32:
        raise ValueError("the residual stream is fp32")
    L = len(packed_layers)
    ws = readme_moe_ffn_stack_workspace_bytes(T, d, I)
    if workspace is None:
        workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=x_resid_grouped.device)
    _dev(x_resid_grouped, offsets, workspace, *packed_layers)
    ptrs = (ctypes.c_void_p * max(L, 1))(*[p.data_ptr() for p in packed_layers])
    if counts is None:
        _call("readme_moe_ffn_stack", T, d, E, I, L, ctypes.cast(ptrs, ctypes.c_void_p),
              _p(offsets), _p(x_resid_grouped), float(rms_eps), _p(workspace),
              workspace.numel() * workspace.element_size(), _stream(x_resid_grouped.device))
    else:
        c, pc = _host_i32(counts)
        _call("readme_moe_ffn_stack_counts", T, d, E, I, L, ctypes.cast(ptrs, ctypes.c_void_p),
              _p(offsets), pc, _p(x_resid_grouped), float(rms_eps), _p(workspace),
              workspace.numel() * workspace.element_size(), _stream(x_resid_grouped.device))
    return x_resid_grouped


def readme_router_tf_packed_bytes(D: int, F: int) -> int:
    return int(load().readme_router_tf_packed_bytes(D, F))


def readme_router_tf_pack(wq, wk, wv, wo, w1, w3, w2, packed=None):
    """Repack the router block's bf16 weights ([out][in] row-major);
    returns the packed bytes."""
    D = wq.shape[0]
    F = w1.shape[0]
    for t, shape in ((wq, (D, D)), (wk, (D, D)), (wv, (D, D)), (wo, (D, D)), (w1, (F, D)),
                     (w3, (F, D)), (w2, (D, F))):
        if tuple(t.shape) != shape or t.dtype != torch.bfloat16:
            raise ValueError("router weights must be bf16 [D][D] x4, [F][D] x2, [D][F]")
    nbytes = readme_router_tf_packed_bytes(D, F)
    if packed is None:
        packed = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=wq.device)
    _dev(wq, wk, wv, wo, w1, w3, w2, packed)
    _call("readme_router_tf_pack", D, F, _p(wq), _p(wk), _p(wv), _p(wo), _p(w1), _p(w3),
          _p(w2), _p(packed), packed.numel() * packed.element_size(), _stream(wq.device))
    return packed


def readme_router_tf_workspace_bytes(T: int, D: int, F: int) -> int:
    return int(load().readme_router_tf_workspace_bytes(T, D, F))


def readme_router_tf_workspace_offset(T: int, D: int, F: int, region: str) -> int:
    return int(load().readme_router_tf_workspace_offset(T, D, F, RTF_REGIONS.index(region)))


def readme_router_tf(tokens, req_offsets, emb, packed, F, w_router, bias=None, rms_eps=1e-5,
                     expert_ids=None, logits=None, workspace=None):
    """The router G over requests of tokens; returns (expert_ids, logits or
    None, workspace).  The workspace keeps every intermediate
    (router_tf_region reads one)."""
    T = tokens.shape[0]
    R = req_offsets.shape[0] - 1
    V, D = emb.shape
    E = w_router.shape[0]
    dev = tokens.device
    if tokens.dtype != torch.int32 or req_offsets.dtype != torch.int32:
        raise ValueError("tokens and req_offsets must be int32")
    if emb.dtype != torch.bfloat16 or w_router.dtype != torch.bfloat16 or \
            w_router.shape[1] != D:
        raise ValueError("emb [V][D] and w_router [E][D] must be bf16")
    if bias is not None and (bias.dtype != torch.float32 or bias.numel() != E):
        raise ValueError("bias must be fp32 [E]")
    if expert_ids is None:
        expert_ids = torch.empty(T, dtype=torch.int32, device=dev)
    ws = readme_router_tf_workspace_bytes(T, D, F)
    if workspace is None:
        workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=dev)
    _dev(tokens, req_offsets, emb, packed, w_router, bias, expert_ids, logits, workspace)
    _call("readme_router_tf", T, R, D, F, E, V, _p(tokens), _p(req_offsets), _p(emb), _p(packed),
          _p(w_router), _p(bias), rms_eps, _p(expert_ids), _p(logits), _p(workspace),
          workspace.numel() * workspace.element_size(), _stream(dev))
    return expert_ids, logits, workspace


def router_tf_region(workspace, T: int, D: int, F: int, region: str):
    """View of one intermediate in readme_router_tf's workspace."""
    off = readme_router_tf_workspace_offset(T, D, F, region)
    Fp = readme_padded_intermediate(F)
    shape, dt = {"X": ((T, D), torch.float32), "A": ((T, D), torch.bfloat16),
                 "QKV": ((T, 3 * D), torch.bfloat16), "O": ((T, D), torch.bfloat16),
                 "M": ((T, D), torch.bfloat16), "H": ((T, Fp), torch.bfloat16),
                 "FEAT": ((T, D), torch.bfloat16), "POS": ((T,), torch.int32),
                 "OFFS": ((2,), torch.int32)}[region]
    n = 1
    for v in shape:
        n *= v
    esz = torch.empty(0, dtype=dt).element_size()
    return workspace[off:off + n * esz].view(dt).view(shape)


def readme_request_positions(req_offsets, T: int, pos=None):
    """Each token's position in its request; returns pos [T] int32."""
    R = req_offsets.shape[0] - 1
    if pos is None:
        pos = torch.empty(T, dtype=torch.int32, device=req_offsets.device)
    _dev(req_offsets, pos)
    _call("readme_request_positions", T, R, _p(req_offsets), _p(pos),
          _stream(req_offsets.device))
    return pos


def readme_rope(x, pos, H: int):
    """RoPE in place on H heads of 128 per row of bf16 x [T][ld]; returns x."""
    T, ld = x.shape
    if x.dtype != torch.bfloat16:
        raise ValueError("x must be bf16")
    _dev(x, pos)
    _call("readme_rope", T, H, _p(pos), _p(x), ld, _stream(x.device))
    return x


def readme_attention_causal(q, k, v, pos, H: int, R: int = 1, o=None):
    """Causal attention inside each request (bf16 [T][ld], heads of 128);
    R (the number of requests) only picks the launch shape."""
    T, ld = q.shape
    if k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v shapes disagree")
    if o is None:
        o = torch.empty(T, H * 128, dtype=torch.bfloat16, device=q.device)
    _dev(q, k, v, pos, o)
    _call("readme_attention_causal", T, H, R, _p(pos), _p(q), _p(k), _p(v), ld, _p(o),
          o.shape[1], _stream(q.device))
    return o


def readme_status_string(status: int) -> str:
    return load().readme_status_string(status).decode()
