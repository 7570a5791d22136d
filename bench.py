"""Benchmark of the pre-gated expert-FFN hot path on one MI355X.

One step = one pass of the whole path over one batch resident in HBM:
route (top-1 router) -> group (histogram, scan, stable permute, row gather)
-> expert FFN (fused gate/up + SiLU*mul, then down) -> ungroup.  For the
stacked decode workload a step is route + group + L layers + ungroup.

Default workload: the expert-aware request batch (256 requests x 32 tokens,
T=8192, d=8192, E=8 experts of intermediate width 3584, bf16, one given
expert id per request), the largest configuration that fits one GPU.
Expert weights rotate through several packed copies so that every step
reads them cold from HBM, as the layers of a real model stack do.

Prints ONE JSON line:  value = tokens per second through one MoE layer,
plus a per-kernel breakdown from HIP events on the launch stream, the
roofline of the dominant kernel (the gate/up GEMM, MFMA-bound here) and
the CPU oracle's rate on a bounded sample (rank 0, one GPU).  Beside it
the same line carries the metric's two halves, each from a short run of
its own: "decode" (the 32-layer decode stack, 64 tokens, against HBM
bandwidth) and "prefill" (the skewed 16-expert prefill layer's gate/up
GEMM, T=16384, against the bf16 MFMA peak).

    python bench.py [--gpus 1] [--steps 100] [--warmup 10] [--workload NAME]
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2410_19123_amd import workloads as wl  # noqa: E402

HBM_GBS = 8000.0          # MI355X HBM3E peak, GB/s
MFMA_BF16_TFLOPS = 2500.0  # dense bf16 MFMA peak
MFMA_F32_TFLOPS = 157.3
VALU_F32_TFLOPS = 78.6     # non-packed fp32 FMA: 256 CU x 64 lanes x 2 x 2.4 GHz


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="wide_requests", choices=sorted(wl.WORKLOADS))
    ap.add_argument("--weight-copies", type=int, default=0,
                    help="packed weight copies to rotate (0 = enough for >= 1 GiB)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target length of the oracle's timed sample")
    ap.add_argument("--unfused", action="store_true",
                    help="separate row gather / ungroup calls instead of the row moves "
                         "fused into the two GEMMs")
    ap.add_argument("--gemm-tile", type=int, default=0,
                    help="force a grouped-GEMM tile configuration (0 = automatic)")
    ap.add_argument("--no-side", action="store_true",
                    help="skip the decode-stack and prefill lines measured beside the main one")
    ap.add_argument("--side-steps", type=int, default=20,
                    help="timed steps of each side line")
    ap.add_argument("--library-gemm", action="store_true",
                    help="also time the same per-expert GEMMs with torch's library GEMM "
                         "(context for the grouped kernels; not part of the path)")
    ap.add_argument("--router-only", action="store_true",
                    help="time only the pre-gating router G (Table 1) on the request "
                         "batch's tokens and print its line")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration)")
    return ap.parse_args()


def serving_schedule(w: wl.Workload, steps: int, lib, seed: int = 0):
    """Expert ids [steps][T] of the decode batches a serving loop forms from
    w.pool waiting requests: first-come first-served, or expert-aware
    batching (Alg. 1, the library's readme_expert_batch).  After a step each
    scheduled request's next token re-enters the pool at the back, keeping
    its expert with probability 2921/4096 (the locality reported in
    Sec. 5.3), else drawing one with probability proportional to 1/(e+1)."""
    import collections
    expert, rng, p = wl.make_pool(w, seed)
    expert = expert.tolist()
    queues = [collections.deque() for _ in range(w.E)]
    arrival = collections.deque(range(w.pool))
    for r in range(w.pool):
        queues[expert[r]].append(r)
    out = np.empty((steps, w.T), np.int32)
    for st in range(steps):
        if w.batching == "alg1":
            batch, taken, _ = lib.readme_expert_batch([list(q) for q in queues], w.T)
            for e in range(w.E):
                for _ in range(taken[e]):
                    queues[e].popleft()
        else:
            batch = [arrival.popleft() for _ in range(w.T)]
        out[st] = [expert[r] for r in batch]
        keep = rng.random(len(batch)) < 2921 / 4096
        fresh = rng.choice(w.E, size=len(batch), p=p)
        for j, r in enumerate(batch):
            expert[r] = expert[r] if keep[j] else int(fresh[j])
            if w.batching == "alg1":
                queues[expert[r]].append(r)
            else:
                arrival.append(r)
    return out


class Path:
    """Pre-marshalled C-ABI calls of one step (host overhead kept small so
    that the GPU, not Python, sets the pace)."""

    def __init__(self, w: wl.Workload, copies: int, seed: int = 0):
        import torch

        from paper_2410_19123_amd import _lib

        class U:  # host -> device copies of the seeded inputs
            to_dev = staticmethod(_lib.to_device)

            @staticmethod
            def weights_to_dev(*ws):
                return tuple(_lib.to_device(a) for a in ws)

        self.torch, self.w, self.lib = torch, w, _lib.load()
        dev = torch.device("cuda:0")
        x = wl.make_x(w, seed)
        self.x = U.to_dev(x)
        wr, b = wl.make_router(w, seed)
        self.wr = U.to_dev(wr) if wr is not None else None
        self.bias = U.to_dev(b) if b is not None else None
        if w.batching:
            # one scheduled batch per weight copy (the copies are the layers)
            self.sched = serving_schedule(w, max(w.layers, 1), _lib, seed)
            self.sched_ids = U.to_dev(self.sched)
            self.ids = self.sched_ids[0]
        else:
            self.ids = (torch.empty(w.T, dtype=torch.int32, device=dev) if w.router
                        else U.to_dev(wl.make_request_ids(w, seed)))
        # Top-K: router logits, then the T*K (token, slot) pairs are routed.
        NP = w.T * w.K
        if w.K > 1:
            self.logits = torch.empty(w.T, w.E, dtype=torch.float32, device=dev)
            self.pair_ids = torch.empty(NP, dtype=torch.int32, device=dev)
            self.weights = torch.empty(NP, dtype=torch.float32, device=dev)
            self.y_pairs = torch.empty(NP, w.d, dtype=self.x.dtype, device=dev)
        self.dt = _lib.README_F32 if w.dtype == "f32" else _lib.README_BF16
        i32 = torch.int32
        self.counts = torch.empty(w.E, dtype=i32, device=dev)
        self.offsets = torch.empty(w.E + 1, dtype=i32, device=dev)
        self.perm = torch.empty(NP, dtype=i32, device=dev)
        self.inv = torch.empty(NP, dtype=i32, device=dev)
        self.xg = torch.empty_like(self.x)
        self.yg = torch.empty_like(self.x)
        self.y = torch.empty_like(self.x)
        self.Ip = _lib.readme_padded_intermediate(w.I)
        # h holds the routed expert's neurons, then the permanent expert's
        # (P / I slices of one expert's width).
        self.h = torch.empty(NP, (1 + w.P // w.I) * self.Ip, dtype=self.x.dtype, device=dev)
        self.packed = []
        for layer in range(w.layers):
            wts = U.weights_to_dev(*wl.make_experts(w, seed, layer=layer))
            if w.P:
                p = _lib.readme_pack_experts_permanent(
                    *wts, *U.weights_to_dev(*wl.make_permanent(w, seed, layer=layer)))
            else:
                p = _lib.readme_pack_experts(*wts)
            self.packed.append(p)
            del wts
        if w.layers == 1:
            for _ in range(copies - 1):
                self.packed.append(self.packed[0].clone())
        self.ex = None
        if w.offload_slots:
            # Weights live in pinned host memory behind a device slot cache.
            self.ex = _lib.Offload(self.packed, w.E, w.d, w.I, w.offload_slots, w.policy)
        if w.layers > 1:
            # The stack's residual stream is fp32; the router reads bf16 features.
            self.x32 = self.x.float()
            self.xres = torch.empty(w.T, w.d, dtype=torch.float32, device=dev)
            self.yres = torch.empty_like(self.xres)
            ws = _lib.readme_moe_ffn_stack_workspace_bytes(w.T, w.d, w.I)
            self.ws = torch.empty(ws, dtype=torch.uint8, device=dev)
            self.layer_ptrs = (ctypes.c_void_p * w.layers)(*[p.data_ptr() for p in self.packed])
        torch.cuda.synchronize()
        self.stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        P = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())  # noqa: E731
        self.P = P

    def _ok(self, st, name):
        if st != 0:
            raise RuntimeError(f"{name} failed with status {st}")

    def route(self):
        if not self.w.router:
            return
        P, w = self.P, self.w
        self._ok(self.lib.readme_route(self.dt, w.T, w.d, w.E, P(self.x), P(self.wr),
                                       P(self.bias), P(self.ids),
                                       P(self.logits) if w.K > 1 else None, self.stream),
                 "route")

    def topk(self):
        P, w = self.P, self.w
        self._ok(self.lib.readme_topk(w.T, w.E, w.K, P(self.logits), P(self.pair_ids),
                                      P(self.weights), self.stream), "topk")

    def group_pairs(self):
        P, w = self.P, self.w
        self._ok(self.lib.readme_group_by_expert(
            w.T * w.K, w.E, P(self.pair_ids), P(self.counts), P(self.offsets), P(self.perm),
            P(self.inv), self.dt, w.d, None, None, self.stream), "group")

    def gate_up_pairs(self, k):
        P, w = self.P, self.w
        self._ok(self.lib.readme_moe_gate_up_gather_topk(
            self.dt, w.T, w.d, w.E, w.I, w.K, P(self.x), P(self.perm), P(self.offsets),
            P(self.packed[k]), P(self.h), self.stream), "gate_up_gather_topk")

    def down_pairs(self, k):
        P, w = self.P, self.w
        self._ok(self.lib.readme_moe_down_scatter(
            self.dt, w.T * w.K, w.d, w.E, w.I, P(self.h), P(self.perm), P(self.offsets),
            P(self.packed[k]), P(self.y_pairs), self.stream), "down_scatter")

    def combine(self):
        P, w = self.P, self.w
        self._ok(self.lib.readme_combine_topk(self.dt, w.T, w.d, w.K, P(self.y_pairs),
                                              P(self.weights), P(self.y), self.stream),
                 "combine")

    def group(self):
        P, w = self.P, self.w
        self._ok(self.lib.readme_group_by_expert(
            w.T, w.E, P(self.ids), P(self.counts), P(self.offsets), P(self.perm), P(self.inv),
            self.dt, w.d, P(self.x), P(self.xg), self.stream), "group")

    def gate_up(self, k):
        P, w = self.P, self.w
        self._ok(self.lib.readme_moe_gate_up(self.dt, w.T, w.d, w.E, w.I, P(self.xg),
                                             P(self.offsets), P(self.packed[k]), P(self.h),
                                             self.stream), "gate_up")

    def down(self, k):
        P, w = self.P, self.w
        self._ok(self.lib.readme_moe_down(self.dt, w.T, w.d, w.E, w.I, P(self.h),
                                          P(self.offsets), P(self.packed[k]), P(self.yg),
                                          self.stream), "down")

    def ungroup(self):
        P, w = self.P, self.w
        self._ok(self.lib.readme_ungroup(self.dt, w.T, w.d, P(self.yg), P(self.inv), P(self.y),
                                         self.stream), "ungroup")

    def group_resid(self, k=0):
        """Group tokens and gather the fp32 residual rows into grouped order
        (a serving loop's k-th scheduled batch when batches are scheduled)."""
        P, w = self.P, self.w
        ids = self.sched_ids[k % self.sched_ids.shape[0]] if w.batching else self.ids
        self._ok(self.lib.readme_group_by_expert(
            w.T, w.E, P(ids), P(self.counts), P(self.offsets), P(self.perm), P(self.inv),
            0, w.d, P(self.x32), P(self.xres), self.stream), "group")

    def stack(self, k=0):
        P, w = self.P, self.w
        if w.batching:
            # The scheduler formed the batch, so its expert counts are known on
            # the host: the library picks tiles for the actual split.
            n = self.sched.shape[0]
            cnt = np.ascontiguousarray(np.bincount(self.sched[k % n], minlength=w.E), np.int32)
            self._ok(self.lib.readme_moe_ffn_stack_counts(
                w.T, w.d, w.E, w.I, w.layers, ctypes.cast(self.layer_ptrs, ctypes.c_void_p),
                P(self.offsets), cnt.ctypes.data_as(ctypes.c_void_p), P(self.xres),
                ctypes.c_float(1e-5), P(self.ws), self.ws.numel(), self.stream), "stack")
            return
        self._ok(self.lib.readme_moe_ffn_stack(
            w.T, w.d, w.E, w.I, w.layers, ctypes.cast(self.layer_ptrs, ctypes.c_void_p),
            P(self.offsets), P(self.xres), ctypes.c_float(1e-5), P(self.ws),
            self.ws.numel(), self.stream), "stack")

    def offload_stack(self, k):
        """The stack through the offload executor; the host knows each
        scheduled batch's expert counts (and the next one's)."""
        n = self.sched.shape[0]
        cnt = np.bincount(self.sched[k % n], minlength=self.w.E)
        nxt = np.bincount(self.sched[(k + 1) % n], minlength=self.w.E)
        self.ex.stack(self.xres, self.offsets, cnt, nxt, workspace=self.ws)

    def ungroup_resid(self):
        P, w = self.P, self.w
        self._ok(self.lib.readme_ungroup(0, w.T, w.d, P(self.xres), P(self.inv),
                                         P(self.yres), self.stream), "ungroup")

    def group_only(self):
        P, w = self.P, self.w
        self._ok(self.lib.readme_group_by_expert(
            w.T, w.E, P(self.ids), P(self.counts), P(self.offsets), P(self.perm), P(self.inv),
            self.dt, w.d, None, None, self.stream), "group")

    def gate_up_gather(self, k):
        P, w = self.P, self.w
        if w.P:
            self._ok(self.lib.readme_moe_gate_up_permanent_gather(
                self.dt, w.T, w.d, w.E, w.I, w.P, P(self.x), P(self.perm), P(self.offsets),
                P(self.packed[k]), P(self.h), self.stream), "gate_up_permanent_gather")
            return
        self._ok(self.lib.readme_moe_gate_up_gather(
            self.dt, w.T, w.d, w.E, w.I, P(self.x), P(self.perm), P(self.offsets),
            P(self.packed[k]), P(self.h), self.stream), "gate_up_gather")

    def down_scatter(self, k):
        P, w = self.P, self.w
        if w.P:
            self._ok(self.lib.readme_moe_down_permanent_scatter(
                self.dt, w.T, w.d, w.E, w.I, w.P, P(self.h), P(self.perm), P(self.offsets),
                P(self.packed[k]), P(self.y), self.stream), "down_permanent_scatter")
            return
        self._ok(self.lib.readme_moe_down_scatter(
            self.dt, w.T, w.d, w.E, w.I, P(self.h), P(self.perm), P(self.offsets),
            P(self.packed[k]), P(self.y), self.stream), "down_scatter")

    def calls(self, k, fused=True):
        """(name, call) of one step, in path order; k picks the weight copy.
        fused: the row gather and the ungroup ride in the two GEMMs."""
        if self.w.layers > 1:
            stack = (lambda: self.offload_stack(k)) if self.ex else (lambda: self.stack(k))
            return [("route", self.route), ("group", lambda: self.group_resid(k)),
                    ("stack", stack), ("ungroup", self.ungroup_resid)]
        if self.w.K > 1:
            return [("route", self.route), ("topk", self.topk), ("group", self.group_pairs),
                    ("gate_up", lambda: self.gate_up_pairs(k)),
                    ("down", lambda: self.down_pairs(k)), ("combine", self.combine)]
        if fused:
            return [("route", self.route), ("group", self.group_only),
                    ("gate_up", lambda: self.gate_up_gather(k)),
                    ("down", lambda: self.down_scatter(k))]
        return [("route", self.route), ("group", self.group),
                ("gate_up", lambda: self.gate_up(k)), ("down", lambda: self.down(k)),
                ("ungroup", self.ungroup)]


# HBM traffic of the dominant kernel, per launch, from two rocprofv3 --pmc runs of
# this script (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each scaled by what
# the same counter reads for a plain 1 GiB device copy in the same run (--copy-probe:
# FETCH_SIZE reads about 524,308 KiB for it, so reads scale by about 1.99992; WRITE_SIZE
# reads exactly 1 GiB, factor 1).  Valid only for the sources the counters were taken
# with: each entry carries their sha256 and is dropped (traffic null) once any of
# them changes.
_GEMM_SOURCES = ["csrc/gemm_kernels.hpp", "csrc/gemm_mix.hpp", "csrc/gemm.hip",
                 "csrc/gemm_mix_gate_up.hip", "csrc/common.hpp", "csrc/internal.hpp",
                 "csrc/pack.hip", "workloads.py"]
_STACK_SOURCES = ["csrc/gemm_kernels.hpp", "csrc/gemm.hip", "csrc/gemm_bf16_gate_up.hip",
                  "csrc/gemm_bf16_resid.hip", "csrc/norm.hip", "csrc/abi.hip",
                  "csrc/common.hpp", "csrc/internal.hpp", "csrc/pack.hip", "workloads.py"]
TRAFFIC = {
    # workload: (sources, their sha256, read bytes, written bytes) per launch of the
    # dominant call: the gate/up GEMM (profiles/traffic_gate_up_wide_requests.md,
    # profiles/traffic_gate_up_prefill_skew16.md), or the whole 32-layer stack
    # (profiles/traffic_stack_llama7b_decode32.md)
    "wide_requests": (_GEMM_SOURCES,
                      "f2e5982ee17904e80e59c9f86a5a9dcabc2500a967656b365c81d094c306a252",
                      2255728392, 58720256),
    "prefill_skew16": (_GEMM_SOURCES,
                       "f2e5982ee17904e80e59c9f86a5a9dcabc2500a967656b365c81d094c306a252",
                       609159683, 23068672),
    "llama7b_decode32": (_STACK_SOURCES,
                         "600e4d122b11f65a2481f6be9870ec15ad14c9dfec5c1e1f0542ef625b3bea90",
                         7873977716, 56098816),
}


def traffic_bytes(workload: str):
    entry = TRAFFIC.get(workload)
    if entry is None:
        return None
    import hashlib
    sources, sha, rd, wr = entry
    root = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2410_19123_amd")
    h = hashlib.sha256()
    for rel in sources:
        with open(os.path.join(root, rel), "rb") as f:
            h.update(f.read())
    if h.hexdigest() != sha:
        return None
    return rd + wr


def algorithmic(w: wl.Workload, counts: np.ndarray, fused: bool = False) -> dict:
    """Algorithmic bytes and flops per launch of each kernel (unpadded I,
    weights of active experts only, each byte counted once)."""
    s = w.elem_bytes
    T, d, E, I = w.T, w.d, w.E, w.I
    active = int((counts > 0).sum())
    n = int(counts.sum())
    if w.layers > 1:
        L = w.layers
        per_layer_w = active * 3 * I * d * s
        return {
            "route": dict(bytes=T * d * s + E * d * s + 4 * T, flops=2.0 * T * d * E),
            "group": dict(bytes=12 * T + 8 * E + 2 * n * d * 4, flops=0.0),
            # per layer: weights once, fp32 residual read twice and written once,
            # bf16 normalised rows and h written and read once each
            "stack": dict(bytes=L * (per_layer_w + 3 * n * d * 4 + 2 * n * (d + I) * 2),
                          flops=6.0 * n * d * I * L),
            "ungroup": dict(bytes=2 * T * d * 4 + 4 * T, flops=0.0),
        }
    P = w.P  # permanent expert: P more neurons for every routed token
    # Top-K: n counts (token, slot) pairs; each pair's activation row is read
    # and its output row written once, the combine reads K rows per token.
    extra = {}
    if w.K > 1:
        extra = {"topk": dict(bytes=T * E * 4 + 8 * T * w.K, flops=0.0),
                 "combine": dict(bytes=n * d * s + T * d * s + 4 * n, flops=2.0 * n * d)}
    return {**extra,
        "route": dict(bytes=T * d * s + E * d * s + 4 * T, flops=2.0 * T * d * E),
        "group": dict(bytes=4 * T + 8 * T + 8 * E + (0 if fused else 2 * n * d * s), flops=0.0),
        "gate_up": dict(bytes=(active * I + P) * 2 * d * s + n * d * s + n * (I + P) * s,
                        flops=4.0 * n * d * (I + P)),
        "down": dict(bytes=(active * I + P) * d * s + n * (I + P) * s + n * d * s,
                     flops=2.0 * n * d * (I + P)),
        "ungroup": dict(bytes=2 * T * d * s + 4 * T, flops=0.0),
    }


def cpu_model() -> str:
    """The host CPU's model name, as /proc/cpuinfo gives it."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w: wl.Workload, target_s: float) -> dict:
    """The oracle as it stands on this host: the full path (route, group,
    gather, fp64 expert FFN, ungroup) on the first S tokens, repeated until
    about target_s seconds of CPU work have been timed."""
    from oracle import oracle

    x_all = wl.make_x(w)
    wr, b = wl.make_router(w)
    wg, wu, wd = wl.make_experts(w)
    perm_expert = wl.make_permanent(w) if w.P else None
    if w.router:
        ids_all = None
    elif w.batching:
        ids_all = wl.make_pool(w)[0]   # the waiting requests' experts
    else:
        ids_all = wl.make_request_ids(w)

    def run(S):
        ids = None if ids_all is None else ids_all[:S]
        t0 = time.perf_counter()
        if w.K > 1:
            oracle.full_path_topk(x_all[:S], wr, b, wg, wu, wd, K=w.K)
        else:
            oracle.full_path(x_all[:S], wr, b, wg, wu, wd, ids=ids, permanent=perm_expert)
        return time.perf_counter() - t0

    S = min(w.T, 16)
    dt = run(S)
    S = int(min(w.T, max(16, S * target_s / max(dt, 1e-6))))
    reps, total = 0, 0.0
    while reps == 0 or total < target_s:
        total += run(S)
        reps += 1
    return {"value": reps * S / total, "unit": "tokens/s", "cores": oracle.threads(),
            "cpu": cpu_model(), "kind": "oracle",
            "sample": f"first {S} of {w.T} tokens of the {w.name} workload, full path "
                      f"(route, {'top-%d, ' % w.K if w.K > 1 else ''}group, gather, fp64 expert FFN"
                      f"{' + permanent expert' if w.P else ''}, "
                      f"{'combine' if w.K > 1 else 'ungroup'}), {reps} pass(es), "
                      f"{total:.1f} s"}


def roofline(w: wl.Workload, wk: dict, dom_all: np.ndarray, dom: str) -> dict:
    """Roofline object of the dominant kernel from its launch durations (us):
    algorithmic bytes or flops over the mean launch, against HBM or MFMA."""
    dom_us = float(dom_all.mean())
    t = dom_us * 1e-6
    t_hbm = wk["bytes"] / (HBM_GBS * 1e9)
    pk = MFMA_F32_TFLOPS if w.dtype == "f32" else MFMA_BF16_TFLOPS
    t_mfma = wk["flops"] / (pk * 1e12)
    if t_hbm >= t_mfma:
        ach = wk["bytes"] / t / 1e9
        roof = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_GBS, "unit": "GB/s",
                "frac": round(ach / HBM_GBS, 4), "traffic": None}
    else:
        ach = wk["flops"] / t / 1e12
        roof = {"bound": "mfma", "achieved": round(ach, 1), "peak": pk, "unit": "TFLOP/s",
                "frac": round(ach / pk, 4), "traffic": None}
    roof["launch_us"] = round(dom_us, 2)
    roof["launch_us_p10_p50_p90"] = [round(float(v), 2)
                                     for v in np.percentile(dom_all, [10, 50, 90])]
    roof["algorithmic_bytes"] = int(wk["bytes"])
    roof["algorithmic_flops"] = wk["flops"]
    return roof


def run_workload(w: wl.Workload, K: int, W: int, fused: bool = True, copies: int = 0,
                 sample_every: int = 8, breakdown: int = 20) -> dict:
    """Times K steps of workload w after W warmup steps (inputs resident in
    HBM, weights rotated over >= 1 GiB of packed copies).  Inside the timed
    region only the dominant kernel is bracketed by HIP events, on every
    sample_every-th step; a separate pass of `breakdown` steps then times
    every call.  Returns the measurements and the path."""
    import torch

    packed_bytes = 3 * (w.E + w.P // w.I) * (-(-w.I // 64) * 64) * w.d * w.elem_bytes
    copies = copies or max(4, -(-(1 << 30) // packed_bytes))
    path = Path(w, copies)
    ncopy = len(path.packed)
    names = [n for n, _ in path.calls(0, fused)]
    ev = {n: [] for n in names}
    dom = "stack" if w.layers > 1 else "gate_up"
    ev_dom = []

    def step(i, mode):
        """mode None: no events; "dom": an event pair around the dominant
        kernel only (the timed region); "all": an event before every call
        (the per-call breakdown pass)."""
        k = i % ncopy
        marks = []
        for n, fn in path.calls(k, fused):
            if mode == "all" or (mode == "dom" and n == dom):
                a = torch.cuda.Event(enable_timing=True)
                a.record()
                marks.append((n, a))
            fn()
            if mode == "dom" and n == dom:
                z = torch.cuda.Event(enable_timing=True)
                z.record()
                ev_dom.append((marks[-1][1], z))
        if mode == "all":
            z = torch.cuda.Event(enable_timing=True)
            z.record()
            for j, (n, a) in enumerate(marks):
                nxt = marks[j + 1][1] if j + 1 < len(marks) else z
                ev[n].append((a, nxt))

    for i in range(W):
        step(i, None)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    # The dominant kernel's event pair goes on every sample_every-th step of
    # the timed region: an event pair costs a few us of the step, so sampling
    # keeps the step time honest while the launch average still spans the
    # whole region.
    for i in range(K):
        step(W + i, "dom" if i % sample_every == 0 else None)
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = start.elapsed_time(stop)
    dom_all = np.array([1e3 * a.elapsed_time(b) for a, b in ev_dom])
    for i in range(min(K, breakdown)):
        step(W + K + i, "all")
    torch.cuda.synchronize()

    counts = path.counts.cpu().numpy()
    work = algorithmic(w, counts, fused)
    offload = None
    if path.ex:
        hits, misses, nbytes = path.ex.stats()
        steps_run = W + K + min(K, breakdown)
        ms = gpu_ms / K
        offload = {"slots": w.offload_slots, "policy": w.policy,
                   "hit_ratio": round(hits / max(hits + misses, 1), 4),
                   "gb_copied_per_step": round(nbytes / steps_run / 1e9, 3),
                   "h2d_gb_s": round(nbytes / steps_run / (ms * 1e-3) / 1e9, 1)}
    if w.batching:
        # the batches differ from step to step: average their work
        per = [algorithmic(w, np.bincount(b, minlength=w.E), fused) for b in path.sched]
        work = {n: {q: float(np.mean([pw[n][q] for pw in per])) for q in ("bytes", "flops")}
                for n in per[0]}
        counts = np.bincount(path.sched.reshape(-1), minlength=w.E) // path.sched.shape[0]
    kern_us = {n: (1e3 * float(np.mean([a.elapsed_time(b) for a, b in ev[n]])) if ev[n] else None)
               for n in names}
    return dict(path=path, ncopy=ncopy, gpu_ms=gpu_ms, wall=wall, dom=dom, dom_all=dom_all,
                counts=counts, work=work, kern_us=kern_us, offload=offload)


def library_gemm(w: wl.Workload, counts: np.ndarray, reps: int = 10) -> dict:
    """The workload's expert GEMMs run one expert at a time through torch's
    library GEMM (hipBLASLt on ROCm), bf16 in, fp32 accumulation: gate and
    up as one [T_e, d] x [d, 2I] product, down as [T_e, I] x [I, d].
    Weights rotate over two copies; timed with events around all experts.
    Context only: the SiLU*mul, the row gather and the scatter are left out,
    so it does less work than the grouped kernels."""
    import torch
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(0)
    rows = [int(c) for c in counts if c > 0]
    xs = [torch.randn(r, w.d, device=dev, dtype=torch.bfloat16, generator=g) for r in rows]
    hs = [torch.randn(r, w.I, device=dev, dtype=torch.bfloat16, generator=g) for r in rows]
    wgu = [[torch.randn(2 * w.I, w.d, device=dev, dtype=torch.bfloat16, generator=g)
            for _ in rows] for _ in range(2)]
    wdn = [[torch.randn(w.d, w.I, device=dev, dtype=torch.bfloat16, generator=g)
            for _ in rows] for _ in range(2)]
    F = torch.nn.functional.linear

    def timed(fn):
        for k in range(3):
            fn(k)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for k in range(reps):
            fn(k)
        b.record()
        torch.cuda.synchronize()
        return 1e3 * a.elapsed_time(b) / reps

    gu = timed(lambda k: [F(x, wt) for x, wt in zip(xs, wgu[k % 2])])
    dn = timed(lambda k: [F(h, wt) for h, wt in zip(hs, wdn[k % 2])])
    n = sum(rows)
    fl_gu, fl_dn = 4.0 * n * w.d * w.I, 2.0 * n * w.d * w.I
    out = {"gate_up_us": round(gu, 2), "down_us": round(dn, 2),
           "gate_up_tflops": round(fl_gu / gu / 1e6, 1), "down_tflops": round(fl_dn / dn / 1e6, 1),
           "kind": "torch.nn.functional.linear per expert (hipBLASLt), bf16"}
    del xs, hs, wgu, wdn
    torch.cuda.empty_cache()
    return out


def side_line(name: str, K: int, W: int) -> dict:
    """One half of the metric measured beside the main line: the decode
    stack's HBM fraction or the prefill gate/up's MFMA fraction."""
    import torch
    w = wl.WORKLOADS[name]
    r = run_workload(w, K, W, sample_every=1, breakdown=0)
    ms = r["gpu_ms"] / K
    value = w.T * K / (r["gpu_ms"] / 1e3) * max(w.layers, 1)
    roof = roofline(w, r["work"][r["dom"]], r["dom_all"], r["dom"])
    roof["traffic"] = traffic_bytes(name)
    roof["kernel"] = ("readme_moe_ffn_stack (all layers)" if w.layers > 1
                      else "k_grouped_gemm (gate/up + SiLU*mul, rows gathered through perm)")
    out = {"workload": name, "T": w.T, "d": w.d, "E": w.E, "I": w.I, "layers": w.layers,
           "steps": K, "ms_per_step": round(ms, 4),
           "tokens_per_s_per_layer": round(value, 1),
           "tokens_per_expert": r["counts"].tolist(), "roofline": roof}
    del r
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def router_flops(shape: wl.RouterShape, lengths) -> float:
    """Algorithmic FLOP of one router call: the projections (q, k, v, o:
    8 D^2 per token), the SwiGLU MLP (6 D F), the gate (2 D E) and causal
    attention (4 * 128 * prefix length per token and head, D / 128 heads)."""
    D, F, E = shape.D, shape.F, shape.E
    T = int(np.sum(lengths))
    prefix = sum(n * (n + 1) // 2 for n in lengths)
    return T * (8.0 * D * D + 6.0 * D * F + 2.0 * D * E) + 4.0 * 128 * prefix * (D // 128)


ROUTER_MIXES = {
    # name: request lengths (8192 tokens each)
    "requests_256x32": [32] * 256,     # the request batch's requests
    "prompts_8x1024": [1024] * 8,      # long prompts: attention over 1024-token prefixes
}


def router_line(K: int, W: int, mix: str = "requests_256x32") -> dict:
    """The pre-gating router G (Sec. 2.3, Table 1: one causal transformer
    block of width 512, four heads, SwiGLU MLP 512, vocabulary 32000, then
    the gate to 8 experts) over 8192 tokens in requests of the given mix
    (by default the request batch's 256 x 32), random-init weights.  One
    call = embedding, block, gate, all on the GPU; HIP events on the launch
    stream around K calls."""
    import torch
    from paper_2410_19123_amd import _lib as L
    shape = wl.ROUTER_TABLE1
    lengths = ROUTER_MIXES[mix]
    wts = wl.make_router_tf(shape, 0)
    tokens, ro = wl.make_router_requests(lengths, shape.V, 0)
    dev = torch.device("cuda:0")
    dw = {n: L.to_device(wts[n], dev) for n in ("emb", "wq", "wk", "wv", "wo", "w1", "w3", "w2",
                                                "w_router")}
    packed = L.readme_router_tf_pack(dw["wq"], dw["wk"], dw["wv"], dw["wo"], dw["w1"],
                                     dw["w3"], dw["w2"])
    tk, rof = L.to_device(tokens, dev), L.to_device(ro, dev)
    T = len(tokens)
    ids = torch.empty(T, dtype=torch.int32, device=dev)
    logits = torch.empty(T, shape.E, dtype=torch.float32, device=dev)
    ws = torch.empty(L.readme_router_tf_workspace_bytes(T, shape.D, shape.F), dtype=torch.uint8,
                     device=dev)

    def call():
        L.readme_router_tf(tk, rof, dw["emb"], packed, shape.F, dw["w_router"], None, 1e-5,
                           expert_ids=ids, logits=logits, workspace=ws)

    for _ in range(W):
        call()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(K):
        call()
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) * 1e3 / K
    fl = router_flops(shape, lengths)
    counts = np.bincount(L.from_device(ids), minlength=shape.E)
    out = {"workload": f"router_tf_table1_{mix}", "T": T, "D": shape.D, "F": shape.F,
           "V": shape.V, "E": shape.E, "heads": shape.D // 128, "requests": len(lengths),
           "steps": K, "us_per_call": round(us, 2), "tokens_per_s": round(T / (us * 1e-6), 1),
           "gflop_per_call": round(fl / 1e9, 3), "tflops": round(fl / (us * 1e-6) / 1e12, 2),
           "tokens_per_expert": counts.tolist()}
    del dw, packed, ws
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: measures one GPU only (asked for --gpus {args.gpus}); "
              "sharding across GPUs is described in the design notes, not measured.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)

    if args.router_only:
        print(json.dumps({"router": router_line(args.steps, args.warmup),
                          "router_long": router_line(args.steps, args.warmup,
                                                     "prompts_8x1024")}), flush=True)
        return

    w = wl.WORKLOADS[args.workload]
    if (w.P or w.K > 1) and args.unfused:
        print("bench.py: the permanent-expert and top-K workloads run the fused path only",
              file=sys.stderr)
        sys.exit(2)
    if args.gemm_tile:
        from paper_2410_19123_amd import _lib
        _lib.load()
        _lib.readme_set_gemm_tile(args.gemm_tile)
    K, W = args.steps, args.warmup
    fused = not args.unfused
    r = run_workload(w, K, W, fused, args.weight_copies)
    gpu_ms, dom, counts, work = r["gpu_ms"], r["dom"], r["counts"], r["work"]
    ms_per_step = gpu_ms / K
    layers = w.layers

    value = w.T * K / (gpu_ms / 1e3)  # tokens/s through one step
    if layers > 1:
        value = value * layers       # per MoE layer
    rows = w.T if w.batching else int(counts.sum())  # routed rows (pairs for top-K)
    ffn_flops = 6.0 * rows * w.d * (w.I + w.P) * layers

    roof = None
    if r["dom_all"].size:
        roof = roofline(w, work[dom], r["dom_all"], dom)
        roof["kernel"] = ("readme_moe_ffn_stack (all layers)" if layers > 1
                          else "k_grouped_gemm (gate/up + SiLU*mul"
                          + (", permanent expert as extra row groups" if w.P else "")
                          + (f", top-{w.K} (token, slot) pairs" if w.K > 1 else "")
                          + (", rows gathered through perm)" if fused else ")"))
        if not args.gemm_tile and (dom == "stack" or fused):
            roof["traffic"] = traffic_bytes(w.name)
    kern_us = r["kern_us"]

    out = {
        "metric": "expert-FFN tokens/sec per MoE layer",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.dtype == "f32" else "bf16",
        "data": "synthetic (seeded N(0,1) tokens, N(0,0.02) weights)",
        "config": {"workload": w.name, "T": w.T, "d": w.d, "E": w.E, "I": w.I, "P": w.P, "K": w.K,
                   "gemm_tile": args.gemm_tile,
                   "row_moves": "separate" if args.unfused or layers > 1 else "fused into GEMMs",
                   "layers": layers, "weight_copies_rotated": r["ncopy"],
                   "tokens_per_expert": counts.tolist(),
                   **({"batching": w.batching, "pool": w.pool,
                       "unique_experts_per_batch": round(float(np.mean(
                           [len(set(b.tolist())) for b in r["path"].sched])), 2)}
                      if w.batching else {}),
                   **({"offload": r["offload"]} if r["offload"] else {})},
        "ffn_tflops": round(ffn_flops / (ms_per_step * 1e-3) / 1e12, 2),
        # event pair before each call, from a separate 20-step pass after the
        # timed region (events between every call add their own gaps)
        "kernels_us": {k: (round(v, 2) if v is not None else None) for k, v in kern_us.items()},
        # algorithmic bytes of each call over its breakdown time (HBM peak 8000 GB/s)
        "kernels_gbs": {k: round(work[k]["bytes"] / (v * 1e-6) / 1e9, 1)
                        for k, v in kern_us.items() if v and k in work},
        "host_wall_ms_per_step": round(1e3 * r["wall"] / K, 4),
        "roofline": roof,
    }
    if args.copy_probe:
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda:0")
        bb = torch.empty_like(a)
        for _ in range(3):
            bb.copy_(a)
        torch.cuda.synchronize()
        out["copy_probe_bytes"] = 1 << 30
        del a, bb
    del r
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    # The metric's two halves beside the main line: % of HBM for the decode
    # step (the 32-layer stack), % of the MFMA peak for the prefill gate/up.
    if not args.no_side and args.workload not in ("llama7b_decode32", "prefill_skew16"):
        out["decode"] = side_line("llama7b_decode32", args.side_steps, 3)
        out["prefill"] = side_line("prefill_skew16", args.side_steps, 3)
        out["router"] = router_line(args.side_steps, 3)
        out["router_long"] = router_line(args.side_steps, 3, "prompts_8x1024")
    if args.library_gemm and w.dtype == "bf16" and w.layers == 1 and w.K == 1 and not w.P:
        out["library_gemm"] = library_gemm(w, counts)
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
