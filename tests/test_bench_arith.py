"""The algorithmic work bench.py divides by its measured times, pinned to
figures derived by hand from the shapes (unpadded intermediate, weights of
active experts only, each byte once): the SwiGLU FFN does 4·T·d·I flops in
gate/up and 2·T·d·I in down, and streams 2·E·I·d and E·I·d weight elements."""
import numpy as np
import pytest

import bench
from paper_2410_19123_amd import workloads as wl


def _all_active(w):
    c = np.full(w.E, w.T // w.E, np.int64)
    c[: w.T - int(c.sum())] += 1
    return c


def test_default_layer_gate_up_bytes_and_flops():
    w = wl.WORKLOADS["llama7b_layer"]
    a = bench.algorithmic(w, _all_active(w), fused=True)
    # 8 experts x 2 x 1376 x 4096 bf16 weights + x read + h written
    assert a["gate_up"]["bytes"] == 8 * 2 * 1376 * 4096 * 2 + 2048 * 4096 * 2 + 2048 * 1376 * 2
    assert a["gate_up"]["bytes"] == 202_768_384
    assert a["gate_up"]["flops"] == 4 * 2048 * 4096 * 1376          # 46.17 GFLOP
    assert a["down"]["flops"] == 2 * 2048 * 4096 * 1376             # 23.09 GFLOP
    assert a["down"]["bytes"] == 8 * 1376 * 4096 * 2 + 2048 * 1376 * 2 + 2048 * 4096 * 2
    # the fused layer moves no rows through the grouping
    assert a["group"]["bytes"] == 12 * 2048 + 8 * 8


@pytest.mark.parametrize("name,gflops,weight_mb", [
    ("prefill_skew16", 184.7, 180.4),   # 4 T d I, 2 E I d elements
    ("wide_requests", 962.1, 939.5),
])
def test_prefill_and_request_batch_gate_up(name, gflops, weight_mb):
    w = wl.WORKLOADS[name]
    a = bench.algorithmic(w, _all_active(w), fused=True)
    assert a["gate_up"]["flops"] / 1e9 == pytest.approx(gflops, abs=0.05)
    weights = 2 * w.E * w.I * w.d * 2
    assert weights / 1e6 == pytest.approx(weight_mb, abs=0.05)
    assert a["gate_up"]["bytes"] == weights + w.T * w.d * 2 + w.T * w.I * 2


def test_roofline_bounds():
    """The default layer is HBM-bound, the large batches MFMA-bound."""
    def bound(name):
        w = wl.WORKLOADS[name]
        g = bench.algorithmic(w, _all_active(w), fused=True)["gate_up"]
        return "hbm" if g["bytes"] / (bench.HBM_GBS * 1e9) >= g["flops"] / (
            bench.MFMA_BF16_TFLOPS * 1e12) else "mfma"
    assert bound("llama7b_layer") == "hbm"
    assert bound("prefill_skew16") == "mfma"
    assert bound("wide_requests") == "mfma"


def test_decode_stack_counts_active_experts_only():
    w = wl.WORKLOADS["llama7b_decode32"]
    counts = np.array([30, 14, 7, 6, 4, 0, 2, 1])
    a = bench.algorithmic(w, counts)
    per_layer_weights = 7 * 3 * 1376 * 4096 * 2                   # expert 5 is empty
    n, d, I = 64, 4096, 1376
    assert a["stack"]["bytes"] == 32 * (per_layer_weights + 3 * n * d * 4 + 2 * n * (d + I) * 2)
    assert a["stack"]["flops"] == 6.0 * n * d * I * 32


def test_more_than_one_gpu_is_refused():
    """bench.py measures one GPU; --gpus N > 1 exits with a message before
    touching a device."""
    import subprocess
    import sys
    from pathlib import Path
    r = subprocess.run([sys.executable, str(Path(bench.__file__)), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_traffic_entries_follow_their_sources(tmp_path, monkeypatch):
    """A calibrated traffic entry gives its read + written bytes only for
    the exact sources it was taken with, and null as soon as any of them
    differs (a kernel changed since the counters were read)."""
    import os
    import shutil
    for name, (sources, sha, rd, wr) in bench.TRAFFIC.items():
        assert bench.traffic_bytes(name) in (None, rd + wr), name
        assert rd > 0 and wr > 0 and len(sha) == 64
    # a copy of the package with one source byte changed
    pkg = os.path.join(os.path.dirname(os.path.abspath(bench.__file__)), "paper_2410_19123_amd")
    fake = tmp_path / "paper_2410_19123_amd"
    for rel in set(r for s, _, _, _ in bench.TRAFFIC.values() for r in s):
        dst = fake / rel
        dst.parent.mkdir(parents=True, exist_ok=True)
        shutil.copyfile(os.path.join(pkg, rel), dst)
    with open(fake / "csrc" / "gemm_kernels.hpp", "ab") as f:
        f.write(b"\n")
    monkeypatch.setattr(bench, "__file__", str(tmp_path / "bench.py"))
    for name in bench.TRAFFIC:
        assert bench.traffic_bytes(name) is None, name
    assert bench.traffic_bytes("tiny_f32") is None   # no entry


def test_router_flops():
    """The router's algorithmic work per call, from the shapes by hand: the
    four D x D projections and the three MLP matrices (2 flops per weight
    per token), the gate, and causal attention's two products (2 x 128
    multiply-adds per (query, key) pair and head, each key up to the query
    inside its request)."""
    shape = wl.ROUTER_TABLE1          # D = F = 512, E = 8, four heads
    per_token = 2 * (4 * 512 * 512 + 3 * 512 * 512 + 8 * 512)
    # one request of 3 tokens: 1 + 2 + 3 = 6 (query, key) pairs
    assert bench.router_flops(shape, [3]) == 3 * per_token + 6 * 4 * 128 * 4
    # empty requests add nothing; pairs never cross requests
    assert bench.router_flops(shape, [3, 0, 2]) == 5 * per_token + (6 + 3) * 4 * 128 * 4
    # the request batch of the benchmark: 256 requests of 32 (528 pairs each)
    f = bench.router_flops(shape, [32] * 256)
    assert f == 8192 * per_token + 256 * 528 * 4 * 128 * 4
    assert f / 1e9 == pytest.approx(30.41, abs=0.01)
