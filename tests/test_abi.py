"""The C-ABI library loads on the CPU, exports every function readme.h
declares, and rejects bad arguments on the host before any launch (no GPU
needed: these calls never reach the HIP runtime)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "readme.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(readme_[a-z0-9_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from paper_2410_19123_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        pytest.skip("libreadme.so not built")
    return _lib.load()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n


def test_binding_covers_header():
    from paper_2410_19123_amd import _lib
    assert set(_declared()) == set(_lib.SIGNATURES)


def test_status_strings_and_version(lib):
    assert lib.readme_abi_version() == 1
    assert lib.readme_status_string(0) == b"ok"
    assert lib.readme_status_string(3) == b"buffer smaller than required"


def test_sizes(lib):
    assert lib.readme_padded_intermediate(1376) == 1408
    assert lib.readme_padded_intermediate(688) == 704
    assert lib.readme_padded_intermediate(512) == 512
    assert lib.readme_packed_experts_bytes(1, 8, 4096, 1376) == 8 * 3 * 1408 * 4096 * 2
    assert lib.readme_packed_experts_bytes(0, 4, 512, 512) == 4 * 3 * 512 * 512 * 4
    assert lib.readme_packed_experts_bytes(1, 0, 4096, 1376) == 0
    assert lib.readme_moe_ffn_workspace_bytes(1, 2048, 1376) == 2048 * 1408 * 2
    assert lib.readme_moe_ffn_stack_workspace_bytes(64, 4096, 1376) == 64 * 4096 * 2 + 64 * 1408 * 2


FAKE = ctypes.c_void_p(4096)   # never dereferenced: every call below fails validation


def test_route_argument_errors(lib):
    r = lib.readme_route
    assert r(7, 4, 64, 2, FAKE, FAKE, None, FAKE, None, None) == 1          # bad dtype
    assert r(1, -1, 64, 2, FAKE, FAKE, None, FAKE, None, None) == 1         # T < 0
    assert r(1, 4, 64, 0, FAKE, FAKE, None, FAKE, None, None) == 2          # E < 1
    assert r(1, 4, 64, 257, FAKE, FAKE, None, FAKE, None, None) == 2        # E > 256
    assert r(1, 4, 60, 2, FAKE, FAKE, None, FAKE, None, None) == 2          # d % 8
    assert r(0, 4, 62, 2, FAKE, FAKE, None, FAKE, None, None) == 2          # d % 4 (fp32)
    assert r(1, 4, 64, 2, None, FAKE, None, FAKE, None, None) == 1          # NULL x
    assert r(1, 4, 64, 2, ctypes.c_void_p(4100), FAKE, None, FAKE, None, None) == 1  # misaligned
    assert r(1, 0, 64, 2, None, None, None, None, None, None) == 0          # T = 0: no-op


def test_group_argument_errors(lib):
    g = lib.readme_group_by_expert
    assert g(-1, 4, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, None, None, None) == 1
    assert g(8, 0, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, None, None, None) == 2
    assert g(8, 4, None, FAKE, FAKE, FAKE, FAKE, 1, 64, None, None, None) == 1
    assert g(8, 4, FAKE, FAKE, FAKE, FAKE, None, 1, 64, None, None, None) == 1
    assert g(8, 4, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 64, FAKE, None, None) == 1   # half a gather
    assert g(8, 4, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 4, FAKE, FAKE, None) == 2    # 8-byte rows


def test_ffn_argument_errors(lib):
    f = lib.readme_moe_ffn
    assert f(1, 16, 4096, 8, 1376, FAKE, FAKE, FAKE, FAKE, FAKE, 10, None) == 3  # workspace
    assert f(1, 16, 4000, 8, 1376, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 2
    assert f(1, 16, 4096, 8, 0, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 1
    assert f(1, 16, 4096, 300, 16, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 2
    assert f(1, 16, 4096, 8, 16, None, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == 1
    assert f(1, 0, 4096, 8, 16, None, None, None, None, None, 0, None) == 0
    p = lib.readme_pack_experts
    assert p(1, 8, 4096, 1376, FAKE, FAKE, FAKE, FAKE, 100, None) == 3
    assert p(1, 8, 4096, 1376, FAKE, None, FAKE, FAKE, 1 << 40, None) == 1
    u = lib.readme_ungroup
    assert u(1, 8, 4, FAKE, FAKE, FAKE, None) == 2
    assert u(1, 8, 64, FAKE, None, FAKE, None) == 1
    s = lib.readme_moe_ffn_stack
    arr = (ctypes.c_void_p * 1)(4096)
    assert s(64, 4096, 8, 1376, 1, arr, FAKE, FAKE, ctypes.c_float(-1.0), FAKE, 1 << 40,
             None) == 1
    assert s(64, 4096, 8, 1376, 1, arr, FAKE, FAKE, ctypes.c_float(1e-5), FAKE, 10, None) == 3
    assert s(64, 4096, 8, 1376, -1, arr, FAKE, FAKE, ctypes.c_float(1e-5), FAKE, 1 << 40,
             None) == 1


def test_permanent_sizes_and_errors(lib):
    # S = P / I slices of one expert's packed shape after the E experts.
    assert lib.readme_packed_experts_permanent_bytes(1, 8, 4096, 1376, 1376) == \
        9 * 3 * 1408 * 4096 * 2
    assert lib.readme_packed_experts_permanent_bytes(1, 8, 4096, 1376, 0) == \
        lib.readme_packed_experts_bytes(1, 8, 4096, 1376)
    assert lib.readme_packed_experts_permanent_bytes(1, 8, 4096, 1376, 1000) == 0  # P % I
    assert lib.readme_packed_experts_permanent_bytes(1, 8, 4096, 16, 17 * 16) == 0  # > 16 slices
    assert lib.readme_moe_ffn_permanent_workspace_bytes(1, 2048, 1376, 2752) == \
        2048 * 3 * 1408 * 2
    f = lib.readme_moe_ffn_permanent_fused
    big = 1 << 40
    assert f(1, 16, 4096, 8, 1376, 1376, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 10, None) == 3
    assert f(1, 16, 4096, 8, 1376, 1000, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, big, None) == 2
    assert f(1, 16, 4096, 8, 1376, -1376, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, big, None) == 1
    assert f(1, 16, 4096, 8, 1376, 1376, FAKE, None, FAKE, FAKE, FAKE, FAKE, big, None) == 1
    assert f(1, 0, 4096, 8, 1376, 1376, None, None, None, None, None, None, 0, None) == 0
    g = lib.readme_moe_ffn_permanent
    assert g(1, 16, 4096, 8, 1376, 1376, FAKE, FAKE, FAKE, FAKE, FAKE, 10, None) == 3
    assert g(1, 16, 4000, 8, 1376, 1376, FAKE, FAKE, FAKE, FAKE, FAKE, big, None) == 2
    p = lib.readme_pack_experts_permanent
    assert p(1, 8, 4096, 1376, 1376, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 100, None) == 3
    assert p(1, 8, 4096, 1376, 1376, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, big, None) == 1
    assert p(1, 8, 4096, 1376, 1000, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, big, None) == 2


def test_topk_argument_errors(lib):
    t = lib.readme_topk
    assert t(16, 8, 0, FAKE, FAKE, FAKE, None) == 1        # K < 1
    assert t(16, 8, 9, FAKE, FAKE, FAKE, None) == 1        # K > E
    assert t(16, 300, 2, FAKE, FAKE, FAKE, None) == 2      # E > 256
    assert t(16, 8, 2, None, FAKE, FAKE, None) == 1
    assert t(0, 8, 2, None, None, None, None) == 0
    f = lib.readme_moe_ffn_topk
    big = 1 << 40
    assert f(1, 16, 4096, 8, 1376, 2, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 10, None) == 3
    assert f(1, 16, 4096, 8, 1376, 9, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, big, None) == 1
    assert f(1, 1 << 30, 4096, 8, 1376, 4, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, big, None) == 2
    assert lib.readme_moe_ffn_workspace_bytes(1, 2048 * 2, 1376) == 4096 * 1408 * 2
    c = lib.readme_combine_topk
    assert c(1, 16, 4, 2, FAKE, FAKE, FAKE, None) == 2     # 8-byte rows
    assert c(1, 16, 64, 0, FAKE, FAKE, FAKE, None) == 1
    assert c(1, 16, 64, 2, FAKE, None, FAKE, None) == 1


def test_stack_counts_argument_errors(lib):
    s = lib.readme_moe_ffn_stack_counts
    arr = (ctypes.c_void_p * 1)(4096)
    assert s(64, 4096, 8, 1376, 1, arr, FAKE, None, FAKE, ctypes.c_float(1e-5), FAKE, 1 << 40,
             None) == 1                                          # no counts
    neg = (ctypes.c_int32 * 8)(1, 2, -1, 0, 0, 0, 0, 0)
    assert s(64, 4096, 8, 1376, 1, arr, FAKE, neg, FAKE, ctypes.c_float(1e-5), FAKE, 1 << 40,
             None) == 1                                          # negative count


def test_streamed_buffers_checked_before_any_launch(lib):
    """Every streamed buffer's alignment is checked on the host before the
    first launch (no GPU here: a launch would report README_ERR_HIP)."""
    big = 1 << 40
    odd = ctypes.c_void_p(4104)     # 8-byte aligned only
    f = lib.readme_moe_ffn
    assert f(1, 16, 4096, 8, 1376, FAKE, FAKE, FAKE, FAKE, odd, big, None) == 1   # workspace
    assert f(1, 16, 4096, 8, 1376, FAKE, FAKE, FAKE, odd, FAKE, big, None) == 1   # y_grouped
    assert f(1, 16, 4096, 8, 1376, odd, FAKE, FAKE, FAKE, FAKE, big, None) == 1   # x_grouped
    assert f(1, 16, 4096, 8, 1376, FAKE, FAKE, odd, FAKE, FAKE, big, None) == 1   # packed
    gu = lib.readme_moe_gate_up
    assert gu(1, 16, 4096, 8, 1376, FAKE, FAKE, FAKE, odd, None) == 1              # h
    dn = lib.readme_moe_down
    assert dn(1, 16, 4096, 8, 1376, FAKE, FAKE, FAKE, odd, None) == 1              # y_grouped
    fu = lib.readme_moe_ffn_fused
    assert fu(1, 16, 4096, 8, 1376, odd, FAKE, FAKE, FAKE, FAKE, FAKE, big, None) == 1  # x
    assert fu(1, 16, 4096, 8, 1376, FAKE, FAKE, FAKE, FAKE, FAKE, odd, big, None) == 1  # workspace
    g = lib.readme_moe_gate_up_gather
    assert g(1, 16, 4096, 8, 1376, FAKE, FAKE, FAKE, FAKE, odd, None) == 1          # h
    sc = lib.readme_moe_down_scatter
    assert sc(1, 16, 4096, 8, 1376, FAKE, FAKE, FAKE, FAKE, odd, None) == 1         # y
    t = lib.readme_moe_ffn_topk
    assert t(1, 16, 4096, 8, 1376, 2, odd, FAKE, FAKE, FAKE, FAKE, FAKE, big, None) == 1


def test_router_tf_sizes_and_errors(lib):
    D, F = 512, 512
    assert lib.readme_router_tf_packed_bytes(D, F) == 4 * D * D * 2 + 3 * F * D * 2
    assert lib.readme_router_tf_packed_bytes(500, F) == 0          # heads of 128
    assert lib.readme_router_tf_packed_bytes(D, 0) == 0
    T = 100
    sizes = [T * D * 4, T * D * 2, T * 3 * D * 2, T * D * 2, T * D * 2, T * F * 2, T * D * 2,
             T * 4, 8]
    off = 0
    for region, n in enumerate(sizes):
        assert lib.readme_router_tf_workspace_offset(T, D, F, region) == off
        off += (n + 255) // 256 * 256
    assert lib.readme_router_tf_workspace_offset(T, D, F, len(sizes)) == off
    assert lib.readme_router_tf_workspace_bytes(T, D, F) == off
    assert lib.readme_router_tf_workspace_offset(T, D, F, len(sizes) + 1) == -1
    assert lib.readme_router_tf_workspace_offset(-1, D, F, 0) == -1
    assert lib.readme_router_tf_workspace_bytes(T, 384, 100) > 0   # F padded to 128
    r = lib.readme_router_tf
    eps = ctypes.c_float(1e-5)
    ws = 1 << 40
    args = lambda **k: [k.get("T", 64), k.get("R", 2), k.get("D", 512), k.get("F", 512),
                        k.get("E", 8), k.get("V", 32000), FAKE, FAKE, FAKE, FAKE, FAKE, None,
                        k.get("eps", eps), FAKE, None, k.get("ws", FAKE),
                        k.get("wsb", ws), None]
    assert r(*args(D=500)) == 2
    assert r(*args(D=16384 + 128)) == 2
    assert r(*args(E=0)) == 2
    assert r(*args(E=257)) == 2
    assert r(*args(R=0)) == 1
    assert r(*args(V=0)) == 1
    assert r(*args(eps=ctypes.c_float(-1.0))) == 1
    assert r(*args(wsb=10)) == 3
    assert r(*args(ws=ctypes.c_void_p(4100))) == 1
    assert r(*args(T=0, R=0)) == 0
    pk = lib.readme_router_tf_pack
    assert pk(512, 512, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 10, None) == 3
    assert pk(512, 512, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == 1
    assert pk(640, 0, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == 1
    at = lib.readme_attention_causal
    assert at(10, 2, 1, FAKE, FAKE, FAKE, FAKE, 200, FAKE, 256, None) == 1   # ld_in < 256
    assert at(10, 2, 1, FAKE, FAKE, FAKE, FAKE, 260, FAKE, 256, None) == 1   # ld_in % 8
    assert at(10, 2, 1, FAKE, ctypes.c_void_p(4104), FAKE, FAKE, 256, FAKE, 256, None) == 1
    assert at(10, 2, -1, FAKE, FAKE, FAKE, FAKE, 256, FAKE, 256, None) == 1  # R < 0
    assert at(0, 2, 0, None, None, None, None, 256, None, 256, None) == 0
    ro = lib.readme_rope
    assert ro(10, 2, FAKE, FAKE, 255, None) == 1
    assert ro(10, 2, FAKE, FAKE, 260, None) == 1                             # ld % 8
    assert ro(10, 2, FAKE, ctypes.c_void_p(4104), 256, None) == 1            # misaligned
    assert ro(0, 2, None, None, 256, None) == 0
    rp = lib.readme_request_positions
    assert rp(10, 0, FAKE, FAKE, None) == 1
    assert rp(0, 0, None, None, None) == 0


def test_tile_override_is_per_thread(lib):
    import threading
    assert lib.readme_set_gemm_tile(32) == 1
    assert lib.readme_set_gemm_tile(-1) == 1
    assert lib.readme_set_gemm_tile(5) == 0
    seen = []
    th = threading.Thread(target=lambda: seen.append(lib.readme_get_gemm_tile()))
    th.start()
    th.join()
    assert seen == [0]                       # another thread keeps the automatic choice
    assert lib.readme_get_gemm_tile() == 5
    assert lib.readme_set_gemm_tile(0) == 0
    assert lib.readme_get_gemm_tile() == 0


def test_noalloc_size_limit(lib):
    """The allocation-free FFN refuses an h larger than its fixed array
    (64 MiB) on the host, before touching the device."""
    f = lib.readme_moe_ffn_fused_noalloc
    # T * padded(I) * 2 bytes: 2^19 * 64 * 2 = 64 MiB fits (then the NULL x
    # is README_ERR_ARG); one more row does not.
    assert f(1, 1 << 19, 64, 2, 64, None, None, None, None, None, None) == 1
    assert f(1, (1 << 19) + 1, 64, 2, 64, None, None, None, None, None, None) == 2
    assert f(0, 1 << 18, 64, 2, 64, None, None, None, None, None, None) == 1   # fp32: fits
    assert f(0, (1 << 18) + 1, 64, 2, 64, None, None, None, None, None, None) == 2
    assert f(1, 0, 64, 2, 64, None, None, None, None, None, None) == 0        # T = 0
    assert f(1, 16, 4000, 2, 64, FAKE, FAKE, FAKE, FAKE, FAKE, None) == 2     # d % 64


def test_weighted_top1_argument_errors(lib):
    g = lib.readme_gate_weights
    assert g(-1, 8, FAKE, FAKE, FAKE, FAKE, None) == 1
    assert g(16, 0, FAKE, FAKE, FAKE, FAKE, None) == 2
    assert g(16, 8, None, FAKE, FAKE, FAKE, None) == 1
    assert g(0, 8, None, None, None, None, None) == 0
    u = lib.readme_ungroup_scaled
    assert u(1, 16, 4, FAKE, FAKE, FAKE, FAKE, None) == 2          # 8-byte rows
    assert u(1, 16, 64, FAKE, FAKE, None, FAKE, None) == 1         # no scale
    assert u(1, 16, 64, ctypes.c_void_p(4104), FAKE, FAKE, FAKE, None) == 1  # misaligned
    assert u(1, 0, 64, None, None, None, None, None) == 0


def test_binding_fails_loudly_without_the_library(tmp_path):
    """With libreadme.so absent the binding raises instead of falling back to
    any other implementation (run in a child so this process keeps its
    loaded library)."""
    import subprocess
    import sys
    code = (
        "from paper_2410_19123_amd import _lib\n"
        f"_lib.LIB_PATH = {str(tmp_path / 'libreadme.so')!r}\n"
        "try:\n"
        "    _lib.readme_padded_intermediate(100)\n"
        "except ImportError as e:\n"
        "    print('ImportError', e)\n"
        "else:\n"
        "    print('no error')\n")
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True,
                         text=True, timeout=120)
    assert out.stdout.startswith("ImportError"), out.stdout + out.stderr


def test_product_path_does_not_reach_the_oracle():
    """The package and the binding never import, load or run anything under
    oracle/ (only tests, the smoke check and the bench's CPU baseline do)."""
    pkg = os.path.join(ROOT, "paper_2410_19123_amd")
    # an import of the oracle package, its shared library, or a path into it
    pat = re.compile(r"^\s*(from|import)\s+oracle\b|liboracle|[\"']oracle[\"'/]", re.M)
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                src = open(os.path.join(dirpath, f)).read()
                assert not pat.search(src), os.path.join(dirpath, f)
