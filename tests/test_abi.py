"""CPU tests of the C ABI: the library loads, exports every declared entry point,
builds region plans, and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_12121_amd import flashdiff as fdl
from paper_2607_12121_amd import workloads as wl

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "flashdiff.h")


def _gpu_visible() -> bool:
    import torch
    return torch.cuda.device_count() > 0


# These tests hand dummy addresses (0x1000) to entry points and rely on the
# argument validation rejecting the call before any launch.  Where a GPU is
# visible a regression in that validation would enqueue a kernel on them, so
# they run only on hosts without one (the CPU tier).
no_gpu = pytest.mark.skipif(_gpu_visible(), reason="passes dummy device addresses; CPU-only hosts")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fd_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = fdl.lib()
    names = _declared()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert set(fdl.exported_symbols()) == set(names)
    assert "gfx950" in fdl.version()


@pytest.mark.parametrize("name", list(wl.WORKLOADS))
def test_plan_build_matches_region_map(name):
    w = wl.WORKLOADS[name]
    rm = wl.region_map(w)
    host = fdl.fd_plan_build(rm.token_region, rm.req_tok_off, rm.n_regions)
    np.testing.assert_array_equal(host["req_reg_off"], rm.req_reg_off)
    np.testing.assert_array_equal(host["region_req"], rm.region_req)
    counts = np.bincount(rm.token_region, minlength=rm.n_regions)
    np.testing.assert_array_equal(np.diff(host["region_ptr"]), counts)
    for r in range(0, rm.n_regions, max(1, rm.n_regions // 17)):
        toks = host["region_tokens"][host["region_ptr"][r]:host["region_ptr"][r + 1]]
        np.testing.assert_array_equal(toks, np.nonzero(rm.token_region == r)[0])
    assert host["max_region_tokens"] == counts.max()
    assert host["max_request_tokens"] == np.diff(rm.req_tok_off).max()


@pytest.mark.parametrize("token_region,req_tok_off,R,why", [
    ([0, 1, 2], [0, 3], 4, "empty region"),
    ([0, 1, 5], [0, 3], 3, "region id out of range"),
    ([0, 1, 0, 1], [0, 2, 4], 2, "region spanning two requests"),
    ([1, 1, 0, 0], [0, 2, 4], 2, "regions not request-major"),
    ([0, 0], [0, 1, 1, 2], 1, "empty request"),
    ([0, 0], [0, 3], 1, "request offsets do not end at N"),
])
def test_plan_build_rejects_bad_maps(token_region, req_tok_off, R, why):
    with pytest.raises(fdl.FlashDiffError):
        fdl.fd_plan_build(np.array(token_region), np.array(req_tok_off), R)


def _fake_plan():
    # host-only descriptor with non-null dummy addresses: validation never dereferences them
    return fdl.FdPlan(16, 4, 1, 4, 16, *([0x1000] * 6))


@no_gpu
def test_entry_points_validate_before_launch():
    lib = fdl.lib()
    plan = _fake_plan()
    null = None
    # null plan
    assert lib.fd_region_score(None, 64, 0x1000, 0x1000, 0x1000, 0x1000, 4096, None) == 1
    # unsupported channel count
    assert lib.fd_region_score(ctypes.byref(plan), 12, 0x1000, 0x1000, 0x1000, 0x1000, 4096, None) == 3
    # workspace too small
    need = lib.fd_region_score_ws_size(ctypes.byref(plan), 64)
    assert need > 0
    assert lib.fd_region_score(ctypes.byref(plan), 64, 0x1000, 0x1000, 0x1000, 0x1000, need - 1, None) == 2
    # misaligned latent
    assert lib.fd_region_score(ctypes.byref(plan), 64, 0x1004, 0x1000, 0x1000, 0x1000, need, None) == 1
    # bad dims: D != H*dh, unsupported head dim
    d_bad = fdl.FdDims(64, 1536, 24, 32, 6144)
    assert lib.fd_block_ws_size(ctypes.byref(plan), ctypes.byref(d_bad)) > 0
    w = fdl.FdBlockWeights(*([0x1000] * 10))
    args = (0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 1 << 40, None)
    assert lib.fd_block_forward(ctypes.byref(plan), ctypes.byref(d_bad), ctypes.byref(w), *args) == 2
    d_bad2 = fdl.FdDims(64, 96 * 2, 2, 96, 256)
    assert lib.fd_block_forward(ctypes.byref(plan), ctypes.byref(d_bad2), ctypes.byref(w), *args) == 3
    # block workspace too small
    d = fdl.FdDims(64, 128, 2, 64, 256)
    small = (0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 1024, None)
    assert lib.fd_block_forward(ctypes.byref(plan), ctypes.byref(d), ctypes.byref(w), *small) == 2
    assert b"workspace" in lib.fd_last_error()
    # null weight
    w0 = fdl.FdBlockWeights(*([0x1000] * 9 + [0]))
    assert lib.fd_block_forward(ctypes.byref(plan), ctypes.byref(d), ctypes.byref(w0), *args) == 1
    # more requests than the attention's schedule tables hold
    many = fdl.FdPlan(2050, 1025, 1025, 2, 2, *([0x1000] * 6))
    assert lib.fd_block_forward(ctypes.byref(many), ctypes.byref(d), ctypes.byref(w), *args) == 3
    assert b"1024 requests" in lib.fd_last_error()
    # select: bad gate parameters, too many regions
    g = fdl.FdGate(-1.0, 0)
    assert lib.fd_select(ctypes.byref(plan), *([0x1000] * 2), g, *([0x1000] * 7), None) == 1
    big = fdl.FdPlan(10000, 5000, 1, 2, 10000, *([0x1000] * 6))
    assert lib.fd_select(ctypes.byref(big), *([0x1000] * 2), fdl.FdGate(0.0, 0), *([0x1000] * 7), None) == 3
    # scatter: unknown skip mode
    assert lib.fd_scatter_update(ctypes.byref(plan), 64, *([0x1000] * 7), 7, None) == 1


def test_block_workspace_size_formula():
    plan = fdl.FdPlan(4096, 64, 1, 64, 4096, *([0x1000] * 6))
    d = fdl.FdDims(64, 1536, 24, 64, 6144)
    got = fdl.lib().fd_block_ws_size(ctypes.byref(plan), ctypes.byref(d))
    rows = 6 * 1536 * 4 + 3 * 4096 * 1536 * 2 + 4096 * 6144 * 2 + 4096 * 24 * 4   # ... + per-query normalisers
    # plus the partial scratch shared by split-K and cut attention items: at least four
    # fp32 128x128 tiles per CU, at most four 256x256 ones (plus alignment)
    cus = 256
    assert rows + 4 * cus * (128 * 128 * 4) <= got <= rows + 4 * cus * (256 * 256 * 4) + 8 * 256


@no_gpu
def test_adaln_validates_before_launch():
    lib = fdl.lib()
    d = fdl.FdDims(64, 128, 2, 64, 256)
    assert lib.fd_adaln(ctypes.byref(d), 2, 768, 1, None, 0x1000, 0x1000, 0x1000, None) == 1
    assert lib.fd_adaln(ctypes.byref(d), 0, 768, 1, 0x1000, 0x1000, 0x1000, 0x1000, None) == 1
    assert lib.fd_adaln(ctypes.byref(d), 2, 768, 1, 0x1008, 0x1000, 0x1000, 0x1000, None) == 1
    bad = fdl.FdDims(64, 96, 2, 64, 256)
    assert lib.fd_adaln(ctypes.byref(bad), 2, 768, 1, 0x1000, 0x1000, 0x1000, 0x1000, None) == 2
    # a block with precomputed modulation needs neither cond nor the adaLN weights
    plan = _fake_plan()
    w = fdl.FdBlockWeights(*([0x1000] * 8 + [0, 0, 0x1000]))
    small = (None, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 1024, None)
    assert lib.fd_block_forward(ctypes.byref(plan), ctypes.byref(d), ctypes.byref(w), *small) == 2   # ws too small
    w0 = fdl.FdBlockWeights(*([0x1000] * 8 + [0, 0, 0]))
    assert lib.fd_block_forward(ctypes.byref(plan), ctypes.byref(d), ctypes.byref(w0), *small) == 1   # no modulation


@no_gpu
def test_importance_validates_before_launch():
    lib = fdl.lib()
    plan = _fake_plan()
    d = fdl.FdDims(64, 128, 2, 64, 256)
    bws = lib.fd_block_ws_size(ctypes.byref(plan), ctypes.byref(d))
    iws = lib.fd_importance_ws_size(ctypes.byref(plan), ctypes.byref(d))
    assert iws >= plan.n_tokens * 4 + plan.n_regions * d.H * 4
    ok = (0x1000, bws, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, None, 0x1000, iws, None)
    # null key cache; block workspace too small; importance workspace too small; misaligned
    assert lib.fd_region_importance(ctypes.byref(plan), ctypes.byref(d), *((0x1000, bws, None) + ok[3:])) == 1
    assert lib.fd_region_importance(ctypes.byref(plan), ctypes.byref(d), *((0x1000, bws - 1) + ok[2:])) == 2
    assert lib.fd_region_importance(ctypes.byref(plan), ctypes.byref(d), *(ok[:10] + (iws - 1, None))) == 2
    assert lib.fd_region_importance(ctypes.byref(plan), ctypes.byref(d), *((0x1010,) + ok[1:])) == 1
    # a region whose key rows of one head exceed the LDS staging
    big = fdl.FdPlan(plan.n_tokens, plan.n_regions, 1, 4096, plan.n_tokens, *([0x1000] * 6))
    d128 = fdl.FdDims(64, 256, 2, 128, 256)
    bws = lib.fd_block_ws_size(ctypes.byref(big), ctypes.byref(d128))
    iws = lib.fd_importance_ws_size(ctypes.byref(big), ctypes.byref(d128))
    assert lib.fd_region_importance(ctypes.byref(big), ctypes.byref(d128), 0x1000, bws, *([0x1000] * 6), None,
                                    0x1000, iws, None) == 3
    assert b"LDS" in lib.fd_last_error()


@no_gpu
def test_partition_validates_before_launch():
    lib = fdl.lib()
    to = np.array([0, 100, 300], np.int32)
    ro = np.array([0, 8, 24], np.int32)
    need = lib.fd_partition_ws_size(300, 2)
    assert need >= 2 * 300 * 4 + 302 * 12
    assert lib.fd_partition_ws_size(300, 0) == 0

    def call(t, r, B=2, ws=0x1000, nbytes=need, sal=0x1000):
        t = np.ascontiguousarray(t, np.int32)
        r = np.ascontiguousarray(r, np.int32)
        return lib.fd_partition(B, t.ctypes.data, r.ctypes.data, sal, 0x1000, ws, nbytes, None)

    assert call(to, ro, sal=None) == 1                          # null saliency
    assert call(to, ro, B=0) == 1                               # no request
    assert call([1, 100, 300], ro) == 1                         # offsets not from 0
    assert call(to, [0, 8, 8]) == 1                             # request without regions
    assert call([0, 5, 300], ro) == 1                           # 5 tokens cannot fill 8 regions
    assert b"cannot fill" in lib.fd_last_error()
    assert call(to, ro, ws=0x1010) == 1                         # misaligned workspace
    assert call(to, ro, nbytes=need - 1) == 2                   # workspace too small
    assert call([0, 65536], [0, 8], B=1, nbytes=1 << 30) == 3   # request of 2^16 tokens
    assert call([0, 4096], [0, 1025], B=1, nbytes=1 << 30) == 3  # 1025 regions
    many = np.arange(66, dtype=np.int32) * 10
    assert call(many, many, B=65, nbytes=1 << 30) == 3          # 65 requests in one call
    assert b"requests" in lib.fd_last_error()


def test_binding_fails_loudly_without_the_library(tmp_path):
    """No CPU fallback: with the shared library missing, the binding raises on
    first use (checked in a fresh interpreter, whose loader cache is empty)."""
    import subprocess
    import sys
    code = ("from paper_2607_12121_amd import flashdiff as f\n"
            "try:\n    f.lib()\nexcept f.FlashDiffError as e:\n    print('raised:', e)\n")
    env = dict(os.environ, FLASHDIFF_LIB=str(tmp_path / "absent.so"))
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    out = subprocess.run([sys.executable, "-c", code], env=env, cwd=root, capture_output=True, text=True,
                         timeout=300)
    assert out.returncode == 0 and "raised:" in out.stdout and "missing" in out.stdout, out.stderr[-2000:]


def test_binding_rejects_host_tensors_and_bad_sizes():
    """The wrappers check every tensor before its pointer reaches the library:
    a host tensor, a wrong element type or too few elements raise on the host."""
    import torch
    x = torch.zeros(16, 64)
    with pytest.raises(fdl.FlashDiffError, match="device tensor"):
        fdl._need("x", x, "f32", 16 * 64)
    # the size and type rules themselves, on a stand-in that reports a device
    class T:
        is_cuda = True
        def __init__(self, n, dtype, es=4):
            self.n, self.dtype, self.es = n, dtype, es
        def numel(self):
            return self.n
        def element_size(self):
            return self.es
    fdl._need("ok", T(10, torch.float32), "f32", 10)
    fdl._need("bigger", T(11, torch.float32), "f32", 10)
    with pytest.raises(fdl.FlashDiffError, match="needs exactly"):
        fdl._need("exact", T(11, torch.float32), "f32", 10, exact=True)
    with pytest.raises(fdl.FlashDiffError, match="holds 9"):
        fdl._need("short", T(9, torch.float32), "f32", 10)
    with pytest.raises(fdl.FlashDiffError, match="must be f64"):
        fdl._need("eps", T(4, torch.float32), "f64", 4)
    fdl._need("bf16 bits", T(8, torch.int16, 2), "b16", 8)
    fdl._need("ws", T(300, torch.uint8, 1), "bytes", 256)
    fdl._need("absent", None, "f64", 4, optional=True)
    with pytest.raises(fdl.FlashDiffError, match="required"):
        fdl._need("absent", None, "f64", 4)
