"""The entry point that allocates nothing, fd_region_score_noalloc (built-in
scratch for the partial sums), against fd_region_score (caller workspace),
through the C ABI: bit-identical scores, and within 1e-12 of the oracle, on two
calls in a row, the second on a smaller input; an input whose partials exceed
the built-in scratch is rejected before anything is enqueued."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import flashdiff_oracle as orc
from paper_2607_12121_amd import flashdiff as fdl
from paper_2607_12121_amd import workloads as wl
from tests import gpu_harness as gh

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    fdl.lib()


def _both(name: str, step: int):
    w = wl.WORKLOADS[name]
    rm = wl.region_map(w)
    plan = fdl.make_plan(rm.token_region, rm.req_tok_off, rm.n_regions)
    inp = wl.step_inputs(w, step, rmap=rm)
    xc, xp = torch.from_numpy(inp.x_cur).cuda(), torch.from_numpy(inp.x_prev).cuda()
    ws = torch.empty(max(fdl.fd_region_score_ws_size(plan, w.C), 256), dtype=torch.uint8, device="cuda")
    ref = torch.full((w.R,), np.nan, dtype=torch.float64, device="cuda")
    got = torch.full((w.R,), np.nan, dtype=torch.float64, device="cuda")
    gh.say(f"no-alloc score {name}: N={w.N} R={w.R} partial bytes={fdl.fd_region_score_ws_size(plan, w.C)}")
    fdl.fd_region_score(plan, w.C, xc, xp, ref, ws)
    fdl.fd_region_score_noalloc(plan, w.C, xc, xp, got)
    torch.cuda.synchronize()
    lay = orc.Layout(rm.token_region.astype(np.int64), rm.req_tok_off.astype(np.int64), rm.n_regions)
    want = orc.region_score(lay, inp.x_cur, inp.x_prev)
    return ref.cpu().numpy(), got.cpu().numpy(), want


def test_noalloc_score_equals_workspace_score_on_two_calls():
    # first the video request (140 regions x 8 chunks of partials), then a smaller
    # input (the image request: 64 regions x 2 chunks) on the same built-in scratch
    for name, step in (("video", 0), ("image", 1)):
        ref, got, want = _both(name, step)
        assert np.array_equal(got, ref), f"{name}: no-alloc scores differ from the workspace entry point"
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=0)


def test_noalloc_score_rejects_partials_beyond_the_scratch():
    """A plan whose (region, chunk) partials need more than the 1 MiB built-in
    scratch: FD_E_UNSUPPORTED from the host-side check, nothing enqueued.  The
    descriptor's device arrays are real (small) tensors; the check reads only its
    sizes."""
    small = torch.zeros(8, dtype=torch.int32, device="cuda")
    x = torch.zeros(16, dtype=torch.float32, device="cuda")
    score = torch.zeros(8, dtype=torch.float64, device="cuda")
    # 300 regions of up to 65536 tokens at C = 16: 300 x 512 chunks x 8 bytes > 1 MiB
    plan = fdl.FdPlan(300 * 65536, 300, 1, 65536, 300 * 65536, *([small.data_ptr()] * 6))
    st = fdl.lib().fd_region_score_noalloc(ctypes.byref(plan), 16, x.data_ptr(), x.data_ptr(), score.data_ptr(),
                                           torch.cuda.current_stream().cuda_stream)
    assert st == 3, st
    assert b"scratch" in fdl.lib().fd_last_error()
    torch.cuda.synchronize()
    assert bool((score == 0).all())
