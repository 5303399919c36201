"""Chained-trajectory parity: T consecutive region-sparse steps with the stateful
gate (frozen change of skipped regions, forced reactivation after K = 5 skips)
in both skip modes, the HIP path against the oracle's trajectory stored by
tests/golden/make_trajectory_goldens.py (recipe in its docstring): image at
2 blocks for 50 steps, audio at 2 blocks for 100.

Each side runs its own trajectory from the same start: the latent after a step
is that side's own update plus the same seeded perturbation, and the K/V and
drift caches carry that side's own values from step to step.  At every step
the active mask, the skip counters and the active count must be identical
(the first divergence fails the test at once, Sec. 3.2 and App. eq.
forced-reactivation); the step's latent increment at sampled active tokens
(and at skipped ones under the cached-drift rule, eq. sf-update) within 2e-2
normwise relative error of the oracle's; after the last step the accumulated
model increment at 64 fixed tokens within 2e-2.
"""
import os

import numpy as np
import pytest
import torch

from paper_2607_12121_amd import flashdiff as fdl
from paper_2607_12121_amd import workloads as wl
from tests import gpu_harness as gh
from tests.golden import make_depth_goldens as mdg
from tests.golden import make_trajectory_goldens as mtg
from tests.helpers import rel_err

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    fdl.lib()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("tag,mode", [("freeze", fdl.FD_SKIP_FREEZE), ("drift", fdl.FD_SKIP_REUSE_DRIFT)])
@pytest.mark.parametrize("name", ["image", "audio"])
def test_chained_trajectory(name, tag, mode):
    path = os.path.join(GOLDEN, f"trajectory_{name}.npz")
    gold = np.load(path, allow_pickle=False)
    assert str(gold["source_sha256"]) == mdg.source_digest(), \
        f"{path} is stale: rerun python -m tests.golden.make_trajectory_goldens {name}"
    T = int(gold["T"])
    w = mtg.traj_workload(name)
    assert int(gold["L"]) == w.L and int(gold["max_skip"]) == mtg.MAX_SKIP
    rm = wl.region_map(w)
    plan = fdl.make_plan(rm.token_region, rm.req_tok_off, rm.n_regions)
    d = fdl.dims(w.C, w.D, w.H, w.dh, w.F)
    params = {k: v.cuda() for k, v in wl.make_params(w).items()}
    st = fdl.SparseStep(plan, d, params, w.L)   # K/V and drift caches start at zero
    inp = wl.step_inputs(w, 0, rmap=rm)
    x = torch.from_numpy(inp.x_cur).cuda()
    x_prev = torch.from_numpy(inp.x_prev).cuda()
    x_start = inp.x_cur.astype(np.float64)
    noise_sum = np.zeros((w.N, w.C))
    dt = torch.from_numpy(wl.dt_per_request(w)).cuda()
    gh.say(f"trajectory {name} {tag}: {T} steps, L={w.L}, K={mtg.MAX_SKIP}")
    worst = {"dx": 0.0, "drift": 0.0}
    for n in range(T):
        x_in = x.clone()
        st.step(x, x_prev, torch.from_numpy(gold[f"{tag}_eps"][n]).cuda(), dt, wl.make_cond(w, n).cuda(),
                max_skip=mtg.MAX_SKIP, skip_mode=mode)
        torch.cuda.synchronize()
        act = st.active.cpu().numpy().astype(bool)
        np.testing.assert_array_equal(act, gold[f"{tag}_active"][n], err_msg=f"{name} {tag}: mask differs at step {n}")
        np.testing.assert_array_equal(st.skip_run.cpu().numpy(), gold[f"{tag}_skip_run"][n],
                                      err_msg=f"{name} {tag}: skip counters differ at step {n}")
        assert int(st.m.item()) == int(gold[f"{tag}_M"][n]), f"step {n}"
        x_new = x.cpu().numpy()
        x_old = x_in.cpu().numpy()
        tok = gold[f"{tag}_tok"][n]
        tok = tok[tok >= 0]
        if len(tok):
            e = rel_err(x_new[tok].astype(np.float64) - x_old[tok], gold[f"{tag}_dx"][n][:len(tok)])
            worst["dx"] = max(worst["dx"], e)
            assert e <= gh.TOL, f"{name} {tag}: step {n} latent increment error {e:.3e}"
        sk = gold[f"{tag}_sk_tok"][n]
        sk = sk[sk >= 0]
        if len(sk):
            e = rel_err(x_new[sk].astype(np.float64) - x_old[sk], gold[f"{tag}_sk_dx"][n][:len(sk)])
            worst["drift"] = max(worst["drift"], e)
            assert e <= gh.TOL, f"{name} {tag}: step {n} drift increment error {e:.3e}"
        skipped = np.nonzero(~act[rm.token_region])[0]
        if mode == fdl.FD_SKIP_FREEZE:
            np.testing.assert_array_equal(x_new[skipped], x_old[skipped])
        if n == T - 1:
            break
        # next step: this side's update plus the shared perturbation
        pert = mtg.perturbation(w, n + 1, rm)
        noise_sum += pert
        x_prev = x_in
        x = torch.from_numpy((x_new.astype(np.float64) + pert).astype(np.float32)).cuda()
        if n % 10 == 0:
            gh.say(f"  step {n}: M={int(st.m.item())} worst dx error {worst['dx']:.2e}")
    ft = gold[f"{tag}_final_tok"]
    acc_gpu = x.cpu().numpy()[ft].astype(np.float64) - x_start[ft] - noise_sum[ft]
    acc_orc = gold[f"{tag}_final_x"].astype(np.float64) - x_start[ft] - noise_sum[ft]
    e_final = rel_err(acc_gpu, acc_orc)
    gh.say(f"  {name} {tag}: masks identical over {T} steps; worst step increment error {worst['dx']:.2e}, "
           f"drift {worst['drift']:.2e}; accumulated model increment error {e_final:.2e}")
    assert e_final <= gh.TOL
