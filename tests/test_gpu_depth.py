"""Full-depth step parity: one region-sparse step through every block of each
workload's model (image, audio and the packed batch: 24 blocks; video: 30), the
HIP path through the C ABI against the oracle.

Image and audio run the oracle inside the test on every active row.  The
video and packed oracle steps take minutes to an hour of CPU time, so their
expected values come from tests/golden/depth_<workload>.npz, written by
tests/golden/make_depth_goldens.py, which calls only the oracle and the seeded
generators (the last block, the final layer and the update on 66 sampled
active rows; written K/V rows of blocks 0, L/2 and L-1 at 32 of them).

Bit-exact: region mask, index list, offsets and count; skipped latent, drift
and K/V rows unchanged in every block.  Within 2e-2 normwise relative error:
hidden rows after the last block, velocity, latent increments, drift rows and
the written K/V rows.
"""
import os

import numpy as np
import pytest
import torch

from oracle import flashdiff_oracle as orc
from paper_2607_12121_amd import flashdiff as fdl
from paper_2607_12121_amd import workloads as wl
from tests import gpu_harness as gh
from tests.golden import make_depth_goldens as mdg
from tests.helpers import rel_err

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    fdl.lib()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["image", "audio"])
def test_full_depth_live(name):
    """Every block of the model, the oracle on every active row in the test."""
    case = gh.make_case(name)
    inp = case.inp
    gh.say(f"full depth {name}: N={case.w.N} L={case.w.L} M={int(inp.hot[case.rmap.token_region].sum())}")
    g, st = gh.run_gpu(case, inp.eps, inp.x_cur, inp.x_prev)
    gh.say(f"  GPU step done; oracle on {g['M']} rows x {case.w.L} blocks")
    o = gh.run_oracle(case, inp.eps, inp.x_cur, inp.x_prev)
    errs = gh.compare_step(case, g, o, inp.x_cur, st)
    gh.say(f"  errors {name} at depth {case.w.L}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["video", "packed"])
def test_full_depth_golden(name):
    """Every block of the model against the oracle's stored step (sampled rows)."""
    path = os.path.join(GOLDEN, f"depth_{name}.npz")
    gold = np.load(path, allow_pickle=False)
    assert str(gold["source_sha256"]) == mdg.source_digest(), \
        f"{path} is stale: rerun python -m tests.golden.make_depth_goldens {name}"
    case = gh.make_case(name)
    w, inp = case.w, case.inp
    assert int(gold["L"]) == w.L
    gh.say(f"full depth {name} (stored oracle step): N={w.N} L={w.L} M={int(gold['M'])}")
    g, st = gh.run_gpu(case, inp.eps, inp.x_cur, inp.x_prev)
    gh.say("  GPU step done")
    # gate: exact, against the stored oracle and a fresh oracle evaluation
    np.testing.assert_array_equal(g["active"], gold["active"])
    np.testing.assert_array_equal(g["idx"], gold["idx"])
    np.testing.assert_array_equal(g["cu_q"], gold["cu_q"])
    assert g["M"] == int(gold["M"])
    s_o = orc.region_score(case.layout, inp.x_cur, inp.x_prev)
    np.testing.assert_allclose(g["score"], s_o, rtol=1e-12, atol=0)
    rows = gold["rows"]
    toks = g["idx"][rows]
    errs = {"h": rel_err(g["h"][rows], gold["h"]), "v": rel_err(g["v"][rows], gold["v"]),
            "dx": rel_err(g["x"][toks] - inp.x_cur[toks], gold["x_rows"].astype(np.float64) - inp.x_cur[toks]),
            "vcache": rel_err(g["vcache"][toks], gold["v"])}
    # skipped rows untouched: latent, drift, and every block's K/V rows
    skipped = np.nonzero(~gold["active"][case.rmap.token_region])[0]
    np.testing.assert_array_equal(g["x"][skipped], inp.x_cur[skipped])
    np.testing.assert_array_equal(g["vcache"][skipped], case.vcache[skipped])
    sk = torch.from_numpy(skipped)
    for l in range(w.L):
        assert torch.equal(st.k_cache[l].cpu()[sk], case.k_cache[l][sk]), f"stale K rows changed in block {l}"
        assert torch.equal(st.v_cache[l].cpu()[sk], case.v_cache[l][sk]), f"stale V rows changed in block {l}"
    kv_toks = torch.from_numpy(g["idx"][gold["kv_rows"]].astype(np.int64))
    kerr = verr = 0.0
    for j, l in enumerate(gold["kv_blocks"]):
        kg = st.k_cache[int(l)].cpu()[kv_toks].to(torch.float64).numpy()
        vg = st.v_cache[int(l)].cpu()[kv_toks].to(torch.float64).numpy()
        kerr = max(kerr, rel_err(kg, gold["k_rows"][j].astype(np.float64)))
        verr = max(verr, rel_err(vg, gold["v_rows"][j].astype(np.float64)))
    errs["k"], errs["v_rows"] = kerr, verr
    gh.say(f"  errors {name} at depth {w.L}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for k, e in errs.items():
        assert e <= gh.TOL, f"{name}: {k} error {e:.3e} > {gh.TOL}"
