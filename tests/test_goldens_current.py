"""The stored oracle values (tests/golden/*.npz) are current: each was written by
its committed script from the code of the oracle and the seeded generators
that this tree holds (digest of that code, comments and docstrings left out),
and holds what the GPU tests read.  CPU only."""
import os

import numpy as np
import pytest

from paper_2607_12121_amd import workloads as wl
from tests.golden import make_depth_goldens as mdg
from tests.golden import make_trajectory_goldens as mtg

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FILES = ["depth_video.npz", "depth_packed.npz", "trajectory_image.npz", "trajectory_audio.npz"]


@pytest.mark.parametrize("fname", FILES)
def test_golden_is_current(fname):
    path = os.path.join(GOLDEN, fname)
    assert os.path.exists(path), f"{path} missing: run its script under tests/golden/"
    g = np.load(path, allow_pickle=False)
    assert str(g["source_sha256"]) == mdg.source_digest(), f"{fname} is stale: rerun its script"


@pytest.mark.parametrize("name", ["video", "packed"])
def test_depth_golden_shapes(name):
    g = np.load(os.path.join(GOLDEN, f"depth_{name}.npz"), allow_pickle=False)
    w = wl.WORKLOADS[name]
    M, rows = int(g["M"]), g["rows"]
    assert int(g["L"]) == w.L and len(g["idx"]) == M and g["cu_q"][-1] == M
    assert g["active"].shape == (w.R,) and rows[0] == 0 and rows[-1] == M - 1
    assert g["h"].shape == (len(rows), w.D) and g["v"].shape == (len(rows), w.C)
    assert g["k_rows"].shape == (len(g["kv_blocks"]), len(g["kv_rows"]), w.D)
    assert np.all(np.isfinite(g["h"])) and np.all(np.isfinite(g["k_rows"].astype(np.float64)))


@pytest.mark.parametrize("name", ["image", "audio"])
def test_trajectory_golden_margins(name):
    """Every gated step's threshold sits far from every weight (the property that
    makes identical masks a fair requirement), and forced reactivation keeps every
    skip run within K."""
    g = np.load(os.path.join(GOLDEN, f"trajectory_{name}.npz"), allow_pickle=False)
    assert int(g["T"]) == mtg.STEPS[name]
    for tag, _ in mtg.MODES:
        m = g[f"{tag}_margin"][1:]
        assert np.all(m >= mtg.MIN_MARGIN)
        assert g[f"{tag}_skip_run"].max() <= mtg.MAX_SKIP
        assert g[f"{tag}_active"][0].all()          # the warm-up step is dense
        assert 0 < g[f"{tag}_M"][1:].min() < wl.WORKLOADS[name].N
