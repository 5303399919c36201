"""Expected values of the chained-trajectory test (tests/test_gpu_trajectory.py):
T consecutive region-sparse steps of a reduced-depth model with the stateful
gate (frozen change, forced reactivation after K = 5 skips), in both skip
modes, the oracle's trajectory written to tests/golden/trajectory_<name>.npz.

Calls only the oracle (oracle/flashdiff_oracle.py) and the seeded input
generators (paper_2607_12121_amd/workloads.py); no stored value comes from the
HIP path.

Trajectory (identical recipe on both sides; the GPU test rebuilds every input
but the thresholds, which it reads from here):
  * model: the workload's DiT at L = 2 blocks; K/V caches and drift cache
    start at zero; conditioning make_cond(w, n) at step n; h = the workload's dt.
  * step 0 is the dense warm-up (eps = 0: every region active), on
    x_cur = x_0, x_prev from step_inputs(w, 0).
  * after step n the latent is updated by the step (eq. sf-update), and a
    seeded per-region perturbation is added:
        x_{n+1} = update_n(x_n) + NOISE_SCALE * xi_{n+1},
    xi_{n+1} = step_inputs(w_noise, n + 1, x_prev = 0).x_cur, w_noise the
    workload with a schedule long enough that sigma stays 1: per region
    amplitude U[1, 2] (hot set of the workload's activity model) or
    U[0.05, 0.45] (cold) times N(0, 1).  It stands in for the structured change
    of a trained model's latent, which random weights do not have (their
    velocity gives every region about the same activity), so that the gate
    sees well separated regions; step n + 1 scores x_{n+1} - x_n.
  * eps at step n >= 1: per request, the geometric midpoint of the widest gap
    of the oracle's sorted gate weights w_i = (s~_i + eta) / D_b (eta = 0),
    with at least one region on each side; the smallest relative distance of
    any weight to eps is asserted >= MIN_MARGIN, far above the differences
    between the two sides' scores.
Stored per skip mode and step: eps, the active mask, the skip counters, the
active count, the latent increment x_{n+1} - x_n of the step's update (before
the perturbation) at ROWS sampled active tokens (and, in the drift mode, at
two skipped tokens); and the final latent at 64 fixed tokens.

Run from the repository root:  python -m tests.golden.make_trajectory_goldens [image] [audio]
"""
from __future__ import annotations

import dataclasses
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import flashdiff_oracle as orc  # noqa: E402
from paper_2607_12121_amd import workloads as wl  # noqa: E402
from tests.golden.make_depth_goldens import source_digest  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))
STEPS = {"image": 50, "audio": 100}
LAYERS = 2
MAX_SKIP = 5
NOISE_SCALE = 0.1
MIN_MARGIN = 0.05
ROWS = 4
FINAL_TOKENS = 64
MODES = (("freeze", orc.FREEZE), ("drift", orc.REUSE_DRIFT))


def traj_workload(name: str) -> wl.Workload:
    return wl.WORKLOADS[name].with_layers(LAYERS)


def perturbation(w: wl.Workload, n: int, rmap) -> np.ndarray:
    """NOISE_SCALE * xi_n (fp32 [N, C]), shared recipe of both sides."""
    w_noise = dataclasses.replace(w, steps=10 ** 9)
    xi = wl.step_inputs(w_noise, n, x_prev=np.zeros((w.N, w.C), np.float32), rmap=rmap).x_cur
    return (NOISE_SCALE * xi.astype(np.float64)).astype(np.float32)


def widest_gap_eps(lay: orc.Layout, s_tilde: np.ndarray, eta: float = 0.0):
    """Per request: eps at the geometric midpoint of the widest relative gap of the
    sorted gate weights (at least one region on each side); returns eps [B] and
    the smallest relative distance of any weight to its request's eps."""
    wts = orc.gate_weights(lay, s_tilde, eta)
    rreq = lay.region_request()
    eps = np.zeros(lay.n_requests)
    margin = np.inf
    for b in range(lay.n_requests):
        wb = np.sort(wts[rreq == b])
        if len(wb) < 2:
            eps[b] = 0.0
            continue
        ratio = wb[1:] / np.maximum(wb[:-1], 1e-300)
        k = int(np.argmax(ratio))
        eps[b] = float(np.sqrt(wb[k] * wb[k + 1]))
        margin = min(margin, float(np.min(np.abs(wb - eps[b]) / eps[b])))
    return eps, margin


def sample_tokens(idx: np.ndarray, n: int, k: int = ROWS) -> np.ndarray:
    rng = np.random.default_rng(1000 + n)
    return np.sort(idx[rng.choice(len(idx), min(k, len(idx)), replace=False)]) if len(idx) else idx[:0]


def skipped_tokens(lay: orc.Layout, active: np.ndarray, n: int, k: int = 2) -> np.ndarray:
    sk = np.nonzero(~active[lay.token_region])[0]
    rng = np.random.default_rng(2000 + n)
    return np.sort(sk[rng.choice(len(sk), min(k, len(sk)), replace=False)]) if len(sk) else sk


def run_mode(name: str, mode: int, T: int):
    w = traj_workload(name)
    rm = wl.region_map(w)
    lay = orc.Layout(rm.token_region.astype(np.int64), rm.req_tok_off.astype(np.int64), rm.n_regions)
    p64 = {k: v.to(torch.float64).numpy() for k, v in wl.make_params(w).items()}
    inp = wl.step_inputs(w, 0, rmap=rm)
    kc = [np.zeros((w.N, w.D)) for _ in range(w.L)]
    vc = [np.zeros((w.N, w.D)) for _ in range(w.L)]
    vcache = np.zeros((w.N, w.C), np.float32)
    gate = orc.GateState.fresh(w.R)
    dt = wl.dt_per_request(w)
    x_prev, x_cur = inp.x_prev, inp.x_cur
    rec = {k: [] for k in ("eps", "active", "skip_run", "M", "tok", "dx", "sk_tok", "sk_dx", "margin")}
    for n in range(T):
        if n == 0:
            eps, margin = np.zeros(w.B), np.inf
        else:
            score = orc.region_score(lay, x_cur, x_prev)
            s_t = np.where(gate.active, score, gate.s_tilde)
            eps, margin = widest_gap_eps(lay, s_t)
            assert margin >= MIN_MARGIN, f"{name} step {n}: threshold margin {margin:.3g}"
        cond = wl.make_cond(w, n).numpy().astype(np.float64)
        out = orc.sparse_step(lay, p64, w.H, cond, x_cur, x_prev, gate, eps, 0.0, MAX_SKIP, kc, vc, vcache, dt,
                              mode)
        tok = sample_tokens(out["idx"], n)
        sk = skipped_tokens(lay, out["active"], n) if mode == orc.REUSE_DRIFT else np.zeros(0, np.int64)
        rec["eps"].append(eps)
        rec["active"].append(out["active"])
        rec["skip_run"].append(out["gate"].skip_run)
        rec["M"].append(len(out["idx"]))
        rec["margin"].append(margin)
        rec["tok"].append(np.pad(tok, (0, ROWS - len(tok)), constant_values=-1))
        d = np.zeros((ROWS, w.C), np.float32)
        d[:len(tok)] = (out["x"][tok].astype(np.float64) - x_cur[tok].astype(np.float64)).astype(np.float32)
        rec["dx"].append(d)
        rec["sk_tok"].append(np.pad(sk, (0, 2 - len(sk)), constant_values=-1))
        e = np.zeros((2, w.C), np.float32)
        e[:len(sk)] = (out["x"][sk].astype(np.float64) - x_cur[sk].astype(np.float64)).astype(np.float32)
        rec["sk_dx"].append(e)
        gate, vcache = out["gate"], out["vcache"]
        x_prev = x_cur
        x_cur = (out["x"].astype(np.float64) + perturbation(w, n + 1, rm)).astype(np.float32)
        if n % 10 == 0:
            print(f"  [{name} mode {mode}] step {n}: M={len(out['idx'])} margin={margin:.3g}", flush=True)
    # x_cur now holds x_T (after the last update and its perturbation); store the
    # last update's result instead: x_T minus the perturbation is out["x"]
    final_tok = np.sort(np.random.default_rng(3000).choice(w.N, FINAL_TOKENS, replace=False))
    arrs = {k: np.asarray(v) for k, v in rec.items()}
    arrs["final_tok"] = final_tok
    arrs["final_x"] = out["x"][final_tok]
    return arrs


def make(name: str) -> str:
    t0 = time.time()
    digest = source_digest()
    T = STEPS[name]
    data = {"workload": name, "T": T, "L": LAYERS, "max_skip": MAX_SKIP, "noise_scale": NOISE_SCALE,
            "source_sha256": digest}
    for tag, mode in MODES:
        print(f"[{name}] {tag}: {T} steps", flush=True)
        for k, v in run_mode(name, mode, T).items():
            data[f"{tag}_{k}"] = v
    path = os.path.join(HERE, f"trajectory_{name}.npz")
    np.savez_compressed(path, **data)
    print(f"[{name}] wrote {path} ({os.path.getsize(path) / 1e6:.2f} MB) after {time.time() - t0:.0f} s", flush=True)
    return path


if __name__ == "__main__":
    for n in (sys.argv[1:] or ["image", "audio"]):
        make(n)
