"""Expected values of the full-depth step parity for the workloads whose oracle
step is too slow to run inside a GPU test: video (32760 tokens, 30 blocks) and
the packed batch (8 requests, 21248 tokens, 24 blocks).

Writes tests/golden/depth_<workload>.npz.  Calls only the oracle
(oracle/flashdiff_oracle.py) and the seeded input generators
(paper_2607_12121_amd/workloads.py); no stored value comes from the HIP path.

The inputs are those of the GPU test (tests/test_gpu_depth.py, through
tests/gpu_harness.make_case): step 0 of the workload's recipe, its designed
thresholds, eta = 0, no forced reactivation, the FREEZE skip mode, the seeded
random K/V caches and drift cache.  Every block runs on every active row (the
oracle needs all of them for the next block's keys and values); the last
block, the final layer and the update run on a sample of active rows.

Stored: the sampled rows and their tokens, the active mask, the index list and
per-request offsets, the last block's hidden rows, the velocity rows, the
updated latent rows (fp32, as the oracle leaves them), and the key and value
rows the oracle wrote at the first KV_ROWS sampled tokens in blocks 0, L/2 and
L-1 (rounded to float16: 2^-11 relative, far below the 2e-2 parity bound).
A digest of the oracle's and the generator module's code (comments and
docstrings left out) is stored too, so a CPU test can tell when the goldens
are stale.

Run from the repository root:  python -m tests.golden.make_depth_goldens [video] [packed]
"""
from __future__ import annotations

import ast
import hashlib
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

HERE = os.path.dirname(os.path.abspath(__file__))
SAMPLE = 64        # sampled active rows of the last block (plus the first and the last row)
KV_ROWS = 32       # sampled rows whose written K/V rows are stored
SOURCES = (os.path.join(ROOT, "oracle", "flashdiff_oracle.py"),
           os.path.join(ROOT, "paper_2607_12121_amd", "workloads.py"))


def source_digest(paths=SOURCES) -> str:
    """sha256 over the code of the given Python modules, comments and docstrings
    left out (the abstract syntax tree without docstring expressions), so that a
    change of wording does not mark the stored values stale."""
    h = hashlib.sha256()
    for p in paths:
        with open(p) as f:
            tree = ast.parse(f.read())
        for node in ast.walk(tree):
            body = getattr(node, "body", None)
            if isinstance(body, list) and body and isinstance(body[0], ast.Expr) and \
                    isinstance(getattr(body[0], "value", None), ast.Constant) and isinstance(body[0].value.value, str):
                node.body = body[1:] or [ast.Pass()]
        h.update(ast.dump(tree, include_attributes=False).encode())
    return h.hexdigest()


def sample_rows(M: int, n: int = SAMPLE, seed: int = 3) -> np.ndarray:
    """Sorted sample of active rows, always holding the first and the last."""
    rng = np.random.default_rng(seed)
    return np.unique(np.concatenate([[0, M - 1], rng.choice(M, n, replace=False)])).astype(np.int64)


class LazyCache:
    """Per-block float64 view of a bf16 [L, N, D] cache, converted when the
    oracle first touches a block (the whole float64 cache of the video model
    would not fit in memory).  The oracle visits blocks in order and writes the
    active rows in place; `on_done(l, array)` sees each block after its turn."""

    def __init__(self, src: torch.Tensor, on_done):
        self.src, self.on_done = src, on_done
        self.cur = None

    def __len__(self):
        return self.src.shape[0]

    def __getitem__(self, l: int) -> np.ndarray:
        if self.cur is not None and self.cur[0] == l:
            return self.cur[1]
        if self.cur is not None:
            self.on_done(*self.cur)
        self.cur = (l, self.src[l].to(torch.float64).numpy())
        return self.cur[1]

    def finish(self):
        if self.cur is not None:
            self.on_done(*self.cur)
            self.cur = None


def make(name: str) -> str:
    w = wl.WORKLOADS[name]
    t0 = time.time()
    digest = source_digest()   # of the code this run executes
    rm = wl.region_map(w)
    lay = orc.Layout(rm.token_region.astype(np.int64), rm.req_tok_off.astype(np.int64), rm.n_regions)
    params = wl.make_params(w)
    inp = wl.step_inputs(w, 0, rmap=rm)
    cond = wl.make_cond(w, 0).numpy().astype(np.float64)
    kc, vc = wl.make_kv_cache(w)
    vcache = np.random.default_rng(w.seed + 5).standard_normal((w.N, w.C)).astype(np.float32)
    print(f"[{name}] inputs drawn in {time.time() - t0:.0f} s", flush=True)

    # the gate alone, for the index list and the row sample
    score = orc.region_score(lay, inp.x_cur, inp.x_prev)
    _, _, active = orc.gate_select(lay, score, np.zeros(w.R), np.zeros(w.R, np.int32), np.ones(w.R, bool),
                                   inp.eps, 0.0, 0)
    idx, cu = orc.active_rows(lay, active)
    M = len(idx)
    rows = sample_rows(M)
    kv_rows = rows[:KV_ROWS]
    kv_blocks = sorted({0, w.L // 2, w.L - 1})
    kept = {}

    def keep(tag):
        def f(l, arr):
            if l in kv_blocks:
                kept[(tag, l)] = arr[idx[kv_rows]].astype(np.float16)
            print(f"[{name}] block {l} {tag} done at {time.time() - t0:.0f} s", flush=True)
        return f

    k_lazy, v_lazy = LazyCache(kc, keep("k")), LazyCache(vc, keep("v"))
    p64 = {k: v.to(torch.float64).numpy() for k, v in params.items()}
    out = orc.sparse_step(lay, p64, w.H, cond, inp.x_cur, inp.x_prev, orc.GateState.fresh(w.R), inp.eps,
                          0.0, 0, k_lazy, v_lazy, vcache, wl.dt_per_request(w), orc.FREEZE, sample_rows=rows)
    k_lazy.finish()
    v_lazy.finish()
    assert np.array_equal(out["active"], active) and np.array_equal(out["idx"], idx)
    toks = idx[rows]
    path = os.path.join(HERE, f"depth_{name}.npz")
    np.savez_compressed(
        path, workload=name, L=w.L, M=M, rows=rows, kv_rows=kv_rows, kv_blocks=np.asarray(kv_blocks),
        active=active, idx=idx.astype(np.int32), cu_q=cu.astype(np.int32),
        h=out["h"].astype(np.float32), v=out["v"].astype(np.float32), x_rows=out["x"][toks],
        k_rows=np.stack([kept[("k", l)] for l in kv_blocks]), v_rows=np.stack([kept[("v", l)] for l in kv_blocks]),
        source_sha256=digest)
    print(f"[{name}] wrote {path} ({os.path.getsize(path) / 1e6:.2f} MB) after {time.time() - t0:.0f} s",
          flush=True)
    return path


if __name__ == "__main__":
    for n in (sys.argv[1:] or ["video", "packed"]):
        make(n)
