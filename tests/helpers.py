"""Shared test helpers: workload -> oracle inputs (float64 numpy views of the drawn values)."""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from paper_2607_12121_amd import workloads as wl
from oracle import flashdiff_oracle as orc


def oracle_layout(w: wl.Workload) -> orc.Layout:
    rm = wl.region_map(w)
    return orc.Layout(rm.token_region.astype(np.int64), rm.req_tok_off.astype(np.int64), rm.n_regions)


def params_f64(params: Dict[str, torch.Tensor]) -> Dict[str, np.ndarray]:
    return {k: v.detach().to("cpu", torch.float64).numpy() for k, v in params.items()}


def small_workload(base: str = "tiny", **kw) -> wl.Workload:
    w = wl.WORKLOADS[base]
    d = dict(w.__dict__)
    d.update(kw)
    return wl.Workload(**d)


def rel_err(a: np.ndarray, b: np.ndarray) -> float:
    """Normwise infinity-relative error max|a - b| / max|b|."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.max(np.abs(b)) if b.size else 0.0
    return float(np.max(np.abs(a - b)) / den) if den > 0 else float(np.max(np.abs(a - b), initial=0.0))


def random_gate_layout(rng: np.random.Generator, B: int, max_regions: int = 6, max_tokens: int = 5):
    """A random request-major layout with contiguous region ids per request."""
    token_region, req_tok_off = [], [0]
    rid = 0
    for _ in range(B):
        nr = int(rng.integers(1, max_regions + 1))
        toks = []
        for r in range(nr):
            toks += [rid + r] * int(rng.integers(1, max_tokens + 1))
        rng.shuffle(toks)
        token_region += toks
        req_tok_off.append(req_tok_off[-1] + len(toks))
        rid += nr
    return orc.Layout(np.asarray(token_region, np.int64), np.asarray(req_tok_off, np.int64), rid)
