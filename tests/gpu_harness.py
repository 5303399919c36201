"""Shared set-up for the GPU parity tests: one workload's seeded inputs on the host
(for the oracle) and on the device (for the HIP path), the two runs, and the
comparisons.  Nothing here computes the method: the HIP side goes through the
C ABI binding, the oracle side through oracle/."""
from __future__ import annotations

import sys
from dataclasses import dataclass
from typing import Dict, List, Optional

import numpy as np
import torch

from oracle import flashdiff_oracle as orc
from paper_2607_12121_amd import flashdiff as fdl
from paper_2607_12121_amd import workloads as wl
from tests.helpers import oracle_layout, params_f64, rel_err

TOL = 2e-2   # max normwise relative error of floating-point outputs (bf16 operands, fp32 accumulate)


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@dataclass
class Case:
    w: wl.Workload
    rmap: wl.RegionMap
    layout: orc.Layout
    params: Dict[str, torch.Tensor]      # host, as drawn
    params_gpu: Dict[str, torch.Tensor]
    inp: wl.StepInputs
    cond: torch.Tensor                    # host fp32 [B, D]
    k_cache: torch.Tensor                 # host bf16 [L, N, D]
    v_cache: torch.Tensor
    vcache: np.ndarray                    # fp32 [N, C] cached drift
    plan: fdl.Plan
    dims: fdl.FdDims


def make_case(name: str, L: Optional[int] = None, step: int = 0, workload: Optional[wl.Workload] = None,
              cache: str = "random") -> Case:
    w = workload or wl.WORKLOADS[name]
    if L is not None:
        w = w.with_layers(L)
    rm = wl.region_map(w)
    params = wl.make_params(w)
    inp = wl.step_inputs(w, step, rmap=rm)
    cond = wl.make_cond(w, step)
    if cache == "random":
        kc, vc = wl.make_kv_cache(w)
    else:
        kc = torch.zeros((w.L, w.N, w.D), dtype=torch.bfloat16)
        vc = torch.zeros((w.L, w.N, w.D), dtype=torch.bfloat16)
    rng = np.random.default_rng(w.seed + 5)
    vcache = rng.standard_normal((w.N, w.C)).astype(np.float32)
    plan = fdl.make_plan(rm.token_region, rm.req_tok_off, rm.n_regions)
    dims = fdl.dims(w.C, w.D, w.H, w.dh, w.F)
    params_gpu = {k: v.cuda() for k, v in params.items()}
    return Case(w, rm, oracle_layout(w), params, params_gpu, inp, cond, kc, vc, vcache, plan, dims)


def run_gpu(case: Case, eps: np.ndarray, x_cur: np.ndarray, x_prev: np.ndarray, eta: float = 0.0,
            max_skip: int = 0, skip_mode: int = fdl.FD_SKIP_FREEZE, state: Optional[fdl.SparseStep] = None,
            signal: str = "delta", importance_block: Optional[int] = None):
    """One step through the C ABI; returns host copies of every output and the step object."""
    w = case.w
    st = state
    if st is None:
        st = fdl.SparseStep(case.plan, case.dims, case.params_gpu, w.L, k_cache=case.k_cache.cuda(),
                            v_cache=case.v_cache.cuda())
        st.vcache.copy_(torch.from_numpy(case.vcache))
    x = torch.from_numpy(np.ascontiguousarray(x_cur)).cuda()
    xp = torch.from_numpy(np.ascontiguousarray(x_prev)).cuda()
    st.step(x, xp, torch.from_numpy(np.asarray(eps, np.float64)).cuda(),
            torch.from_numpy(wl.dt_per_request(w)).cuda(), case.cond.cuda(), eta=eta, max_skip=max_skip,
            skip_mode=skip_mode, signal=signal, importance_block=importance_block)
    torch.cuda.synchronize()
    M = int(st.m.item())
    return dict(score=st.score.cpu().numpy(), active=st.active.cpu().numpy().astype(bool),
                importance=st.importance.cpu().numpy(), r_bar=st.r_bar.cpu().numpy(),
                delta=st.delta.cpu().numpy(),
                idx=st.idx[:M].cpu().numpy(), cu_q=st.cu_q.cpu().numpy(), M=M, x=x.cpu().numpy(),
                vcache=st.vcache.cpu().numpy(), h=st.h[:M].cpu().numpy(), v=st.v[:M].cpu().numpy(),
                s_tilde=st.s_tilde.cpu().numpy(), skip_run=st.skip_run.cpu().numpy()), st


def oracle_caches(case: Case) -> (List[np.ndarray], List[np.ndarray]):
    kc = [case.k_cache[l].to(torch.float64).numpy() for l in range(case.w.L)]
    vc = [case.v_cache[l].to(torch.float64).numpy() for l in range(case.w.L)]
    return kc, vc


def run_oracle(case: Case, eps: np.ndarray, x_cur: np.ndarray, x_prev: np.ndarray, eta: float = 0.0,
               max_skip: int = 0, skip_mode: int = orc.FREEZE, gate: Optional[orc.GateState] = None,
               caches=None, vcache: Optional[np.ndarray] = None, sample_rows=None, signal: str = "delta",
               importance_block: Optional[int] = None, importance_regions=None):
    w = case.w
    p64 = params_f64(case.params)
    kc, vc = caches if caches is not None else oracle_caches(case)
    out = orc.sparse_step(case.layout, p64, w.H, case.cond.numpy().astype(np.float64), x_cur, x_prev,
                          gate or orc.GateState.fresh(w.R), np.asarray(eps, np.float64), eta, max_skip, kc, vc,
                          case.vcache if vcache is None else vcache, wl.dt_per_request(w), skip_mode,
                          sample_rows=sample_rows, signal=signal, importance_block=importance_block,
                          importance_regions=importance_regions)
    out["k_cache"], out["v_cache"] = kc, vc
    return out


def compare_step(case: Case, g: dict, o: dict, x_cur: np.ndarray, gpu_state: fdl.SparseStep,
                 k_in: Optional[torch.Tensor] = None, v_in: Optional[torch.Tensor] = None,
                 skip_mode: int = orc.FREEZE, tol: float = TOL, check_score: bool = True) -> dict:
    """Bit-exact checks on the integer/gate outputs and skipped rows; normwise
    tolerance on the floating-point outputs.  Returns the measured errors.
    check_score=False when the gate ran on a signal other than the region score."""
    w = case.w
    if check_score:
        np.testing.assert_allclose(g["score"], o["score"], rtol=1e-12, atol=0)
    np.testing.assert_array_equal(g["active"], o["active"])
    np.testing.assert_array_equal(g["idx"], o["idx"])
    np.testing.assert_array_equal(g["cu_q"], o["cu_q"])
    assert g["M"] == len(o["idx"])
    rows = o["rows"]
    errs = {}
    if len(rows):
        errs["h"] = rel_err(g["h"][rows], o["h"])
        errs["v"] = rel_err(g["v"][rows], o["v"])
        toks = o["idx"][rows]
        errs["dx"] = rel_err(g["x"][toks] - x_cur[toks], o["x"][toks] - x_cur[toks])
        errs["vcache"] = rel_err(g["vcache"][toks], o["v"])
    skipped = np.nonzero(~o["active"][case.rmap.token_region])[0]
    if skip_mode == orc.FREEZE:
        np.testing.assert_array_equal(g["x"][skipped], x_cur[skipped])
    else:
        np.testing.assert_array_equal(g["x"][skipped], o["x"][skipped])
    np.testing.assert_array_equal(g["vcache"][skipped], case.vcache[skipped])
    # K/V caches: written rows near the oracle's, skipped rows untouched (bitwise)
    k_in = case.k_cache if k_in is None else k_in
    v_in = case.v_cache if v_in is None else v_in
    kerr = verr = 0.0
    for l in range(w.L):
        kg = gpu_state.k_cache[l].cpu()
        vg = gpu_state.v_cache[l].cpu()
        assert torch.equal(kg[skipped], k_in[l][skipped]), f"stale K rows changed in block {l}"
        assert torch.equal(vg[skipped], v_in[l][skipped]), f"stale V rows changed in block {l}"
        if len(o["idx"]):
            kerr = max(kerr, rel_err(kg[o["idx"]].to(torch.float64).numpy(), o["k_cache"][l][o["idx"]]))
            verr = max(verr, rel_err(vg[o["idx"]].to(torch.float64).numpy(), o["v_cache"][l][o["idx"]]))
    errs["k"], errs["v_rows"] = kerr, verr
    for k, e in errs.items():
        assert e <= tol, f"{w.name}: {k} error {e:.3e} > {tol}"
    return errs
