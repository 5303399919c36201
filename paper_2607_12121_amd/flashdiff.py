"""Python binding of libflashdiff.so (the region-sparse DiT step's C ABI).

Argument marshalling only: every function below passes device pointers, sizes
and torch's current HIP stream to the C entry point of the same name; all
computation runs in the library's HIP kernels.  torch provides device memory
and streams.  If the library is missing this module raises on import of the
library (there is no fallback path).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Dict, Optional, Sequence

import numpy as np
import torch

LIB_PATH = os.environ.get("FLASHDIFF_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                            "libflashdiff.so")

FD_SKIP_FREEZE = 0
FD_SKIP_REUSE_DRIFT = 1

KERNELS = {"score": 1, "select": 2, "gather": 3, "embed": 4, "adaln": 5, "ln": 6, "gemm_qkv": 7,
           "attn": 8, "gemm_o": 9, "gemm_mlp1": 10, "gemm_mlp2": 11, "final": 12, "scatter": 13,
           "importance": 14, "partition": 15}

_p = ctypes.c_void_p
_i32 = ctypes.c_int32


class FdPlan(ctypes.Structure):
    _fields_ = [("n_tokens", _i32), ("n_regions", _i32), ("n_requests", _i32),
                ("max_region_tokens", _i32), ("max_request_tokens", _i32),
                ("region_ptr", _p), ("region_tokens", _p), ("region_req", _p),
                ("token_region", _p), ("req_tok_off", _p), ("req_reg_off", _p)]


class FdDims(ctypes.Structure):
    _fields_ = [("C", _i32), ("D", _i32), ("H", _i32), ("dh", _i32), ("F", _i32)]


class FdBlockWeights(ctypes.Structure):
    _fields_ = [(n, _p) for n in ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2",
                                  "w_ada", "b_ada", "mod")]


class FdFinalWeights(ctypes.Structure):
    _fields_ = [(n, _p) for n in ("w_ada", "b_ada", "w_out", "b_out")]


class FdGate(ctypes.Structure):
    _fields_ = [("eta", ctypes.c_double), ("max_skip", _i32)]


class FlashDiffError(RuntimeError):
    pass


_lib: Optional[ctypes.CDLL] = None


def lib() -> ctypes.CDLL:
    """Load libflashdiff.so (built by paper_2607_12121_amd.build); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise FlashDiffError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_12121_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    sig = {
        "fd_last_error": ([], ctypes.c_char_p),
        "fd_version": ([], ctypes.c_char_p),
        "fd_plan_build": ([_i32, _i32, _i32, _p, _p, _p, _p, _p, _p, _p, _p], _i32),
        "fd_region_score_ws_size": ([P(FdPlan), _i32], ctypes.c_size_t),
        "fd_region_score": ([P(FdPlan), _i32, _p, _p, _p, _p, ctypes.c_size_t, _p], _i32),
        "fd_region_score_noalloc": ([P(FdPlan), _i32, _p, _p, _p, _p], _i32),
        "fd_select": ([P(FdPlan), _p, _p, FdGate, _p, _p, _p, _p, _p, _p, _p, _p], _i32),
        "fd_gather": ([P(FdPlan), _i32, _p, _p, _p, _p, _p], _i32),
        "fd_embed": ([P(FdPlan), P(FdDims), _p, _p, _p, _p, _p, _p, _p, _p], _i32),
        "fd_adaln": ([P(FdDims), _i32, _i32, _i32, _p, _p, _p, _p, _p], _i32),
        "fd_block_ws_size": ([P(FdPlan), P(FdDims)], ctypes.c_size_t),
        "fd_block_forward": ([P(FdPlan), P(FdDims), P(FdBlockWeights), _p, _p, _p, _p, _p, _p, _p, _p,
                              ctypes.c_size_t, _p], _i32),
        "fd_final": ([P(FdPlan), P(FdDims), P(FdFinalWeights), _p, _p, _p, _p, _p, _p, ctypes.c_size_t, _p],
                     _i32),
        "fd_scatter_update": ([P(FdPlan), _i32, _p, _p, _p, _p, _p, _p, _p, _i32, _p], _i32),
        "fd_importance_ws_size": ([P(FdPlan), P(FdDims)], ctypes.c_size_t),
        "fd_region_importance": ([P(FdPlan), P(FdDims), _p, ctypes.c_size_t, _p, _p, _p, _p, _p, _p, _p, _p,
                                  ctypes.c_size_t, _p], _i32),
        "fd_partition_ws_size": ([_i32, _i32], ctypes.c_size_t),
        "fd_partition": ([_i32, _p, _p, _p, _p, _p, ctypes.c_size_t, _p], _i32),
        "fd_timer_arm": ([_i32, _i32], _i32),
        "fd_timer_read": ([_p, _i32], _i32),
        "fd_timer_disarm": ([], None),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


def exported_symbols() -> Sequence[str]:
    return ("fd_last_error", "fd_version", "fd_plan_build", "fd_region_score_ws_size", "fd_region_score",
            "fd_region_score_noalloc",
            "fd_select", "fd_gather", "fd_embed", "fd_adaln", "fd_block_ws_size", "fd_block_forward", "fd_final",
            "fd_scatter_update", "fd_importance_ws_size", "fd_region_importance", "fd_partition_ws_size",
            "fd_partition", "fd_timer_arm", "fd_timer_read", "fd_timer_disarm")


def _check(name: str, status: int) -> None:
    if status != 0:
        msg = lib().fd_last_error().decode(errors="replace")
        raise FlashDiffError(f"{name} failed with status {status}: {msg}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise FlashDiffError("tensor arguments must be contiguous")
    return t.data_ptr()


_DT = {"f32": (torch.float32,), "f64": (torch.float64,), "i32": (torch.int32,), "u8": (torch.uint8,),
       "b16": (torch.bfloat16, torch.int16, torch.uint16), "bytes": None}


def _need(name: str, t: Optional[torch.Tensor], kind: str, numel: int, exact: bool = False,
          optional: bool = False) -> None:
    """Host-side check of one tensor argument before its pointer reaches the library:
    on a GPU, contiguous, of the element type the C entry point reads (`kind`;
    "b16" = any 2-byte bf16 bit pattern, "bytes" = any type) and with at least
    (or, with exact=True, exactly) `numel` elements."""
    if t is None:
        if optional:
            return
        raise FlashDiffError(f"{name} is required")
    if not t.is_cuda:
        raise FlashDiffError(f"{name} must be a device tensor")
    allowed = _DT[kind]
    if allowed is not None and t.dtype not in allowed:
        raise FlashDiffError(f"{name} must be {kind}, got {t.dtype}")
    n = t.numel() if kind != "bytes" else t.numel() * t.element_size()
    if (n != numel) if exact else (n < numel):
        raise FlashDiffError(f"{name} holds {n} elements, needs {'exactly ' if exact else ''}{numel}")


def _stream(stream: Optional[torch.cuda.Stream] = None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def version() -> str:
    return lib().fd_version().decode()


# ------------------------------------------------------------------ plan

@dataclass
class Plan:
    """Region plan uploaded to the device, with its C descriptor."""

    c: FdPlan
    tensors: Dict[str, torch.Tensor]
    host: Dict[str, np.ndarray]

    @property
    def n_tokens(self) -> int:
        return self.c.n_tokens

    @property
    def n_regions(self) -> int:
        return self.c.n_regions

    @property
    def n_requests(self) -> int:
        return self.c.n_requests


def fd_plan_build(token_region: np.ndarray, req_tok_off: np.ndarray, n_regions: int) -> Dict[str, np.ndarray]:
    """Host CSR plan (calls the C builder)."""
    tr = np.ascontiguousarray(token_region, dtype=np.int32)
    to = np.ascontiguousarray(req_tok_off, dtype=np.int32)
    N, B = len(tr), len(to) - 1
    out = {"region_ptr": np.zeros(n_regions + 1, np.int32), "region_tokens": np.zeros(N, np.int32),
           "region_req": np.zeros(n_regions, np.int32), "req_reg_off": np.zeros(B + 1, np.int32)}
    mx_r, mx_b = _i32(0), _i32(0)
    st = lib().fd_plan_build(N, n_regions, B, tr.ctypes.data, to.ctypes.data, out["region_ptr"].ctypes.data,
                             out["region_tokens"].ctypes.data, out["region_req"].ctypes.data,
                             out["req_reg_off"].ctypes.data, ctypes.addressof(mx_r), ctypes.addressof(mx_b))
    _check("fd_plan_build", st)
    out["token_region"] = tr
    out["req_tok_off"] = to
    out["max_region_tokens"] = np.int32(mx_r.value)
    out["max_request_tokens"] = np.int32(mx_b.value)
    return out


def make_plan(token_region: np.ndarray, req_tok_off: np.ndarray, n_regions: int, device="cuda") -> Plan:
    host = fd_plan_build(token_region, req_tok_off, n_regions)
    keys = ("region_ptr", "region_tokens", "region_req", "token_region", "req_tok_off", "req_reg_off")
    t = {k: torch.from_numpy(host[k]).to(device) for k in keys}
    c = FdPlan(len(host["token_region"]), n_regions, len(host["req_tok_off"]) - 1,
               int(host["max_region_tokens"]), int(host["max_request_tokens"]),
               *[t[k].data_ptr() for k in keys])
    return Plan(c, t, host)


def dims(C: int, D: int, H: int, dh: int, F: int) -> FdDims:
    return FdDims(C, D, H, dh, F)


# ------------------------------------------------------------------ entry points

def fd_region_score_ws_size(plan: Plan, C: int) -> int:
    return int(lib().fd_region_score_ws_size(ctypes.byref(plan.c), C))


def fd_region_score(plan: Plan, C: int, x_cur, x_prev, score, ws, stream=None) -> None:
    N, R = plan.n_tokens, plan.n_regions
    _need("x_cur", x_cur, "f32", N * C)
    _need("x_prev", x_prev, "f32", N * C)
    _need("score", score, "f64", R)
    _need("ws", ws, "bytes", fd_region_score_ws_size(plan, C))
    _check("fd_region_score", lib().fd_region_score(ctypes.byref(plan.c), C, _ptr(x_cur), _ptr(x_prev),
                                                    _ptr(score), _ptr(ws), ws.numel() * ws.element_size(),
                                                    _stream(stream)))


def fd_region_score_noalloc(plan: Plan, C: int, x_cur, x_prev, score, stream=None) -> None:
    """fd_region_score with the library's built-in scratch (no workspace argument)."""
    N, R = plan.n_tokens, plan.n_regions
    _need("x_cur", x_cur, "f32", N * C)
    _need("x_prev", x_prev, "f32", N * C)
    _need("score", score, "f64", R)
    _check("fd_region_score_noalloc", lib().fd_region_score_noalloc(ctypes.byref(plan.c), C, _ptr(x_cur), _ptr(x_prev),
                                                                    _ptr(score), _stream(stream)))


def fd_select(plan: Plan, score, eps, eta: float, max_skip: int, s_tilde, skip_run, prev_active, active,
              idx, cu_q, m, stream=None) -> None:
    N, R, B = plan.n_tokens, plan.n_regions, plan.n_requests
    for n_, t_, k_, c_ in (("score", score, "f64", R), ("eps", eps, "f64", B), ("s_tilde", s_tilde, "f64", R),
                           ("skip_run", skip_run, "i32", R), ("prev_active", prev_active, "u8", R),
                           ("active", active, "u8", R), ("idx", idx, "i32", N), ("cu_q", cu_q, "i32", B + 1),
                           ("m", m, "i32", 1)):
        _need(n_, t_, k_, c_)
    _check("fd_select", lib().fd_select(ctypes.byref(plan.c), _ptr(score), _ptr(eps), FdGate(eta, max_skip),
                                        _ptr(s_tilde), _ptr(skip_run), _ptr(prev_active), _ptr(active),
                                        _ptr(idx), _ptr(cu_q), _ptr(m), _stream(stream)))


def fd_gather(plan: Plan, C: int, x_cur, idx, m, xa, stream=None) -> None:
    N = plan.n_tokens
    _need("x_cur", x_cur, "f32", N * C)
    _need("idx", idx, "i32", N)
    _need("m", m, "i32", 1)
    _need("xa", xa, "b16", N * C)
    _check("fd_gather", lib().fd_gather(ctypes.byref(plan.c), C, _ptr(x_cur), _ptr(idx), _ptr(m), _ptr(xa),
                                        _stream(stream)))


def fd_embed(plan: Plan, d: FdDims, xa, w_e, b_e, pos, idx, m, h, stream=None) -> None:
    N = plan.n_tokens
    for n_, t_, k_, c_ in (("xa", xa, "b16", N * d.C), ("w_e", w_e, "b16", d.D * d.C), ("b_e", b_e, "f32", d.D),
                           ("pos", pos, "f32", N * d.D), ("idx", idx, "i32", N), ("m", m, "i32", 1),
                           ("h", h, "f32", N * d.D)):
        _need(n_, t_, k_, c_)
    _check("fd_embed", lib().fd_embed(ctypes.byref(plan.c), ctypes.byref(d), _ptr(xa), _ptr(w_e), _ptr(b_e),
                                      _ptr(pos), _ptr(idx), _ptr(m), _ptr(h), _stream(stream)))


def fd_block_ws_size(plan: Plan, d: FdDims) -> int:
    return int(lib().fd_block_ws_size(ctypes.byref(plan.c), ctypes.byref(d)))


def fd_adaln(d: FdDims, n_blocks: int, n_out: int, n_requests: int, w_ada, b_ada, cond, mod, stream=None) -> None:
    _need("w_ada", w_ada, "b16", n_blocks * n_out * d.D)
    _need("b_ada", b_ada, "f32", n_blocks * n_out)
    _need("cond", cond, "f32", n_requests * d.D)
    _need("mod", mod, "f32", n_blocks * n_requests * n_out)
    _check("fd_adaln", lib().fd_adaln(ctypes.byref(d), n_blocks, n_out, n_requests, _ptr(w_ada), _ptr(b_ada),
                                      _ptr(cond), _ptr(mod), _stream(stream)))


def block_weights(params: Dict[str, torch.Tensor], l: int, mod: Optional[torch.Tensor] = None) -> FdBlockWeights:
    """Weights of block l; `mod` ([B, 6D] fp32, from fd_adaln) replaces the block's own adaLN."""
    names = ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1", "w_2", "b_2", "w_ada", "b_ada")
    return FdBlockWeights(*[_ptr(params[n][l]) for n in names], _ptr(mod))


def final_weights(params: Dict[str, torch.Tensor]) -> FdFinalWeights:
    return FdFinalWeights(_ptr(params["w_adaf"]), _ptr(params["b_adaf"]), _ptr(params["w_out"]),
                          _ptr(params["b_out"]))


def fd_block_forward(plan: Plan, d: FdDims, w: FdBlockWeights, cond, h, idx, cu_q, m, k_cache, v_cache, ws,
                     stream=None) -> None:
    N, B = plan.n_tokens, plan.n_requests
    _need("cond", cond, "f32", B * d.D, optional=bool(w.mod))
    for n_, t_, k_, c_ in (("h", h, "f32", N * d.D), ("idx", idx, "i32", N), ("cu_q", cu_q, "i32", B + 1),
                           ("m", m, "i32", 1), ("k_cache", k_cache, "b16", N * d.D),
                           ("v_cache", v_cache, "b16", N * d.D), ("ws", ws, "bytes", fd_block_ws_size(plan, d))):
        _need(n_, t_, k_, c_)
    _check("fd_block_forward", lib().fd_block_forward(
        ctypes.byref(plan.c), ctypes.byref(d), ctypes.byref(w), _ptr(cond), _ptr(h), _ptr(idx), _ptr(cu_q),
        _ptr(m), _ptr(k_cache), _ptr(v_cache), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def fd_final(plan: Plan, d: FdDims, w: FdFinalWeights, cond, h, cu_q, m, v, ws, stream=None) -> None:
    N, B = plan.n_tokens, plan.n_requests
    for n_, t_, k_, c_ in (("cond", cond, "f32", B * d.D), ("h", h, "f32", N * d.D), ("cu_q", cu_q, "i32", B + 1),
                           ("m", m, "i32", 1), ("v", v, "f32", N * d.C), ("ws", ws, "bytes", fd_block_ws_size(plan, d))):
        _need(n_, t_, k_, c_)
    _check("fd_final", lib().fd_final(ctypes.byref(plan.c), ctypes.byref(d), ctypes.byref(w), _ptr(cond), _ptr(h),
                                      _ptr(cu_q), _ptr(m), _ptr(v), _ptr(ws), ws.numel() * ws.element_size(),
                                      _stream(stream)))


def fd_scatter_update(plan: Plan, C: int, x, v, idx, m, dt, vcache, active, skip_mode: int, stream=None) -> None:
    N, R, B = plan.n_tokens, plan.n_regions, plan.n_requests
    for n_, t_, k_, c_ in (("x", x, "f32", N * C), ("v", v, "f32", N * C), ("idx", idx, "i32", 1), ("m", m, "i32", 1),
                           ("dt", dt, "f32", B), ("vcache", vcache, "f32", N * C), ("active", active, "u8", R)):
        _need(n_, t_, k_, c_)
    _check("fd_scatter_update", lib().fd_scatter_update(ctypes.byref(plan.c), C, _ptr(x), _ptr(v), _ptr(idx),
                                                        _ptr(m), _ptr(dt), _ptr(vcache), _ptr(active),
                                                        skip_mode, _stream(stream)))


def fd_importance_ws_size(plan: Plan, d: FdDims) -> int:
    return int(lib().fd_importance_ws_size(ctypes.byref(plan.c), ctypes.byref(d)))


def fd_region_importance(plan: Plan, d: FdDims, block_ws, k_cache, idx, m, active, r_bar, delta, importance, ws,
                         stream=None) -> None:
    N, R = plan.n_tokens, plan.n_regions
    for n_, t_, k_, c_ in (("block_ws", block_ws, "bytes", fd_block_ws_size(plan, d)),
                           ("k_cache", k_cache, "b16", N * d.D), ("idx", idx, "i32", N), ("m", m, "i32", 1),
                           ("active", active, "u8", R), ("r_bar", r_bar, "f64", R), ("delta", delta, "f64", R),
                           ("ws", ws, "bytes", fd_importance_ws_size(plan, d))):
        _need(n_, t_, k_, c_)
    _need("importance", importance, "f64", R, optional=True)
    _check("fd_region_importance", lib().fd_region_importance(
        ctypes.byref(plan.c), ctypes.byref(d), _ptr(block_ws), block_ws.numel() * block_ws.element_size(),
        _ptr(k_cache), _ptr(idx), _ptr(m), _ptr(active), _ptr(r_bar), _ptr(delta), _ptr(importance), _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def fd_partition_ws_size(n_tokens: int, n_requests: int) -> int:
    return int(lib().fd_partition_ws_size(n_tokens, n_requests))


def fd_partition(req_tok_off, req_reg_off, saliency, token_region, ws, stream=None) -> None:
    """Patch partitioner.  req_tok_off, req_reg_off: host int sequences [B+1];
    saliency: device 2-byte tensor [N] holding uint16 values; token_region:
    device int32 [N] (output); ws: device bytes of fd_partition_ws_size(N, B)."""
    to = np.ascontiguousarray(req_tok_off, dtype=np.int32)
    ro = np.ascontiguousarray(req_reg_off, dtype=np.int32)
    if to.shape != ro.shape or to.ndim != 1 or len(to) < 2:
        raise FlashDiffError("req_tok_off and req_reg_off must both have B + 1 entries")
    if saliency.element_size() != 2 or token_region.dtype != torch.int32:
        raise FlashDiffError("saliency must hold 16-bit values and token_region int32")
    n = int(to[-1])
    _need("saliency", saliency, "bytes", 2 * n, exact=True)
    _need("token_region", token_region, "i32", n, exact=True)
    _need("ws", ws, "bytes", fd_partition_ws_size(n, len(to) - 1))
    _check("fd_partition", lib().fd_partition(len(to) - 1, to.ctypes.data, ro.ctypes.data, _ptr(saliency),
                                              _ptr(token_region), _ptr(ws), ws.numel() * ws.element_size(),
                                              _stream(stream)))


def partition(saliency: torch.Tensor, req_tok_off, req_reg_off, stream=None) -> torch.Tensor:
    """fd_partition with its output and workspace allocated here: the global
    region id of every token (device int32 [N])."""
    N, B = int(saliency.numel()), len(req_tok_off) - 1
    out = torch.empty(N, dtype=torch.int32, device=saliency.device)
    ws = torch.empty(max(fd_partition_ws_size(N, B), 256), dtype=torch.uint8, device=saliency.device)
    if stream is not None:
        # the buffers come from the current stream's pool and the saliency may still be
        # written there: the launch stream waits for that work, and both buffers are
        # marked as used on it (ws is freed here while the kernel may still run)
        stream.wait_stream(torch.cuda.current_stream())
    fd_partition(req_tok_off, req_reg_off, saliency, out, ws, stream)
    if stream is not None:
        ws.record_stream(stream)
        out.record_stream(stream)
    return out


def fd_timer_arm(kernel: str, capacity: int) -> None:
    _check("fd_timer_arm", lib().fd_timer_arm(KERNELS[kernel], capacity))


def fd_timer_read(capacity: int) -> np.ndarray:
    out = np.zeros(capacity, np.float32)
    n = lib().fd_timer_read(out.ctypes.data, capacity)
    return out[:n]


def fd_timer_disarm() -> None:
    lib().fd_timer_disarm()


# ------------------------------------------------------------------ step state

class SparseStep:
    """Device buffers of one batch and the call sequence of one region-sparse step.

    Holds the plan, model parameters (device tensors from workloads.make_params),
    per-block K/V caches, the gate state and the row workspaces; `step()` issues
    fd_region_score, fd_select, fd_gather, fd_embed, fd_adaln (the modulation of
    all L blocks in one pass), L x fd_block_forward, fd_final and
    fd_scatter_update on the current stream.  With the importance signal the
    gate thresholds `delta` (carried from the previous step) instead of the
    region score, and fd_region_importance runs after the chosen block.
    """

    def __init__(self, plan: Plan, d: FdDims, params: Dict[str, torch.Tensor], n_layers: int,
                 k_cache: Optional[torch.Tensor] = None, v_cache: Optional[torch.Tensor] = None,
                 device: str = "cuda"):
        self.plan, self.d, self.params, self.L = plan, d, params, n_layers
        N, R, B, C, D = plan.n_tokens, plan.n_regions, plan.n_requests, d.C, d.D
        dev = torch.device(device)
        self.k_cache = k_cache if k_cache is not None else torch.zeros((n_layers, N, D), dtype=torch.bfloat16,
                                                                        device=dev)
        self.v_cache = v_cache if v_cache is not None else torch.zeros((n_layers, N, D), dtype=torch.bfloat16,
                                                                        device=dev)
        self.score = torch.zeros(R, dtype=torch.float64, device=dev)
        self.s_tilde = torch.zeros(R, dtype=torch.float64, device=dev)
        self.skip_run = torch.zeros(R, dtype=torch.int32, device=dev)
        self.active = torch.ones(R, dtype=torch.uint8, device=dev)
        self.all_active = torch.ones(R, dtype=torch.uint8, device=dev)
        self.idx = torch.zeros(N, dtype=torch.int32, device=dev)
        self.cu_q = torch.zeros(B + 1, dtype=torch.int32, device=dev)
        self.m = torch.zeros(1, dtype=torch.int32, device=dev)
        self.xa = torch.zeros((N, C), dtype=torch.bfloat16, device=dev)
        self.h = torch.zeros((N, D), dtype=torch.float32, device=dev)
        self.v = torch.zeros((N, C), dtype=torch.float32, device=dev)
        self.vcache = torch.zeros((N, C), dtype=torch.float32, device=dev)
        self.ws_score = torch.empty(max(fd_region_score_ws_size(plan, C), 256), dtype=torch.uint8, device=dev)
        self.ws_block = torch.empty(fd_block_ws_size(plan, d), dtype=torch.uint8, device=dev)
        self.mod = torch.zeros((n_layers, B, 6 * D), dtype=torch.float32, device=dev)
        self.block_w = [block_weights(params, l, self.mod[l]) for l in range(n_layers)]
        self.final_w = final_weights(params)
        self.r_bar = torch.zeros(R, dtype=torch.float64, device=dev)
        self.delta = torch.zeros(R, dtype=torch.float64, device=dev)
        self.importance = torch.zeros(R, dtype=torch.float64, device=dev)
        self.ws_imp = torch.empty(max(fd_importance_ws_size(plan, d), 256), dtype=torch.uint8, device=dev)

    def reset_gate(self) -> None:
        self.s_tilde.zero_()
        self.skip_run.zero_()
        self.active.fill_(1)
        self.r_bar.zero_()
        self.delta.zero_()

    def step(self, x: torch.Tensor, x_prev: torch.Tensor, eps: torch.Tensor, dt: torch.Tensor,
             cond: torch.Tensor, eta: float = 0.0, max_skip: int = 0, skip_mode: int = FD_SKIP_FREEZE,
             stateless: bool = False, stream=None, signal: str = "delta",
             importance_block: Optional[int] = None) -> None:
        """One step on the latent x (updated in place); eps fp64 [B], dt fp32 [B], cond fp32 [B, D].

        stateless=True gates on fresh scores only (every region counts as
        executed at the previous step).  signal="importance" gates on `delta`;
        importance_block (a block index) updates r_bar and delta from that
        block's self-attention for the next step."""
        p, d, C = self.plan, self.d, self.d.C
        prev = self.all_active if stateless else self.active
        if signal == "importance":
            score = self.delta
        else:
            fd_region_score(p, C, x, x_prev, self.score, self.ws_score, stream)
            score = self.score
        fd_select(p, score, eps, eta, max_skip, self.s_tilde, self.skip_run, prev, self.active,
                  self.idx, self.cu_q, self.m, stream)
        fd_gather(p, C, x, self.idx, self.m, self.xa, stream)
        fd_embed(p, d, self.xa, self.params["w_e"], self.params["b_e"], self.params["pos"], self.idx, self.m,
                 self.h, stream)
        fd_adaln(d, self.L, 6 * d.D, p.n_requests, self.params["w_ada"], self.params["b_ada"], cond, self.mod,
                 stream)
        for l in range(self.L):
            fd_block_forward(p, d, self.block_w[l], cond, self.h, self.idx, self.cu_q, self.m, self.k_cache[l],
                             self.v_cache[l], self.ws_block, stream)
            if importance_block == l:
                fd_region_importance(p, d, self.ws_block, self.k_cache[l], self.idx, self.m, self.active, self.r_bar,
                                     self.delta, self.importance, self.ws_imp, stream)
        fd_final(p, d, self.final_w, cond, self.h, self.cu_q, self.m, self.v, self.ws_block, stream)
        fd_scatter_update(p, C, x, self.v, self.idx, self.m, dt, self.vcache, self.active, skip_mode, stream)

    def capture(self, x: torch.Tensor, x_prev: torch.Tensor, eps: torch.Tensor, dt: torch.Tensor,
                cond: torch.Tensor, **kw) -> "torch.cuda.CUDAGraph":
        """Records one step on these tensors into a HIP graph (nothing runs during the
        capture); each replay() runs the step on whatever the tensors then hold, with
        the same state buffers as step().  The step makes no host round trip and no
        allocation, and no kernel keeps state from one launch to the next, so replays
        are independent of each other.  Keyword arguments are those of step() except
        `stream`."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.step(x, x_prev, eps, dt, cond, **kw)
        return g
