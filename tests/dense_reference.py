"""Dense adaLN DiT forward built from torch library routines (float64, CPU).

Used only to pin the oracle: F.linear ([out, in] weights), F.layer_norm,
F.scaled_dot_product_attention, F.gelu(approximate='tanh') and F.silu are
independent implementations of the primitives the oracle writes out by hand.
Every token is computed (no gate, no cache): the dense step of the paper's
baseline policy ("full execution", Appendix, Setup and Notation).
"""
from __future__ import annotations

from typing import Dict, List

import numpy as np
import torch
import torch.nn.functional as F


def _t(a) -> torch.Tensor:
    return torch.as_tensor(np.asarray(a, dtype=np.float64))


def dense_block(h: torch.Tensor, tok_req: torch.Tensor, req_tok_off, blk: Dict[str, np.ndarray],
                cond: torch.Tensor, n_heads: int):
    """All N tokens through one block; returns (h', k, v)."""
    N, D = h.shape
    dh = D // n_heads
    mod = F.linear(F.silu(cond), _t(blk["w_ada"]), _t(blk["b_ada"]))
    sh1, sc1, g1, sh2, sc2, g2 = [m[tok_req] for m in mod.chunk(6, dim=-1)]
    a = F.layer_norm(h, (D,), eps=1e-6) * (1 + sc1) + sh1
    qkv = F.linear(a, _t(blk["w_qkv"]), _t(blk["b_qkv"]))
    q, k, v = qkv.split(D, dim=-1)
    o = torch.zeros_like(q)
    for b in range(len(req_tok_off) - 1):
        lo, hi = int(req_tok_off[b]), int(req_tok_off[b + 1])
        qh = q[lo:hi].reshape(hi - lo, n_heads, dh).transpose(0, 1).contiguous()
        kh = k[lo:hi].reshape(hi - lo, n_heads, dh).transpose(0, 1).contiguous()
        vh = v[lo:hi].reshape(hi - lo, n_heads, dh).transpose(0, 1).contiguous()
        oh = F.scaled_dot_product_attention(qh, kh, vh)
        o[lo:hi] = oh.transpose(0, 1).reshape(hi - lo, D)
    h = h + g1 * F.linear(o, _t(blk["w_o"]), _t(blk["b_o"]))
    a = F.layer_norm(h, (D,), eps=1e-6) * (1 + sc2) + sh2
    mlp = F.linear(F.gelu(F.linear(a, _t(blk["w_1"]), _t(blk["b_1"])), approximate="tanh"),
                   _t(blk["w_2"]), _t(blk["b_2"]))
    return h + g2 * mlp, k, v


def dense_velocity(x: np.ndarray, tok_req: np.ndarray, req_tok_off, params: Dict[str, np.ndarray],
                   cond: np.ndarray, n_heads: int, n_layers: int):
    """Velocity f(x) of every token and the per-block K/V of the dense pass."""
    condt = _t(cond)
    treq = torch.as_tensor(np.asarray(tok_req, dtype=np.int64))
    D = params["w_e"].shape[0]
    h = F.linear(_t(x), _t(params["w_e"]), _t(params["b_e"])) + _t(params["pos"])
    ks: List[np.ndarray] = []
    vs: List[np.ndarray] = []
    for l in range(n_layers):
        blk = {k: params[k][l] for k in ("w_qkv", "b_qkv", "w_o", "b_o", "w_1", "b_1",
                                         "w_2", "b_2", "w_ada", "b_ada")}
        h, k, v = dense_block(h, treq, req_tok_off, blk, condt, n_heads)
        ks.append(k.numpy())
        vs.append(v.numpy())
    mod = F.linear(F.silu(condt), _t(params["w_adaf"]), _t(params["b_adaf"]))
    sh, sc = [m[treq] for m in mod.chunk(2, dim=-1)]
    a = F.layer_norm(h, (D,), eps=1e-6) * (1 + sc) + sh
    vel = F.linear(a, _t(params["w_out"]), _t(params["b_out"]))
    return vel.numpy(), h.numpy(), ks, vs
