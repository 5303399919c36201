"""Seeded synthetic workloads for the region-sparse DiT denoising step.

This module only draws inputs: region maps, latents with a designed per-region
activity, gate thresholds placed between the designed activity groups, bf16
weights, conditioning vectors, position tables and K/V caches.  It holds none of
the method's arithmetic (no scores, gates, norms, GEMMs or updates) and is shared
by the HIP path, the tests and the benchmark.

Shapes follow the paper's workloads (image, video and audio DiTs and a packed
batch of image requests; FlashDiff evaluation, Table "models"); no dataset item
or trained weight is used: every value is drawn from a seeded generator.

Recipe (per request, per step n):
  * x_prev ~ N(0, 1) fp32 [N, C].
  * Each region r gets an amplitude a_r: "hot" regions a_r ~ U[1, 2], "cold"
    regions a_r ~ U[0.05, 0.45].  The hot set follows the workload's activity
    model (fixed count, moving band, Bernoulli, or a per-request fraction).
  * x_cur = x_prev + sigma_n * a_r * xi, xi ~ N(0, 1), sigma_n = 1 - n / steps
    (a decaying schedule).  The tiny workload instead rotates, x_cur =
    sqrt(1 - a^2) x_prev + a xi with hot a ~ U[0.9, 1.0] and cold a ~ U[0.1, 0.35],
    so that both latents are N(0, 1).
  * The designed activity of region r is E_r = E[(x_cur - x_prev)^2]; the gate
    threshold of request b is placed at the midpoint between its largest cold
    and smallest hot designed activity, normalised by the request's total
    designed activity: eps_b = (mid_b + eta) / sum_r (E_r + eta).  The realised
    activities differ from E_r by sampling noise only, far below the designed
    gap, so the realised active set is the hot set.
  * Weights ~ N(0, 0.02) rounded to bf16 (round to nearest even); biases,
    position table ~ N(0, 0.02) fp32; conditioning ~ N(0, 1) fp32.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch

HOT_RANGE = (1.0, 2.0)
COLD_RANGE = (0.05, 0.45)
TINY_HOT_RANGE = (0.9, 1.0)
TINY_COLD_RANGE = (0.1, 0.35)
WEIGHT_STD = 0.02


@dataclass(frozen=True)
class RequestShape:
    """One request's latent token grid and its region tiling.

    kind 'grid2d': dims (gy, gx), region (ry, rx), token = y * gx + x.
    kind 'grid3d': dims (t, y, x), region (rt, ry, rx), token = (t * Y + y) * X + x.
    kind 'seq':    dims (n,), region (r,), token = position.
    """

    kind: str
    dims: Tuple[int, ...]
    region: Tuple[int, ...]

    @property
    def n_tokens(self) -> int:
        return int(np.prod(self.dims))

    @property
    def region_grid(self) -> Tuple[int, ...]:
        return tuple(-(-d // r) for d, r in zip(self.dims, self.region))

    @property
    def n_regions(self) -> int:
        return int(np.prod(self.region_grid))

    def token_region(self) -> np.ndarray:
        """Local region id of every local token (int32 [n_tokens])."""
        coords = np.indices(self.dims).reshape(len(self.dims), -1)
        blocks = [c // r for c, r in zip(coords, self.region)]
        grid = self.region_grid
        rid = np.zeros(coords.shape[1], dtype=np.int64)
        for axis, blk in enumerate(blocks):
            rid = rid * grid[axis] + blk
        return rid.astype(np.int32)


@dataclass(frozen=True)
class Workload:
    name: str
    C: int              # latent channels per token
    D: int              # hidden size
    H: int              # attention heads
    dh: int             # head dim
    F: int              # MLP hidden size
    L: int              # DiT blocks
    requests: Tuple[RequestShape, ...]
    activity: str       # 'count' | 'band' | 'bernoulli' | 'frac'
    activity_args: Tuple[float, ...]
    dt: float           # Euler step h (negative: time runs from T to 0)
    steps: int          # denoising steps of the schedule
    seed: int
    description: str = ""

    @property
    def B(self) -> int:
        return len(self.requests)

    @property
    def N(self) -> int:
        return sum(r.n_tokens for r in self.requests)

    @property
    def R(self) -> int:
        return sum(r.n_regions for r in self.requests)

    def with_layers(self, L: int) -> "Workload":
        """Same workload with a different block count (parity at reduced depth)."""
        d = dict(self.__dict__)
        d["L"] = L
        return Workload(**d)


def _img(side: int, reg: int = 8) -> RequestShape:
    return RequestShape("grid2d", (side, side), (reg, reg))


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload(
        "tiny", C=16, D=64, H=4, dh=16, F=256, L=1,
        requests=(RequestShape("grid2d", (16, 16), (4, 4)),),
        activity="count", activity_args=(8,), dt=-0.02, steps=2, seed=1234,
        description="1 block, hidden 64, 4x16 heads, 16x16 tokens, 16 regions of 4x4, 8/16 active"),
    "image": Workload(
        "image", C=64, D=1536, H=24, dh=64, F=6144, L=24,
        requests=(_img(64),),
        activity="count", activity_args=(26,), dt=-0.02, steps=50, seed=1235,
        description="1024^2 image: 64x64 tokens, hidden 1536, 24x64 heads, 24 blocks, "
                    "64 regions of 8x8, 26/64 (~40%) active"),
    "video": Workload(
        "video", C=64, D=1536, H=12, dh=128, F=6144, L=30,
        requests=(RequestShape("grid3d", (21, 30, 52), (3, 6, 13)),),
        activity="band", activity_args=(), dt=-0.02, steps=50, seed=1236,
        description="21x30x52 = 32760 tokens, hidden 1536, 12x128 heads, 30 blocks, "
                    "140 regions of 3x6x13, 42/140 (30%) active in a moving band"),
    "audio": Workload(
        "audio", C=64, D=1024, H=16, dh=64, F=4096, L=24,
        requests=(RequestShape("seq", (2048,), (32,)),),
        activity="bernoulli", activity_args=(0.5,), dt=-0.01, steps=100, seed=1237,
        description="2048 tokens x 64 ch, hidden 1024, 16x64 heads, 24 blocks, "
                    "64 regions of 32, Bernoulli(0.5) active"),
    "packed": Workload(
        "packed", C=64, D=1536, H=24, dh=64, F=6144, L=24,
        requests=(_img(32), _img(32), _img(48), _img(48), _img(48), _img(64), _img(64), _img(64)),
        activity="frac", activity_args=(0.2, 0.7), dt=-0.02, steps=50, seed=1238,
        description="8 image requests (2x 512^2, 3x 768^2, 3x 1024^2) = 21248 tokens, "
                    "8x8 regions, per-request active fraction U[0.2, 0.7]"),
}


@dataclass
class RegionMap:
    """Global (request-major) token and region numbering of a workload."""

    token_region: np.ndarray   # int32 [N]: global region of each global token
    req_tok_off: np.ndarray    # int32 [B+1]: token range of each request
    req_reg_off: np.ndarray    # int32 [B+1]: region range of each request
    region_req: np.ndarray     # int32 [R]: request of each region
    n_regions: int


def region_map(w: Workload) -> RegionMap:
    toks, tok_off, reg_off = [], [0], [0]
    for rq in w.requests:
        toks.append(rq.token_region() + reg_off[-1])
        tok_off.append(tok_off[-1] + rq.n_tokens)
        reg_off.append(reg_off[-1] + rq.n_regions)
    region_req = np.repeat(np.arange(w.B, dtype=np.int32),
                           [rq.n_regions for rq in w.requests]).astype(np.int32)
    return RegionMap(np.concatenate(toks).astype(np.int32),
                     np.asarray(tok_off, np.int32), np.asarray(reg_off, np.int32),
                     region_req, reg_off[-1])


def _hot_regions(w: Workload, rmap: RegionMap, rng: np.random.Generator, step: int) -> np.ndarray:
    hot = np.zeros(rmap.n_regions, dtype=bool)
    for b, rq in enumerate(w.requests):
        lo, hi = int(rmap.req_reg_off[b]), int(rmap.req_reg_off[b + 1])
        nr = hi - lo
        if w.activity == "count":
            k = int(w.activity_args[0])
            hot[lo + rng.permutation(nr)[:k]] = True
        elif w.activity == "frac":
            f = rng.uniform(*w.activity_args)
            k = max(1, int(round(f * nr)))
            hot[lo + rng.permutation(nr)[:k]] = True
        elif w.activity == "bernoulli":
            p = float(w.activity_args[0])
            while True:
                sel = rng.random(nr) < p
                if sel.any():
                    break
            hot[lo:hi] = sel
        elif w.activity == "band":
            # A band of region columns that moves with the time block and the step:
            # per time block, one full column of regions plus one neighbour region.
            nt, ny, nx = rq.region_grid
            for tb in range(nt):
                xc = (tb + step) % nx
                for y in range(ny):
                    hot[lo + (tb * ny + y) * nx + xc] = True
                hot[lo + (tb * ny + (tb + step) % ny) * nx + (xc + 1) % nx] = True
        else:
            raise ValueError(w.activity)
    return hot


@dataclass
class StepInputs:
    x_prev: np.ndarray      # fp32 [N, C]
    x_cur: np.ndarray       # fp32 [N, C]
    hot: np.ndarray         # bool [R]: designed active set
    eps: np.ndarray         # fp64 [B]: gate threshold per request
    expected: np.ndarray    # fp64 [R]: designed activity E_r


def step_inputs(w: Workload, step: int = 0, x_prev: Optional[np.ndarray] = None,
                eta: float = 0.0, rmap: Optional[RegionMap] = None) -> StepInputs:
    """Latent pair and thresholds for denoising step `step` (see module recipe)."""
    rmap = rmap or region_map(w)
    rng = np.random.default_rng([w.seed, step])
    hot = _hot_regions(w, rmap, rng, step)
    R = rmap.n_regions
    if w.name == "tiny":
        amp = np.where(hot, rng.uniform(*TINY_HOT_RANGE, R), rng.uniform(*TINY_COLD_RANGE, R))
    else:
        amp = np.where(hot, rng.uniform(*HOT_RANGE, R), rng.uniform(*COLD_RANGE, R))
    if x_prev is None:
        x_prev = rng.standard_normal((w.N, w.C), dtype=np.float32)
    xi = rng.standard_normal((w.N, w.C), dtype=np.float32)
    a_tok = amp[rmap.token_region][:, None]
    if w.name == "tiny":
        x_cur = (np.sqrt(1.0 - a_tok ** 2) * x_prev + a_tok * xi).astype(np.float32)
        expected = 2.0 - 2.0 * np.sqrt(1.0 - amp ** 2)
    else:
        sigma = 1.0 - step / max(w.steps, 1)
        x_cur = (x_prev + sigma * a_tok * xi).astype(np.float32)
        expected = (sigma * amp) ** 2
    eps = np.zeros(w.B, dtype=np.float64)
    for b in range(w.B):
        lo, hi = int(rmap.req_reg_off[b]), int(rmap.req_reg_off[b + 1])
        e, h = expected[lo:hi], hot[lo:hi]
        if h.all():
            eps[b] = 0.0
            continue
        mid = 0.5 * (e[~h].max() + e[h].min())
        eps[b] = (mid + eta) / float(np.sum(e + eta))
    return StepInputs(np.ascontiguousarray(x_prev, dtype=np.float32), x_cur, hot, eps, expected)


# ----------------------------------------------------------------------------------
# Model parameters (random init of a DiT of the workload's shape).
# ----------------------------------------------------------------------------------

BLOCK_WEIGHTS = ("w_qkv", "w_o", "w_1", "w_2", "w_ada")
BLOCK_BIASES = ("b_qkv", "b_o", "b_1", "b_2", "b_ada")


def block_shapes(w: Workload) -> Dict[str, Tuple[int, ...]]:
    """Per-block parameter shapes; matrices are [out, in] (y = x W^T + b)."""
    D, F = w.D, w.F
    return {"w_qkv": (3 * D, D), "b_qkv": (3 * D,), "w_o": (D, D), "b_o": (D,),
            "w_1": (F, D), "b_1": (F,), "w_2": (D, F), "b_2": (D,),
            "w_ada": (6 * D, D), "b_ada": (6 * D,)}


def head_shapes(w: Workload) -> Dict[str, Tuple[int, ...]]:
    D, C = w.D, w.C
    return {"w_e": (D, C), "b_e": (D,), "w_adaf": (2 * D, D), "b_adaf": (2 * D,),
            "w_out": (C, D), "b_out": (C,), "pos": (w.N, D)}


def make_params(w: Workload, seed: Optional[int] = None, device: str = "cpu") -> Dict[str, torch.Tensor]:
    """All model parameters, stacked over blocks: w_* bf16 [L, out, in], b_* fp32 [L, out].

    Drawn block by block from one seeded torch generator on `device`, so the same
    seed and device give the same values.
    """
    seed = w.seed if seed is None else seed
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    out: Dict[str, torch.Tensor] = {}
    bs = block_shapes(w)
    for k, shp in bs.items():
        dtype = torch.bfloat16 if k.startswith("w_") else torch.float32
        out[k] = torch.empty((w.L,) + shp, dtype=dtype, device=device)
    for l in range(w.L):
        for k, shp in bs.items():
            v = torch.randn(shp, generator=g, device=device, dtype=torch.float32) * WEIGHT_STD
            out[k][l].copy_(v)   # fp32 -> bf16 copy rounds to nearest even
            del v
    for k, shp in head_shapes(w).items():
        v = torch.randn(shp, generator=g, device=device, dtype=torch.float32) * WEIGHT_STD
        out[k] = v.to(torch.bfloat16) if k.startswith("w_") else v
    return out


def make_cond(w: Workload, step: int = 0, device: str = "cpu") -> torch.Tensor:
    """Conditioning vector per request (timestep + prompt embedding), fp32 [B, D]."""
    g = torch.Generator(device=device)
    g.manual_seed(int(w.seed) * 7919 + step)
    return torch.randn((w.B, w.D), generator=g, device=device, dtype=torch.float32)


def make_kv_cache(w: Workload, seed: int = 99, device: str = "cpu", layers: Optional[int] = None
                  ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Synthetic per-block K/V caches ~ N(0, 1), bf16 [L, N, D] each (round to
    nearest even).

    Stands in for a cache filled by earlier steps when a test or timing run
    does not start from a dense warm-up step.  On the host the values come from
    numpy's PCG64 generator, one independent stream per block and tensor
    (children 2l and 2l + 1 of one seed sequence: block l's keys and values),
    drawn by a few threads at once: the 6 GB cache of the video model takes
    seconds, and the values do not depend on the thread count.  On a GPU
    device they come from torch's device generator (other values, same
    distribution: timing runs only).
    """
    L = w.L if layers is None else layers
    if device == "cpu":
        from concurrent.futures import ThreadPoolExecutor
        streams = np.random.SeedSequence([int(w.seed), 31, int(seed)]).spawn(2 * L)
        k = torch.empty((L, w.N, w.D), dtype=torch.bfloat16)
        v = torch.empty((L, w.N, w.D), dtype=torch.bfloat16)
        dst = [t for l in range(L) for t in (k[l], v[l])]

        def draw(i: int) -> None:
            a = np.random.default_rng(streams[i]).standard_normal((w.N, w.D), dtype=np.float32)
            dst[i].copy_(torch.from_numpy(a))   # fp32 -> bf16, round to nearest even

        with ThreadPoolExecutor(max_workers=8) as ex:
            list(ex.map(draw, range(2 * L)))
        return k, v
    g = torch.Generator(device=device)
    g.manual_seed(int(w.seed) * 31 + seed)
    k = torch.empty((L, w.N, w.D), dtype=torch.bfloat16, device=device)
    v = torch.empty((L, w.N, w.D), dtype=torch.bfloat16, device=device)
    for l in range(L):
        k[l].copy_(torch.randn((w.N, w.D), generator=g, device=device))
        v[l].copy_(torch.randn((w.N, w.D), generator=g, device=device))
    return k, v


def dt_per_request(w: Workload) -> np.ndarray:
    return np.full(w.B, w.dt, dtype=np.float32)


def saliency_map(shape: RequestShape, seed: int, levels: int = 4096) -> np.ndarray:
    """Synthetic saliency map of one request (uint16 [n_tokens], values in
    [0, levels)): a stand-in for the cross-attention of the prompt's salient
    tokens averaged over those tokens, which concentrates on a few objects of
    the latent.  Recipe: K ~ U{3, ..., 6} Gaussian blobs over the request's
    grid in normalised coordinates (each axis in [0, 1]), centres uniform,
    per-axis widths U[0.05, 0.25], amplitudes U[0.3, 1], plus a background
    U[0, 0.05] per token; the field is scaled so that its maximum maps to
    levels - 1 and rounded down (a quantised map)."""
    rng = np.random.default_rng(seed)
    coords = np.indices(shape.dims).reshape(len(shape.dims), -1).astype(np.float64)
    coords /= np.maximum(np.array(shape.dims, dtype=np.float64) - 1.0, 1.0)[:, None]
    field = rng.uniform(0.0, 0.05, coords.shape[1])
    for _ in range(int(rng.integers(3, 7))):
        centre = rng.uniform(0.0, 1.0, (len(shape.dims), 1))
        width = rng.uniform(0.05, 0.25, (len(shape.dims), 1))
        field += rng.uniform(0.3, 1.0) * np.exp(-0.5 * (((coords - centre) / width) ** 2).sum(axis=0))
    q = np.floor(field / field.max() * (levels - 1))
    return np.clip(q, 0, levels - 1).astype(np.uint16)


def saliency_maps(w: Workload, seed: Optional[int] = None, levels: int = 4096) -> np.ndarray:
    """saliency_map of every request of the workload, concatenated in request
    order (uint16 [N]); request b uses seed + b."""
    s = w.seed + 7 if seed is None else seed
    return np.concatenate([saliency_map(rq, s + b, levels) for b, rq in enumerate(w.requests)])
