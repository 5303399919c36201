"""GPU parity of the patch partitioner (fd_partition, through the C ABI) against
the oracle's recursive Otsu partition: the region of every token, bit-exact, on
the workloads' synthetic saliency maps and on the method's degenerate cases
(constant maps, few distinct values, one region, one token per region, the
limits of the entry point)."""
import numpy as np
import pytest
import torch

from oracle import flashdiff_oracle as orc
from paper_2607_12121_amd import flashdiff as fdl
from paper_2607_12121_amd import workloads as wl
from tests import gpu_harness as gh

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    fdl.lib()


def _oracle_regions(sal, tok_off, reg_off):
    out = np.empty(len(sal), np.int64)
    for b in range(len(tok_off) - 1):
        t0, t1 = tok_off[b], tok_off[b + 1]
        out[t0:t1] = reg_off[b] + orc.otsu_partition(sal[t0:t1], reg_off[b + 1] - reg_off[b])
    return out


def _gpu_regions(sal, tok_off, reg_off):
    d_sal = torch.from_numpy(np.ascontiguousarray(sal, np.uint16).view(np.int16)).cuda()
    out = fdl.partition(d_sal, tok_off, reg_off)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.int64)


def _check(label, sal, tok_off, reg_off):
    gh.say(f"partition {label}: B={len(tok_off) - 1} N={len(sal)} R={reg_off[-1]}")
    got = _gpu_regions(sal, tok_off, reg_off)
    want = _oracle_regions(sal, tok_off, reg_off)
    bad = np.nonzero(got != want)[0]
    assert len(bad) == 0, f"{label}: {len(bad)} tokens differ, first {bad[:5]} got {got[bad[:5]]} want {want[bad[:5]]}"
    return got


@pytest.mark.parametrize("name", ["tiny", "image", "audio", "video", "packed"])
def test_partition_workload_maps(name):
    """The workloads' blob-shaped saliency maps (4096 levels), every request of
    the batch partitioned into its own region count in one call; the result is
    a valid token->region map for the plan builder."""
    w = wl.WORKLOADS[name]
    rm = wl.region_map(w)
    sal = wl.saliency_maps(w)
    reg_off = np.concatenate([[0], np.cumsum([rq.n_regions for rq in w.requests])]).astype(np.int32)
    got = _check(name, sal, rm.req_tok_off, reg_off)
    plan = fdl.make_plan(got.astype(np.int32), rm.req_tok_off.astype(np.int32), int(reg_off[-1]))
    assert plan is not None
    assert np.array_equal(_gpu_regions(sal, rm.req_tok_off, reg_off), got)   # deterministic


def test_partition_full_16_bit_range():
    """Values spanning 0 .. 65535 (class sums beyond 2^32); a map of about 14000
    distinct values (that many candidate thresholds at the root)."""
    shape = wl.RequestShape("grid2d", (64, 64), (8, 8))
    sal = wl.saliency_map(shape, seed=5, levels=65536)
    assert sal.max() == 65535
    _check("16-bit image", sal, [0, 4096], [0, 64])
    many = np.random.default_rng(6).integers(0, 65536, 16000).astype(np.uint16)
    assert len(np.unique(many)) > 14000
    _check("many distinct values", many, [0, 16000], [0, 64])


def test_partition_constant_and_few_values():
    """Degenerate maps: one value (the whole request is cut by token index), two
    levels, three levels with many regions (chunk nodes below a split), and a map
    whose runs of equal values force chunks at several depths."""
    rng = np.random.default_rng(3)
    _check("constant", np.full(1000, 77, np.uint16), [0, 1000], [0, 7])
    _check("two levels", np.where(rng.random(3000) < 0.3, 65535, 0).astype(np.uint16), [0, 3000], [0, 10])
    _check("three levels", rng.choice(np.array([5, 900, 901], np.uint16), 2500), [0, 2500], [0, 32])
    sal = np.repeat(np.arange(6, dtype=np.uint16) * 1000, [700, 20, 20, 20, 20, 1220])
    _check("runs", rng.permutation(sal), [0, 2000], [0, 40])


def test_partition_region_count_limits():
    """One region; one token per region; the largest region count (1024) and
    token count (65535) per request; 64 requests in one call."""
    rng = np.random.default_rng(4)
    _check("one region", rng.integers(0, 4096, 500).astype(np.uint16), [0, 500], [0, 1])
    _check("one token", np.array([9], np.uint16), [0, 1], [0, 1])
    _check("token per region", rng.integers(0, 40, 50).astype(np.uint16), [0, 50], [0, 50])
    _check("1024 regions", rng.integers(0, 65536, 8000).astype(np.uint16), [0, 8000], [0, 1024])
    _check("65535 tokens", rng.integers(0, 300, 65535).astype(np.uint16), [0, 65535], [0, 96])
    n = rng.integers(20, 400, 64)
    r = np.minimum(rng.integers(1, 24, 64), n)
    tok_off = np.concatenate([[0], np.cumsum(n)]).astype(np.int32)
    reg_off = np.concatenate([[0], np.cumsum(r)]).astype(np.int32)
    sal = np.concatenate([rng.integers(0, int(rng.choice([2, 50, 65536])), k) for k in n]).astype(np.uint16)
    _check("64 requests", sal, tok_off, reg_off)


def test_partition_binding_rejects_mismatched_sizes():
    """The binding checks the buffers against the offsets before the call: a
    saliency map of 60 tokens with offsets [0, 61] (whose workspace size would
    still pass the library's rounded check) raises on the host, no launch."""
    sal = torch.zeros(60, dtype=torch.int16, device="cuda")
    out = torch.zeros(61, dtype=torch.int32, device="cuda")
    ws = torch.empty(max(fdl.fd_partition_ws_size(61, 1), 256), dtype=torch.uint8, device="cuda")
    with pytest.raises(fdl.FlashDiffError, match="saliency"):
        fdl.fd_partition([0, 61], [0, 4], sal, out, ws)
    with pytest.raises(fdl.FlashDiffError, match="token_region"):
        fdl.fd_partition([0, 60], [0, 4], sal, out, ws)


def test_partition_on_a_side_stream_is_ordered_after_the_current_stream():
    """partition(stream=s): the launch stream waits for the current stream's
    writes to the saliency map (issued just before, not synchronised)."""
    rq = wl.WORKLOADS["image"].requests[0]
    sal = wl.saliency_map(rq, seed=5)
    want = orc.otsu_partition(sal, rq.n_regions)
    d_sal = torch.zeros(rq.n_tokens, dtype=torch.int16, device="cuda")
    src = torch.from_numpy(sal.view(np.int16)).cuda()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    d_sal.copy_(src)                       # on the current stream
    got = fdl.partition(d_sal, [0, rq.n_tokens], [0, rq.n_regions], stream=side)
    side.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), want)
