"""One step recorded into a HIP graph and replayed: every replay (with eager work
and synchronisations of the program between replays) matches, bit for bit, the
same step run eagerly on a second state with identical inputs."""
import numpy as np
import pytest
import torch

from paper_2607_12121_amd import flashdiff as fdl
from paper_2607_12121_amd import workloads as wl
from tests import gpu_harness as gh
from tests.helpers import small_workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    fdl.lib()


def _many_requests_workload():
    """40 requests of 64 to 512 tokens, hidden 256: the attention's schedule tables
    and its merge pass with tables, and the matrix-core adaLN."""
    rng = np.random.default_rng(40)
    reqs = tuple(wl.RequestShape("seq", (32 * int(n),), (32,)) for n in rng.integers(2, 17, size=40))
    return small_workload("audio", requests=reqs, activity="frac", activity_args=(0.2, 0.7), L=2, D=256, H=4, dh=64,
                          F=1024)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", ["image", "tiny", "many"])
def test_graph_replays_match_eager(name):
    if name == "many":
        case = gh.make_case("audio", workload=_many_requests_workload())
    else:
        case = gh.make_case(name, L=2 if name == "image" else None)
    w = case.w

    def state():
        st = fdl.SparseStep(case.plan, case.dims, case.params_gpu, w.L, k_cache=case.k_cache.cuda(),
                            v_cache=case.v_cache.cuda())
        st.vcache.copy_(torch.from_numpy(case.vcache))
        return st

    st_e, st_g = state(), state()
    dt = torch.from_numpy(wl.dt_per_request(w)).cuda()
    cond = case.cond.cuda()
    # static inputs of the graph
    x_g = torch.empty((w.N, w.C), dtype=torch.float32, device="cuda")
    xp_g = torch.empty_like(x_g)
    eps_g = torch.empty(w.B, dtype=torch.float64, device="cuda")
    graph = st_g.capture(x_g, xp_g, eps_g, dt, cond, max_skip=2, skip_mode=fdl.FD_SKIP_REUSE_DRIFT)
    for n in range(4):
        inp = wl.step_inputs(w, n, rmap=case.rmap)
        eps = torch.from_numpy(inp.eps if n else np.zeros(w.B)).cuda()
        x_e = torch.from_numpy(inp.x_cur).cuda()
        xp_e = torch.from_numpy(inp.x_prev).cuda()
        x_g.copy_(x_e)
        xp_g.copy_(xp_e)
        eps_g.copy_(eps)
        st_e.step(x_e, xp_e, eps, dt, cond, max_skip=2, skip_mode=fdl.FD_SKIP_REUSE_DRIFT)
        torch.cuda.synchronize()
        _ = (torch.randn(1 << 16, device="cuda") * 2).sum().item()   # eager work between replays
        graph.replay()
        torch.cuda.synchronize()
        M = int(st_e.m.item())
        assert int(st_g.m.item()) == M
        for a, b, what in ((x_g, x_e, "latent"), (st_g.active, st_e.active, "mask"), (st_g.idx[:M], st_e.idx[:M], "idx"),
                           (st_g.h[:M], st_e.h[:M], "h"), (st_g.v[:M], st_e.v[:M], "v"),
                           (st_g.vcache, st_e.vcache, "drift"), (st_g.skip_run, st_e.skip_run, "skip runs"),
                           (st_g.k_cache, st_e.k_cache, "K cache"), (st_g.v_cache, st_e.v_cache, "V cache")):
            assert torch.equal(a, b), f"{name} replay {n}: {what} differs from the eager step"
        gh.say(f"{name} replay {n}: M={M}, every output equal to the eager step")
