"""The allocation-free entry point pd_denoiser_forward_static against
pd_denoiser_forward, through the C ABI: two calls in a row (the second with a
smaller batch, so the static scratch holds the first call's rows), for the MLP
that uses the scratch and for the two models that do not."""
import numpy as np
import pytest
import torch

import paper_2305_16317_amd as pd
import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pd.load()


def _rel(a, b):
    a = np.asarray(a, np.float64); b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


CASES = {
    # the policy network: 300 rows use 300 * 2 * 1024 of the 2^20 floats
    "mlp": (W.ModelSpec("mlp", (16, 10), width=1024), W.ScheduleSpec("ddpm", 100, 100), (300, 37)),
    "conv": (W.ModelSpec("conv1x1", (4, 8, 12), width=320), W.ScheduleSpec("ddpm", 1000, 1000),
             (9, 2)),
    "gmm": (W.ModelSpec("gmm2d", (2,)), W.ScheduleSpec("ddpm", 100, 100), (5000, 3)),
}


@pytest.mark.parametrize("name", list(CASES))
def test_static_forward_matches_forward(name):
    model, sch, sizes = CASES[name]
    wl = W.Workload("t", sch, model, p=8, tau=0.1)
    sched, den = pd.from_workload(wl, W.make_weights(model))
    rng = np.random.default_rng(17)
    for M in sizes:
        print(f"case {name} M={M}", flush=True)
        x = torch.from_numpy(rng.standard_normal((M, model.D)).astype(np.float32)).cuda()
        n = torch.from_numpy(rng.integers(0, sch.T_train, M).astype(np.int32)).cuda()
        ref = torch.full((M, model.D), np.nan, device="cuda")
        got = torch.full((M, model.D), np.nan, device="cuda")
        pd.pd_denoiser_forward(den, x, n, ref)
        torch.cuda.synchronize()
        pd.pd_denoiser_forward_static(den, x, n, got)
        torch.cuda.synchronize()
        g, r = got.cpu().numpy(), ref.cpu().numpy()
        assert np.isfinite(g).all()
        assert _rel(g, r) <= 1e-5, (M, _rel(g, r))
        # the same kernels on the same inputs: the same bits
        assert np.array_equal(g.view(np.uint32), r.view(np.uint32)), M


def test_static_forward_rejects_rows_beyond_the_scratch():
    model, sch, _ = CASES["mlp"]
    wl = W.Workload("t", sch, model, p=8, tau=0.1)
    sched, den = pd.from_workload(wl, W.make_weights(model))
    M = 513                                          # 513 * 2 * 1024 > 2^20
    x = torch.zeros((M, model.D), device="cuda")
    n = torch.zeros(M, dtype=torch.int32, device="cuda")
    e = torch.full((M, model.D), 7.0, device="cuda")
    with pytest.raises(pd.PdError) as err:
        pd.pd_denoiser_forward_static(den, x, n, e)
    assert err.value.code == pd.PD_ERR_INVALID_ARG and "static scratch" in str(err.value)
    torch.cuda.synchronize()
    assert torch.all(e == 7.0)                       # nothing was launched
