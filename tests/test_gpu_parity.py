"""Device path vs oracle, element by element on the same seeded inputs.

Bars: bit-exact for integers (iteration counts, strides, evaluation counts);
relative L2 <= 1e-5 for float32 results, over every element of the sample
(full-size samples against the oracle's stored float32 arrays); the
generated normals equal the
oracle's up to a handful of one-ulp roundings (Box-Muller runs in double on
both sides with different libm implementations, then rounds once to float).
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import paper_2305_16317_amd as pd
import workloads as W
from oracle import Problem, denoisers, philox, schedule

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
REL_F32 = 1e-5


def _dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device="cuda", dtype=dtype) if dtype else t.cuda()


def _rel(a, b):
    a = np.asarray(a, np.float64); b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pd.load()


# ------------------------------------------------------------------ normals
@pytest.mark.parametrize("seed,stream,count", [(0, 0, 1), (0, 0, 7), (3, 1, 4096),
                                               (1 << 33, 1, 1_000_003), (12345, 0, 36_864)])
def test_normals_match_oracle(seed, stream, count):
    out = torch.empty(count, device="cuda")
    pd.pd_normals(seed, stream, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    ref = philox.normals(seed, stream, count)
    diff = got.view(np.int32).astype(np.int64) - ref.view(np.int32).astype(np.int64)
    assert np.abs(diff).max() <= 1
    assert np.count_nonzero(diff) <= max(2, count // 1_000_000 + 2)


# ------------------------------------------------------------------ denoisers
def _forward(wl, weights, x, n):
    sched, den = pd.from_workload(wl, weights)
    M = x.shape[0]
    eps = torch.empty((M, wl.model.D), device="cuda")
    pd.pd_denoiser_forward(den, _dev(x.reshape(M, -1)), _dev(n, torch.int32), eps)
    torch.cuda.synchronize()
    return eps.cpu().numpy()


def _oracle_eps(wl, weights, x, n, bf16=None):
    tb = schedule.from_spec(wl.schedule)
    f = denoisers.Denoiser(wl.model, weights, tb.alphabar, np.float32, bf16)
    return f(x.reshape(x.shape[0], -1) if wl.model.kind != "conv1x1" else x, n).reshape(x.shape[0], -1)


def _wl(kind, shape, width=0, T=100, cond=0, dtype="f32", seed=1):
    sch = W.ScheduleSpec("ddpm", T, T)
    m = W.ModelSpec(kind, tuple(shape), width=width, cond_dim=cond, guidance=7.5,
                    dtype=dtype, weight_seed=seed, cond_seed=seed + 1)
    return W.Workload("t", sch, m, p=8, tau=0.1)


@pytest.mark.parametrize("M", [1, 5, 1000])
def test_gmm_forward(M):
    wl = W.WORKLOADS["gmm2d_ddpm100"]
    w = W.make_weights(wl.model)
    rng = np.random.default_rng(M)
    x = (rng.standard_normal((M, 2)) * 3).astype(np.float32)
    n = rng.integers(0, 100, M).astype(np.int32)
    got = _forward(wl, w, x, n)
    ref = _oracle_eps(wl, w, x, n)
    assert _rel(got, ref) <= REL_F32
    assert np.allclose(got, ref, rtol=1e-4, atol=1e-5)


@pytest.mark.parametrize("shape,width,M", [((4, 3), 32, 3), ((4, 3), 32, 37), ((16, 10), 1024, 100),
                                           ((16, 10), 1024, 1), ((4, 5), 40, 50), ((2, 2), 4, 17)])
def test_mlp_forward(shape, width, M):
    wl = _wl("mlp", shape, width)
    w = W.make_weights(wl.model)
    rng = np.random.default_rng(M)
    x = rng.standard_normal((M, int(np.prod(shape)))).astype(np.float32)
    n = rng.integers(0, 100, M).astype(np.int32)
    got = _forward(wl, w, x, n)
    ref = _oracle_eps(wl, w, x, n)
    assert _rel(got, ref) <= REL_F32


@pytest.mark.parametrize("shape,width,M,cond", [
    ((4, 8, 8), 32, 3, 0),        # two full pixel tiles per row
    ((4, 6, 7), 64, 5, 0),        # ragged last tile (42 pixels)
    ((4, 5, 5), 128, 2, 0),
    ((4, 7, 9), 96, 3, 0),        # odd number of 32-feature blocks: the halves own 2 and 1
    ((4, 1, 3), 64, 9, 0),        # three pixels: one tile per row, 29 idle lanes
    ((4, 16, 16), 320, 7, 0),     # production width, 8 tiles per row, idle waves
    ((4, 96, 96), 320, 2, 0),     # production shape
    ((4, 6, 6), 64, 3, 24),       # classifier-free guidance, w = 7.5
])
def test_conv1x1_forward(shape, width, M, cond):
    wl = _wl("conv1x1", shape, width, T=1000, cond=cond)
    w = W.make_weights(wl.model)
    rng = np.random.default_rng(M + width)
    x = rng.standard_normal((M,) + shape).astype(np.float32)
    n = rng.integers(0, 1000, M).astype(np.int32)
    got = _forward(wl, w, x, n)
    ref = _oracle_eps(wl, w, x, n)
    assert _rel(got, ref) <= REL_F32


@pytest.mark.parametrize("w1_scale,w2_scale", [(1, 1e-6), (1, 1e-3), (1, 1e2), (100, 1e3)])
def test_conv1x1_fp32_hidden_scales(w1_scale, w2_scale):
    """Hidden activations far below fp16's range (W2 scaled down: layer-3
    inputs near 1e-6) and far above it (W1 and W2 scaled up: layer-3 inputs
    near 1e5): the per-tile power-of-two scale keeps the split products as
    accurate as float32 against a float64 evaluation."""
    wl = _wl("conv1x1", (4, 16, 16), 320, T=1000)
    w = dict(W.make_weights(wl.model))
    w["W1"] = (w["W1"].astype(np.float64) * w1_scale).astype(np.float32)
    w["W2"] = (w["W2"].astype(np.float64) * w2_scale).astype(np.float32)
    rng = np.random.default_rng(11)
    x = rng.standard_normal((3, 4, 16, 16)).astype(np.float32)
    n = rng.integers(0, 1000, 3).astype(np.int32)
    got = _forward(wl, w, x, n)
    tb = schedule.from_spec(wl.schedule)
    ref64 = denoisers.Denoiser(wl.model, w, tb.alphabar, np.float64, False)(x.astype(np.float64), n)
    ref64 = ref64.reshape(3, -1)
    e_dev, e_32 = _rel(got, ref64), _rel(_oracle_eps(wl, w, x, n), ref64)
    assert np.isfinite(got).all()
    assert e_dev <= max(2 * e_32, 1e-7), (e_dev, e_32)


def test_conv1x1_fp32_rejects_weights_beyond_fp16():
    """A weight the two-part fp16 split cannot hold fails creation."""
    wl = _wl("conv1x1", (4, 8, 8), 32, T=1000)
    w = dict(W.make_weights(wl.model))
    w["W3"] = w["W3"].copy()
    w["W3"][0, 0] = 1e5
    with pytest.raises(pd.PdError) as e:
        pd.from_workload(wl, w)
    assert e.value.code == pd.PD_ERR_UNSUPPORTED


@pytest.mark.parametrize("scale", [1.0, 1e3, 1e-3])
def test_conv1x1_forward_is_fp32_accurate(scale):
    """The fp32 network runs on fp16 matrix cores with each operand split into
    an fp16 part and a scaled fp16 remainder: against a float64 evaluation it
    must be at least as accurate as a plain float32 one, at any input scale."""
    wl = _wl("conv1x1", (4, 16, 16), 320, T=1000)
    w = W.make_weights(wl.model)
    rng = np.random.default_rng(7)
    x = (rng.standard_normal((3, 4, 16, 16)) * scale).astype(np.float32)
    n = rng.integers(0, 1000, 3).astype(np.int32)
    got = _forward(wl, w, x, n)
    tb = schedule.from_spec(wl.schedule)
    ref64 = denoisers.Denoiser(wl.model, w, tb.alphabar, np.float64, False)(x.astype(np.float64), n)
    ref64 = ref64.reshape(3, -1)
    ref32 = _oracle_eps(wl, w, x, n)
    e_dev, e_32 = _rel(got, ref64), _rel(ref32, ref64)
    assert e_dev <= max(2 * e_32, 1e-7), (e_dev, e_32)


@pytest.mark.parametrize("shape,width,M,cond", [
    ((4, 8, 8), 32, 3, 0),
    ((4, 6, 7), 64, 5, 0),        # ragged last tile
    ((4, 16, 16), 320, 3, 0),     # production width
    ((4, 96, 96), 320, 2, 768),   # production shape with guidance, 768-d condition
    ((4, 6, 6), 128, 3, 24),
    ((4, 7, 9), 96, 3, 0),
])
def test_conv1x1_bf16_forward(shape, width, M, cond):
    """bf16 operands, fp32 accumulation: against the oracle's bf16-operand mode
    the only differences are summation order and the rare activation that
    rounds to the neighbouring bf16 value; against float32 it is ~1e-3."""
    wl = _wl("conv1x1", shape, width, T=1000, cond=cond, dtype="bf16")
    w = W.make_weights(wl.model)
    rng = np.random.default_rng(M + width + cond)
    x = rng.standard_normal((M,) + shape).astype(np.float32)
    n = rng.integers(0, 1000, M).astype(np.int32)
    got = _forward(wl, w, x, n)
    ref = _oracle_eps(wl, w, x, n)                     # bf16-operand oracle
    ref32 = _oracle_eps(wl, w, x, n, bf16=False)
    assert _rel(got, ref) <= 1e-3, _rel(got, ref)
    assert _rel(got, ref32) <= 2e-2, _rel(got, ref32)


def test_mlp_forward_chunks_and_concurrent_streams():
    """pd_denoiser_forward allocates nothing: the MLP runs through the
    denoiser's own scratch, 1024 rows at a time.  2500 rows span three chunks;
    two calls enqueued on two streams share the scratch in turn and both match
    the oracle."""
    wl = _wl("mlp", (4, 3), 32)
    w = W.make_weights(wl.model)
    sched, den = pd.from_workload(wl, w)
    rng = np.random.default_rng(3)
    xs = [rng.standard_normal((M, 12)).astype(np.float32) for M in (2500, 1100)]
    ns = [rng.integers(0, 100, x.shape[0]).astype(np.int32) for x in xs]
    outs = [torch.empty((x.shape[0], 12), device="cuda") for x in xs]
    xd = [_dev(x) for x in xs]
    nd = [_dev(n, torch.int32) for n in ns]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    torch.cuda.synchronize()
    for x, n, o, st in zip(xd, nd, outs, streams):
        pd.pd_denoiser_forward(den, x, n, o, stream=st)
    torch.cuda.synchronize()
    for x, n, o in zip(xs, ns, outs):
        assert _rel(o.cpu().numpy(), _oracle_eps(wl, w, x, n)) <= REL_F32


def test_forward_empty_batch_is_noop():
    wl = _wl("conv1x1", (4, 8, 8), 32, T=10)
    sched, den = pd.from_workload(wl, W.make_weights(wl.model))
    e = torch.full((1, 256), 7.0, device="cuda")
    pd.pd_denoiser_forward(den, torch.empty((0, 256), device="cuda"),
                           torch.empty(0, dtype=torch.int32, device="cuda"), e)
    torch.cuda.synchronize()
    assert torch.all(e == 7.0)


# ------------------------------------------------------------------ samplers
def _run(wl, weights, sampler="picard", p=None, tau=None, workspace=None, seed=None,
         tol_offset=0, rule="relaxed"):
    sched, den = pd.from_workload(wl, weights, tol_offset, rule)
    x = torch.empty(wl.batch * wl.model.D, device="cuda")
    seed = wl.noise_seed if seed is None else seed
    if sampler == "picard":
        st = pd.pd_sample_picard(sched, den, wl.p if p is None else p,
                                 wl.tau if tau is None else tau, seed, wl.batch,
                                 wl.model.sample_shape, x, workspace=workspace)
    else:
        st = pd.pd_sample_sequential(sched, den, seed, wl.batch, wl.model.sample_shape, x,
                                     workspace=workspace)
    torch.cuda.synchronize()
    return x.cpu().numpy().reshape(wl.batch, -1), st


SMALL = {
    "gmm_full": lambda: W.WORKLOADS["gmm2d_ddpm100"],
    "gmm_p7_b3": lambda: W.small_variant("gmm2d_ddpm100", p=7, batch=3),
    # too large for the single-workgroup loop: runs the general kernels
    "gmm_b48_general": lambda: W.small_variant("gmm2d_ddpm100", p=100, batch=48),
    # component counts past the register-held means (16) and between 8 and 16
    "gmm_k12": lambda: W.small_variant("gmm2d_ddpm100", p=20, batch=2, n_components=12),
    "gmm_k40": lambda: W.small_variant("gmm2d_ddpm100", p=33, batch=5, n_components=40),
    # the fused loop's wave-per-column running sums: two columns per wave and
    # one ragged run of rows; one column per wave and two full runs of 64
    "gmm_wave_b2": lambda: W.small_variant("gmm2d_ddpm100", p=40, batch=2),
    "gmm_wave_p128": lambda: W.small_variant("gmm2d_ddpm100", T=200, p=128, batch=1),
    "mlp_full": lambda: W.WORKLOADS["policy_mlp_ddpm100"],
    "mlp_small": lambda: W.small_variant("policy_mlp_ddpm100", T=30, p=9, shape=(4, 3), width=32, batch=2),
    # eight samples sharing the window: 40-row layer launches, any-of-batch strides
    "mlp_b8": lambda: W.small_variant("policy_mlp_ddpm100", T=40, p=5, shape=(8, 6), width=64, batch=8),
    "conv_ddpm": lambda: W.small_variant("latent_ddpm1000_p64", T=40, p=16, shape=(4, 16, 16), width=64),
    "conv_w96": lambda: W.small_variant("latent_ddpm1000_p64", T=30, p=12, shape=(4, 9, 10), width=96),
    "conv_ddpm_w320": lambda: W.small_variant("latent_ddpm1000_p64", T=60, p=32, shape=(4, 8, 12), width=320),
    "conv_ddim_b3": lambda: W.small_variant("latent_ddim200_b4", T=30, p=8, shape=(4, 6, 7), width=32, batch=3),
    "conv_p128": lambda: W.small_variant("latent_ddpm1000_p64", T=200, p=128, shape=(4, 4, 8), width=32),
    "conv_p_clamped": lambda: W.small_variant("latent_ddpm1000_p64", T=20, p=500, shape=(4, 4, 8), width=32),
    # degenerate and extreme shapes: one step; the shortest DDPM chain; DDIM
    # with noise; the largest window with several samples (conv and mlp)
    "conv_T1": lambda: W.Workload("t1", W.ScheduleSpec("ddim", 10, 1),
                                  W.ModelSpec("conv1x1", (4, 4, 8), width=32), p=4, tau=0.1),
    "gmm_T2": lambda: W.Workload("t2", W.ScheduleSpec("ddpm", 2, 2), W.ModelSpec("gmm2d", (2,)),
                                 p=4, tau=0.1, batch=3),
    # the mixture loop drawing its own prior without noise (DDIM) and with it
    # (DDIM, eta > 0), on the wave-per-column running sums
    "gmm_ddim": lambda: W.Workload("gmm_ddim", W.ScheduleSpec("ddim", 100, 50),
                                   W.ModelSpec("gmm2d", (2,)), p=50, tau=0.1),
    "gmm_ddim_eta": lambda: W.Workload("gmm_eta", W.ScheduleSpec("ddim", 200, 40, eta=0.5),
                                       W.ModelSpec("gmm2d", (2,)), p=40, tau=0.1, batch=2),
    "conv_ddim_eta": lambda: W.Workload("eta", W.ScheduleSpec("ddim", 300, 30, eta=0.7),
                                        W.ModelSpec("conv1x1", (4, 6, 7), width=32), p=8,
                                        tau=0.1, batch=2),
    "conv_p128_b3": lambda: W.small_variant("latent_ddpm1000_p64", T=160, p=128, shape=(4, 4, 8),
                                            width=32, batch=3),
    "mlp_p128_b2": lambda: W.small_variant("policy_mlp_ddpm100", T=150, p=128, shape=(4, 3),
                                           width=32, batch=2),
    "conv_cfg_f32": lambda: W.Workload("cfg", W.ScheduleSpec("ddpm", 50, 50),
                                       W.ModelSpec("conv1x1", (4, 8, 8), width=64, cond_dim=24,
                                                   guidance=7.5), p=16, tau=0.1),
    # the scan variants of the full-size latent workloads at small size: windows
    # of 33-64 points (eight waves of up to eight rows), four columns per lane,
    # several column blocks per sample (the finalize step as its own launch);
    # with noise (DDPM, as the 4x96x96 T = 1000 workload) and without (DDIM,
    # as the four-sample T = 200 workload), the latter with a ragged last block
    "conv_ddpm_p64_blocks": lambda: W.small_variant("latent_ddpm1000_p64", T=150, p=64,
                                                    shape=(4, 16, 16), width=64),
    "conv_ddpm_p48_ragged": lambda: W.small_variant("latent_ddpm1000_p64", T=100, p=48,
                                                    shape=(4, 10, 10), width=32),
    "conv_ddim_p64_b3": lambda: W.small_variant("latent_ddim200_b4", T=80, p=64,
                                                shape=(4, 10, 10), width=32, batch=3),
    "conv_ddim_p40_w320": lambda: W.small_variant("latent_ddim200_b4", T=60, p=40,
                                                  shape=(4, 8, 12), width=320, batch=2),
    # grids wide enough for the scan to share the columns out evenly over the
    # compute units: one 4x92x92 sample (249 blocks of 136 columns, the last
    # ragged) and four 4x48x48 samples (64 blocks of 144 columns each)
    "conv_even_split_b1": lambda: W.small_variant("latent_ddpm1000_p64", T=60, p=40,
                                                  shape=(4, 92, 92), width=32),
    "conv_even_split_b4": lambda: W.small_variant("latent_ddim200_b4", T=40, p=24,
                                                  shape=(4, 48, 48), width=32, batch=4),
}

BF16 = {
    "cfg_bf16_small": lambda: W.small_variant("latent_cfg_bf16_ddpm1000_p128", T=60, p=32,
                                              shape=(4, 8, 8), width=64),
    "cfg_bf16_w320": lambda: W.small_variant("latent_cfg_bf16_ddpm1000_p128", T=150, p=128,
                                             shape=(4, 8, 16), width=320),
}


@pytest.mark.parametrize("name", list(BF16))
def test_picard_bf16_matches_oracle(name):
    """bf16 denoiser: the sample is within relative L2 2e-2 of the oracle run
    with the same bf16 operand rounding; the iteration count may differ where
    a stride decision sits within rounding noise of the tolerance."""
    wl = BF16[name]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w)
    ref = Problem(wl, w, np.float32).picard()
    assert st.network_rows == st.evals_per_sample * 2
    assert _rel(got, ref.x) <= 2e-2, _rel(got, ref.x)
    assert abs(st.iters - ref.iters) <= max(1, ref.iters // 10), (st.iters, ref.iters)


@pytest.mark.parametrize("name", list(BF16))
def test_sequential_bf16_matches_oracle(name):
    """bf16 denoiser, sequential chain: within 2e-2 of the oracle run with the
    same bf16 operand rounding, and Picard with p = 1 gives it bit for bit."""
    wl = BF16[name]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w, "sequential")
    ref = Problem(wl, w, np.float32).sequential()
    assert st.evals_per_sample == wl.schedule.T and st.network_rows == 2 * wl.schedule.T
    assert _rel(got, ref) <= 2e-2, _rel(got, ref)
    one, _ = _run(wl, w, "picard", p=1)
    assert np.array_equal(one.view(np.uint32), got.view(np.uint32))


@pytest.mark.parametrize("name", list(SMALL))
def test_picard_matches_oracle(name):
    wl = SMALL[name]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w)
    pr = Problem(wl, w, np.float32)
    ref = pr.picard()
    assert (st.iters, st.trace, st.evals_per_sample) == (ref.iters, ref.trace, ref.evals)
    assert st.network_rows == ref.evals * wl.batch * (2 if wl.model.cond_dim else 1)
    assert _rel(got, ref.x) <= REL_F32, _rel(got, ref.x)


@pytest.mark.parametrize("name", ["gmm_p7_b3", "gmm_k12", "gmm_k40", "mlp_small", "conv_ddpm",
                                  "conv_ddim_b3", "conv_T1", "gmm_T2", "conv_ddim_eta"])
def test_sequential_matches_oracle(name):
    wl = SMALL[name]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w, "sequential")
    ref = Problem(wl, w, np.float32).sequential()
    assert st.iters == wl.schedule.T and st.evals_per_sample == wl.schedule.T
    assert _rel(got, ref) <= REL_F32


@pytest.mark.parametrize("name", ["gmm_p7_b3", "gmm_k40", "gmm_ddim", "gmm_ddim_eta", "mlp_small", "conv_ddpm", "conv_ddim_b3"])
def test_window_of_one_is_sequential_bitwise(name):
    wl = SMALL[name]()
    w = W.make_weights(wl.model)
    a, st = _run(wl, w, "picard", p=1)
    b, _ = _run(wl, w, "sequential")
    assert st.iters == wl.schedule.T and st.trace == [1] * wl.schedule.T
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("name", ["conv_ddpm", "mlp_b8", "mlp_full"])
def test_runs_are_deterministic_and_workspace_reuse(name):
    """Two runs are bitwise equal, and so is a run on a workspace that served
    another seed first (for the MLP this also checks that the fused last
    layer's arrival counters are back at zero after every call)."""
    wl = SMALL[name]()
    w = W.make_weights(wl.model)
    a, sa = _run(wl, w)
    b, sb = _run(wl, w)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32)) and sa == sb
    sched, den = pd.from_workload(wl, w)
    ws = pd.pd_workspace_create(sched, den, wl.p, wl.batch)
    for seed in (5, 0):
        x = torch.empty(wl.batch * wl.model.D, device="cuda")
        st = pd.pd_sample_picard(sched, den, wl.p, wl.tau, seed, wl.batch, wl.model.sample_shape,
                                 x, workspace=ws)
        torch.cuda.synchronize()
    assert np.array_equal(x.cpu().numpy().reshape(a.shape).view(np.uint32), a.view(np.uint32))
    assert st == sa


@pytest.mark.parametrize("name", ["gmm_p7_b3", "gmm_b48_general", "mlp_small", "conv_ddpm",
                                  "conv_ddim_b3"])
def test_tolerance_offset_matches_oracle(name):
    """The sigma_{t+j-1} reading of the stride test's variance index
    (tol_index_offset = -1): strides and samples as the oracle's."""
    wl = SMALL[name]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w, tol_offset=-1)
    ref = Problem(wl, w, np.float32).picard(tol_offset=-1)
    assert (st.iters, st.trace, st.evals_per_sample) == (ref.iters, ref.trace, ref.evals)
    assert _rel(got, ref.x) <= REL_F32, _rel(got, ref.x)


PROP2 = [("gmm_p7_b3", 1.0), ("gmm_p7_b3", 40.0), ("gmm_b48_general", 5.0),
         ("mlp_small", 2.0), ("mlp_small", 50.0), ("mlp_b8", 10.0), ("conv_ddpm", 20.0),
         ("conv_ddpm", 300.0), ("conv_ddim_b3", 50.0), ("conv_ddpm_p64_blocks", 200.0),
         ("conv_ddim_p64_b3", 100.0)]


@pytest.mark.parametrize("name,eps", PROP2)
def test_prop2_rule_matches_oracle(name, eps):
    """Prop. 2's stopping rule |x^{k+1} - x^k|^2 <= 4 eps^2 sigma^2 / T^2: the
    strides bit for bit and the sample within 1e-5 of the oracle's."""
    wl = SMALL[name]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w, tau=eps, rule="prop2")
    ref = Problem(wl, w, np.float32).picard(tau=eps, rule="prop2")
    assert (st.iters, st.trace, st.evals_per_sample) == (ref.iters, ref.trace, ref.evals)
    assert _rel(got, ref.x) <= REL_F32, _rel(got, ref.x)


def test_prop2_rule_is_relaxed_rule_at_matching_tau():
    """On the device as in the oracle: Prop. 2 at eps equals the relaxed rule
    at tau = 2 eps / (T sqrt D) (D = 16, T = 32: exact binary fractions)."""
    wl = W.Workload("p2", W.ScheduleSpec("ddpm", 32, 32),
                    W.ModelSpec("mlp", (4, 4), width=32, weight_seed=9), p=8, tau=0.1,
                    batch=2, noise_seed=4)
    w = W.make_weights(wl.model)
    for eps in (0.5, 4.0, 64.0):
        a, sa = _run(wl, w, tau=eps, rule="prop2")
        b, sb = _run(wl, w, tau=2.0 * eps / (32 * 4.0))
        assert sa == sb and np.array_equal(a.view(np.uint32), b.view(np.uint32)), eps


def test_infinite_tolerance_single_sweeps():
    wl = SMALL["conv_ddpm"]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w, tau=float("inf"))
    ref = Problem(wl, w, np.float32).picard(tau=float("inf"))
    assert st.trace == ref.trace
    assert _rel(got, ref.x) <= REL_F32


def test_overflowing_error_reports_numeric_error():
    """Huge but finite points (the last bias 1e20): the squared differences
    overflow float32, the error is non-finite, and the sampler returns
    PD_ERR_NUMERIC, as the oracle raises NumericError on the same input."""
    from oracle.samplers import NumericError
    wl = SMALL["conv_ddpm"]()
    w = dict(W.make_weights(wl.model))
    w["b4"] = np.full_like(w["b4"], 1e20)
    with pytest.raises(NumericError):
        Problem(wl, w, np.float32).picard()
    with pytest.raises(pd.PdError) as e:
        _run(wl, w)
    assert e.value.code == pd.PD_ERR_NUMERIC


def test_non_finite_reports_numeric_error():
    wl = SMALL["conv_ddpm"]()
    w = W.make_weights(wl.model)
    w["b4"] = w["b4"].copy()
    w["b4"][1] = np.float32(np.inf)
    with pytest.raises(pd.PdError) as e:
        _run(wl, w)
    assert e.value.code == pd.PD_ERR_NUMERIC


def test_workspace_mismatch_rejected():
    wl = SMALL["conv_ddpm"]()
    w = W.make_weights(wl.model)
    sched, den = pd.from_workload(wl, w)
    ws = pd.pd_workspace_create(sched, den, 4, 1)
    x = torch.empty(wl.model.D, device="cuda")
    with pytest.raises(pd.PdError) as e:
        pd.pd_sample_picard(sched, den, 16, 0.1, 0, 1, wl.model.sample_shape, x, workspace=ws)
    assert e.value.code == pd.PD_ERR_INVALID_ARG


# ------------------------------------------------------------ full-size workloads
def _golden(name):
    """The oracle's stored result of a full-size workload: the JSON summary
    (K, strides, evaluations, squared norm) and the complete float32 samples."""
    path = os.path.join(HERE, "golden", f"{name}.json")
    arr = os.path.join(HERE, "golden", f"{name}.npz")
    if not (os.path.exists(path) and os.path.exists(arr)):
        pytest.fail(f"{path} or its .npz missing: run tests/golden/make_golden.py {name}")
    g = json.load(open(path))
    with np.load(arr) as z:
        for key in z.files:
            g[key]["x"] = z[key]
    return g


def _check_full(got, g, tol):
    """Every element: relative L2 over the whole sample within ``tol``; the
    message names the worst element."""
    ref = np.asarray(g["x"], np.float32)
    got = np.asarray(got, np.float32).reshape(ref.shape)
    assert np.isfinite(got).all()
    rel = _rel(got, ref)
    diff = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    worst = np.unravel_index(int(np.argmax(diff)), ref.shape)
    msg = (f"rel L2 {rel:.3e} over {ref.size} values; worst element {worst}: "
           f"{got[worst]!r} vs {ref[worst]!r}")
    assert rel <= tol, msg
    n2 = float(np.sum(got.astype(np.float64) ** 2))
    assert abs(math.sqrt(n2) - math.sqrt(g["norm2"])) <= tol * math.sqrt(g["norm2"]), msg


@pytest.mark.parametrize("name", ["gmm2d_ddpm100", "policy_mlp_ddpm100", "latent_ddpm1000_p64",
                                  "latent_ddim200_b4", "policy_mlp_heun20", "latent_heun100_p32",
                                  "policy_mlp_dpm15", "latent_dpm200_p64"])
def test_full_size_picard_matches_oracle(name):
    """Every value of the sample (147,456 for the four 4x96x96 samples of the
    DDIM workload) within relative L2 1e-5 of the oracle's float32 sample;
    K, strides and evaluations bit for bit."""
    g = _golden(name)
    wl = W.WORKLOADS[name]
    got, st = _run(wl, W.make_weights(wl.model))
    gp = g["picard"]
    assert (st.iters, st.trace, st.evals_per_sample) == (gp["iters"], gp["trace"], gp["evals"])
    _check_full(got, gp, REL_F32)


@pytest.mark.parametrize("name", ["gmm2d_ddpm100", "policy_mlp_ddpm100", "latent_ddpm1000_p64",
                                  "policy_mlp_dpm15", "latent_dpm200_p64"])
def test_full_size_sequential_matches_oracle(name):
    g = _golden(name)
    wl = W.WORKLOADS[name]
    got, st = _run(wl, W.make_weights(wl.model), "sequential")
    _check_full(got, g["sequential"], REL_F32)


@pytest.mark.parametrize("name,eps", [("gmm2d_ddpm100", 1.0), ("policy_mlp_ddpm100", 1.0),
                                      ("policy_mlp_ddpm100", 10.0)])
def test_full_size_prop2_matches_oracle(name, eps):
    """Prop. 2's stopping rule at full size: strides bit for bit, every value
    of the sample within 1e-5."""
    g = _golden(name)[f"picard_prop2_eps{eps:g}"]
    wl = W.WORKLOADS[name]
    got, st = _run(wl, W.make_weights(wl.model), tau=eps, rule="prop2")
    assert (st.iters, st.trace, st.evals_per_sample) == (g["iters"], g["trace"], g["evals"])
    _check_full(got, g, REL_F32)


@pytest.mark.parametrize("name", ["latent_ddpm1000_p64", "policy_mlp_ddpm100"])
def test_full_size_tolerance_offset_matches_oracle(name):
    """The sigma^2_{t+j-1} reading of the stride test at full size."""
    g = _golden(name)["picard_tol_offset_m1"]
    wl = W.WORKLOADS[name]
    got, st = _run(wl, W.make_weights(wl.model), tol_offset=-1)
    assert (st.iters, st.trace, st.evals_per_sample) == (g["iters"], g["trace"], g["evals"])
    _check_full(got, g, REL_F32)


def test_full_size_headline_in_bench_configuration():
    """The 4x96x96 DDPM T=1000, p=64 sample run as bench.py times it: a workspace
    made once, the current torch stream, per-kernel events on, then a second
    call on the same workspace with events off; both match the oracle's
    golden (K, strides, evaluations, sampled values)."""
    name = "latent_ddpm1000_p64"
    g = _golden(name)["picard"]
    wl = W.WORKLOADS[name]
    sched, den = pd.from_workload(wl, W.make_weights(wl.model))
    ws = pd.pd_workspace_create(sched, den, wl.p, wl.batch)
    x = torch.empty(wl.batch * wl.model.D, device="cuda")
    stream = torch.cuda.current_stream()
    for timed in (True, False):
        st = pd.pd_sample_picard(sched, den, wl.p, wl.tau, wl.noise_seed, wl.batch,
                                 wl.model.sample_shape, x, workspace=ws, stream=stream,
                                 time_kernels=timed)
        torch.cuda.synchronize()
        assert (st.iters, st.trace, st.evals_per_sample) == (g["iters"], g["trace"], g["evals"])
        _check_full(x.cpu().numpy().reshape(wl.batch, -1), g, REL_F32)


def test_full_size_bf16_picard_matches_oracle():
    """Guided bf16 workload at full size (4x96x96, width 320, T=1000, p=128):
    sampled outputs and the norm within 2e-2 of the oracle run with the same
    bf16 operand rounding; the iteration count within 10% (a stride decision
    may sit within rounding noise of the tolerance)."""
    name = "latent_cfg_bf16_ddpm1000_p128"
    g = _golden(name)
    wl = W.WORKLOADS[name]
    got, st = _run(wl, W.make_weights(wl.model))
    gp = g["picard"]
    assert abs(st.iters - gp["iters"]) <= max(1, gp["iters"] // 10), (st.iters, gp["iters"])
    assert st.network_rows == st.evals_per_sample * 2
    _check_full(got, gp, 2e-2)


# ------------------------------------------------------- Heun drift (DDIM ODE)
def _heun(model, T, p, batch, tau=0.05, seed=0):
    return W.Workload("heun", W.ScheduleSpec("ddim", 10 * T, T, solver="heun"), model,
                      p=p, tau=tau, batch=batch, noise_seed=seed)


HEUN = {
    # the mixture runs the general kernels here (its fused loop is Euler only)
    "heun_gmm": lambda: _heun(W.ModelSpec("gmm2d", (2,)), 40, 12, 2),
    "heun_mlp": lambda: _heun(W.ModelSpec("mlp", (4, 3), width=32), 30, 9, 2),
    # the last layer's fused prediction over many row tiles, three samples a row group
    "heun_mlp_wide": lambda: _heun(W.ModelSpec("mlp", (4, 5), width=32), 80, 64, 3),
    "heun_conv": lambda: _heun(W.ModelSpec("conv1x1", (4, 6, 7), width=32), 24, 8, 3),
    "heun_conv_full_window": lambda: _heun(W.ModelSpec("conv1x1", (4, 8, 8), width=64), 16, 16, 1),
}


@pytest.mark.parametrize("name", list(HEUN))
def test_heun_picard_matches_oracle(name):
    wl = HEUN[name]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w)
    ref = Problem(wl, w, np.float32).picard()
    assert (st.iters, st.trace, st.evals_per_sample) == (ref.iters, ref.trace, ref.evals)
    assert st.network_rows == ref.evals * wl.batch
    assert _rel(got, ref.x) <= REL_F32, _rel(got, ref.x)


@pytest.mark.parametrize("name", ["heun_gmm", "heun_mlp", "heun_conv"])
def test_heun_sequential_matches_oracle_and_window_of_one(name):
    wl = HEUN[name]()
    w = W.make_weights(wl.model)
    seq, st = _run(wl, w, "sequential")
    T = wl.schedule.T
    assert st.evals_per_sample == 2 * T - 1
    assert _rel(seq, Problem(wl, w, np.float32).sequential()) <= REL_F32
    one, st1 = _run(wl, w, "picard", p=1)
    assert st1.iters == T and st1.evals_per_sample == 2 * T - 1
    assert np.array_equal(one.view(np.uint32), seq.view(np.uint32))


# ------------------------------------------- DPM-Solver++(2M) (ParaDPMSolver)
def _dpm(model, T, p, batch, tau=0.05, seed=0, T_train=None):
    return W.Workload("dpm", W.ScheduleSpec("ddim", T_train or 10 * T, T, solver="dpm2m"), model,
                      p=p, tau=tau, batch=batch, noise_seed=seed)


DPM = {
    # two columns: the scan's one-column-per-lane layout (the mixture's fused
    # loop is Euler only, so this runs the general kernels)
    "dpm_gmm": lambda: _dpm(W.ModelSpec("gmm2d", (2,)), 40, 12, 2),
    "dpm_mlp": lambda: _dpm(W.ModelSpec("mlp", (4, 5), width=32), 30, 9, 2),
    "dpm_conv": lambda: _dpm(W.ModelSpec("conv1x1", (4, 6, 7), width=32), 24, 8, 3),
    # several scan blocks per sample (finalize runs as its own launch)
    "dpm_conv_blocks": lambda: _dpm(W.ModelSpec("conv1x1", (4, 16, 17), width=32), 20, 7, 1),
    # 40-point window: waves hold 4 rows each, so the step before a wave's
    # first row sits in the previous wave's chunk
    "dpm_mlp_wide": lambda: _dpm(W.ModelSpec("mlp", (4, 3), width=32), 60, 40, 2, tau=0.1),
    "dpm_conv_full_window": lambda: _dpm(W.ModelSpec("conv1x1", (4, 8, 8), width=64), 16, 16, 1),
    # whole-window slides (x_{t-1} is the previous window's last point) and
    # single-point slides
    "dpm_mlp_tau_inf": lambda: _dpm(W.ModelSpec("mlp", (4, 3), width=32), 25, 6, 2,
                                    tau=float("inf")),
    "dpm_mlp_tau0": lambda: _dpm(W.ModelSpec("mlp", (4, 3), width=32), 12, 5, 1, tau=0.0),
}


@pytest.mark.parametrize("name", list(DPM))
def test_dpm_picard_matches_oracle(name):
    wl = DPM[name]()
    w = W.make_weights(wl.model)
    got, st = _run(wl, w)
    ref = Problem(wl, w, np.float32).picard()
    assert (st.iters, st.trace, st.evals_per_sample) == (ref.iters, ref.trace, ref.evals)
    assert st.network_rows == ref.evals * wl.batch
    assert _rel(got, ref.x) <= REL_F32, _rel(got, ref.x)


@pytest.mark.parametrize("name", ["dpm_gmm", "dpm_mlp", "dpm_conv"])
def test_dpm_sequential_matches_oracle_and_window_of_one(name):
    """The sequential multistep loop against the oracle; Picard with p = 1
    re-evaluates x_{t-1} each step (T - 1 extra evaluations) and must give the
    sequential sample bit for bit."""
    wl = DPM[name]()
    w = W.make_weights(wl.model)
    seq, st = _run(wl, w, "sequential")
    T = wl.schedule.T
    assert st.evals_per_sample == T
    assert _rel(seq, Problem(wl, w, np.float32).sequential()) <= REL_F32
    one, st1 = _run(wl, w, "picard", p=1)
    assert st1.iters == T and st1.evals_per_sample == 2 * T - 1
    assert np.array_equal(one.view(np.uint32), seq.view(np.uint32))


@pytest.mark.parametrize("name,table", [("dpm_conv", "DPM"), ("dpm_mlp", "DPM"),
                                        ("heun_conv", "HEUN")])
def test_multistep_and_heun_workspace_reuse(name, table):
    """A workspace reused across calls (its ring and state hold the previous
    call's end) gives each call's fresh-workspace result bit for bit."""
    wl = (DPM if table == "DPM" else HEUN)[name]()
    w = W.make_weights(wl.model)
    sched, den = pd.from_workload(wl, w)
    ws = pd.pd_workspace_create(sched, den, wl.p, wl.batch)
    x = torch.empty(wl.batch * wl.model.D, device="cuda")
    for seed in (0, 3, 0):
        ref, sr = _run(wl, w, seed=seed)
        st = pd.pd_sample_picard(sched, den, wl.p, wl.tau, seed, wl.batch, wl.model.sample_shape, x,
                                 workspace=ws)
        torch.cuda.synchronize()
        got = x.cpu().numpy().reshape(wl.batch, -1)
        assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), seed
        assert (st.iters, st.trace, st.evals_per_sample) == (sr.iters, sr.trace, sr.evals_per_sample)
        seq_ref, _ = _run(wl, w, "sequential", seed=seed)
        pd.pd_sample_sequential(sched, den, seed, wl.batch, wl.model.sample_shape, x, workspace=ws)
        torch.cuda.synchronize()
        assert np.array_equal(x.cpu().numpy().reshape(wl.batch, -1).view(np.uint32),
                              seq_ref.view(np.uint32)), seed
