"""CPU-side checks of the C ABI: the library loads, exports what the header
declares, validates arguments without touching a device, reports a missing
GPU, and builds schedule tables bitwise equal to the oracle's."""
import ctypes
import math
import os
import re

import numpy as np
import pytest
import torch

import paper_2305_16317_amd as pd
from oracle import schedule as osched

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "paradigms.h")


def _declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(pd_[a-z_]+)\s*\(", txt)))


def test_library_built_and_loads():
    assert os.path.exists(pd.lib_path()), "run python -m paper_2305_16317_amd.build first"
    L = pd.load()
    assert L.pd_version().decode().startswith("paradigms-gfx950")


def test_every_declared_symbol_is_exported():
    L = pd.load()
    decl = _declared()
    assert set(decl) == set(pd.EXPORTED_SYMBOLS)
    for name in decl:
        assert hasattr(L, name), name


def test_library_is_gfx950_only():
    data = open(pd.lib_path(), "rb").read()
    assert b"gfx950" in data
    assert b"gfx942" not in data and b"gfx90a" not in data


def _status(fn, *args):
    code = fn(*args)
    return code, pd.load().pd_last_error().decode()


@pytest.mark.parametrize("kw,msg", [
    (dict(kind=7), "kind"),
    (dict(T_train=1, T=1), "T_train"),
    (dict(T=0), "T must"),
    (dict(T=50), "DDPM needs"),
    (dict(kind=pd.PD_DDIM, T=300), "T_train % T"),
    (dict(beta_start=0.0), "beta"),
    (dict(beta_end=1.0), "beta"),
    (dict(beta_start=0.03), "beta"),
    (dict(beta_start=float("nan")), "beta"),
    (dict(kind=pd.PD_DDIM, T=200, eta=1.5), "eta"),
    (dict(tol_index_offset=2), "tol_index_offset"),
    (dict(kind=pd.PD_DDIM_HEUN, T=200, eta=0.5), "Heun"),
    (dict(kind=pd.PD_DDIM_HEUN, T=300), "T_train % T"),
    (dict(kind=pd.PD_DDIM_DPM2M, T=200, eta=0.3), "DPM-Solver"),
    (dict(kind=4, T=200), "kind"),
    (dict(stop_rule=2), "stop_rule"),
    (dict(stop_rule=-1), "stop_rule"),
])
def test_schedule_validation(kw, msg):
    args = dict(kind=pd.PD_DDPM, T_train=1000, T=1000, beta_start=1e-4, beta_end=0.02,
                eta=0.0, tol_index_offset=0)
    args.update(kw)
    with pytest.raises(pd.PdError) as e:
        pd.pd_init_schedule(**args)
    assert e.value.code == pd.PD_ERR_INVALID_ARG and msg in str(e.value)


@pytest.mark.parametrize("spec", [("ddpm", 1000, 1000, 0.0), ("ddpm", 100, 100, 0.0),
                                  ("ddim", 1000, 200, 0.0), ("ddim", 1000, 50, 0.7),
                                  ("ddpm", 2, 2, 0.0), ("heun", 1000, 100, 0.0),
                                  ("dpm2m", 1000, 200, 0.0), ("dpm2m", 90, 15, 0.0),
                                  ("dpm2m", 1000, 2, 0.0), ("dpm2m", 999, 3, 0.0)])
def test_schedule_tables_bitwise_equal_oracle(spec):
    kind, Tt, T, eta = spec
    k = {"ddpm": pd.PD_DDPM, "ddim": pd.PD_DDIM, "heun": pd.PD_DDIM_HEUN,
         "dpm2m": pd.PD_DDIM_DPM2M}[kind]
    s = pd.pd_init_schedule(k, Tt, T, eta=eta)
    tb = s.tables()
    ref = osched.ddpm(T) if kind == "ddpm" else osched.ddim(
        Tt, T, eta, solver=kind if kind in ("heun", "dpm2m") else "euler")
    A, B, zs, tv = ref.as_dtype(np.float32)
    R, S = ref.rs_dtype(np.float32)
    for name, ours, theirs in (("A", tb["A"], A), ("B", tb["B"], B),
                               ("noise_std", tb["noise_std"], zs), ("tol_var", tb["tol_var"], tv),
                               ("R", tb["R"], R), ("S", tb["S"], S)):
        # the library evaluates the same double-precision formulas in C; libm
        # and Python's math may differ in the last double bit, which rounding
        # to float absorbs except at a tie, so allow one float ulp
        d = np.abs(ours.view(np.int32).astype(np.int64) - theirs.view(np.int32).astype(np.int64))
        assert d.max(initial=0) <= (1 if kind == "dpm2m" else 0), name
    assert np.array_equal(tb["model_t"], ref.model_t)


def test_null_and_range_arguments_rejected_without_device():
    L = pd.load()
    out = ctypes.c_void_p()
    assert _status(L.pd_init_schedule, None, ctypes.byref(out))[0] == pd.PD_ERR_INVALID_ARG
    assert _status(L.pd_normals, 0, 0, -1, None, None)[0] == pd.PD_ERR_INVALID_ARG
    assert _status(L.pd_normals, 0, 0, 5, None, None)[0] == pd.PD_ERR_INVALID_ARG
    assert _status(L.pd_normals, 0, 0, 0, None, None)[0] == pd.PD_OK        # empty is a no-op
    assert _status(L.pd_denoiser_forward, None, None, None, 4, None, None)[0] == pd.PD_ERR_INVALID_ARG
    s = pd.pd_init_schedule(pd.PD_DDPM, 10, 10)
    shp = (ctypes.c_int64 * 1)(2)
    st = pd._Stats()
    for p, tau, msg in ((0, 0.1, "p must"), (4, -1.0, "tau"), (4, float("nan"), "tau")):
        code, m = _status(L.pd_sample_picard, s.handle, None, p, tau, 0, 1, shp, 1, None,
                          ctypes.byref(st), None, None)
        assert code == pd.PD_ERR_INVALID_ARG and msg in m
    code, m = _status(L.pd_sample_picard, s.handle, None, 4, 0.1, 0, 1, shp, 1, None,
                      ctypes.byref(st), None, None)
    assert code == pd.PD_ERR_INVALID_ARG and "NULL" in m
    code, m = _status(L.pd_sample_sequential, None, None, 0, 1, shp, 1, None, None, None, None)
    assert code == pd.PD_ERR_INVALID_ARG


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-GPU path")
def test_missing_gpu_reported_as_device_error():
    s = pd.pd_init_schedule(pd.PD_DDPM, 10, 10)
    w = {"means": np.zeros((8, 2), np.float32), "sigma0": np.ones(1, np.float32)}
    with pytest.raises(pd.PdError) as e:
        pd.pd_denoiser_create(pd.PD_MODEL_GMM2D, (2,), w, s)
    assert e.value.code == pd.PD_ERR_DEVICE


def test_denoiser_argument_validation_precedes_device():
    s = pd.pd_init_schedule(pd.PD_DDPM, 10, 10)
    w = {"means": np.zeros((8, 2), np.float32), "sigma0": np.ones(1, np.float32)}
    with pytest.raises(pd.PdError) as e:
        pd.pd_denoiser_create(pd.PD_MODEL_GMM2D, (3,), w, s)       # gmm2d is 2-D
    assert e.value.code == pd.PD_ERR_INVALID_ARG
    conv = {k: np.zeros((4, 4), np.float32) for k in pd.WEIGHT_ORDER[pd.PD_MODEL_CONV1X1]}
    with pytest.raises(pd.PdError) as e:
        pd.pd_denoiser_create(pd.PD_MODEL_CONV1X1, (4, 8, 8), conv, s, width=160)
    assert e.value.code == pd.PD_ERR_UNSUPPORTED


C_PROGRAM = r"""
#include <stdio.h>
#include "paradigms.h"

int main(void) {
    pd_schedule_desc d = {PD_DDPM, 1000, 1000, 0, PD_STOP_RELAXED, 1e-4, 0.02, 0.0};
    pd_schedule* s = NULL;
    if (pd_init_schedule(&d, &s) != PD_OK) { printf("init: %s\n", pd_last_error()); return 1; }
    int32_t T = 0;
    float A[1000], B[1000];
    if (pd_schedule_tables(s, &T, A, B, NULL, NULL, NULL) != PD_OK) return 2;
    d.T = 0;                              /* invalid: reported, no abort */
    pd_schedule* bad = NULL;
    const pd_status st = pd_init_schedule(&d, &bad);
    printf("%d %.9g %.9g %d %s\n", T, A[0], B[0], st, st == PD_ERR_INVALID_ARG ? "ok" : "no");
    pd_destroy_schedule(s);
    return 0;
}
"""


def test_plain_c_program_builds_and_runs(tmp_path):
    """The header is plain C and the library links into a C program: the
    schedule calls need no GPU, and an invalid argument comes back as a status."""
    import shutil
    import subprocess
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use.c"
    src.write_text(C_PROGRAM)
    exe = tmp_path / "use"
    libdir = os.path.dirname(pd.lib_path())
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                        str(src), "-L", libdir, "-lparadigms", f"-Wl,-rpath,{libdir}",
                        "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
    T, A0, B0, status, ok = r.stdout.split()
    tb = pd.pd_init_schedule(pd.PD_DDPM, 1000, 1000).tables()
    assert int(T) == 1000 and ok == "ok" and int(status) == pd.PD_ERR_INVALID_ARG
    assert np.float32(float(A0)) == tb["A"][0] and np.float32(float(B0)) == tb["B"][0]
