"""Host-side checks that need no GPU: the benchmark's one-GPU contract, the
product path failing loudly without its HIP library, and the separation of
the product path from the oracle."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    import paper_2305_16317_amd as pd
    monkeypatch.setattr(pd, "_LIB", None)
    monkeypatch.setattr(pd, "lib_path", lambda: str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        pd.load()


def test_product_path_does_not_touch_the_oracle():
    """The package neither imports nor names the oracle (only tests, the
    smoke check and the benchmark's CPU baseline may)."""
    pkg = os.path.join(ROOT, "paper_2305_16317_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f), encoding="utf-8").read()
                assert "oracle" not in text, os.path.join(dirpath, f)
    code = ("import sys; sys.path.insert(0, %r); import paper_2305_16317_amd, workloads; "
            "print(any(m == 'oracle' or m.startswith('oracle.') for m in sys.modules))" % ROOT)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "False"


def test_seeded_input_module_holds_no_method_arithmetic():
    """workloads/ (shared by the oracle and the GPU path) only generates
    inputs: it must not name the sampler's quantities."""
    text = open(os.path.join(ROOT, "workloads", "__init__.py"), encoding="utf-8").read()
    for word in ("alphabar", "cumsum", "picard", "drift", "stride"):
        assert word not in text.lower(), word


def test_bench_window_accounting():
    """Window points and history rows of a stride trace (the update's
    algorithmic bytes are priced from them)."""
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    b = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(b)
    # T = 10, p = 4: windows start at 0, 1, 3, 7 -> sizes 4, 4, 4, 3
    assert b.window_points([1, 2, 4, 3], 4, 10) == 15
    assert b.history_rows([1, 2, 4, 3], 10) == 3
    import workloads as W
    wl = W.WORKLOADS["policy_mlp_dpm15"]
    assert b.update_bytes(wl, 15, False, 3) == 160 * (12 * 15 + 8 * 3)
    assert b.sampler_name(wl).startswith("ParaDPMSolver")
    assert b.metric_name(W.WORKLOADS["latent_ddpm1000_p64"]) == b.METRIC
