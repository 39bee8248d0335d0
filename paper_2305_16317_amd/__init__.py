"""Python binding of the gfx950 ParaDiGMS library (libparadigms.so).

Argument marshalling only: every step of the sampling path runs in the HIP
library through its C ABI (include/paradigms.h), whose entry points carry
the same names.  PyTorch supplies device memory and streams; it is imported
before the library is loaded so that the process uses one HIP runtime.

If the library has not been built, ``load()`` raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch  # noqa: F401  (loads the HIP runtime first)

__all__ = [
    "PdError", "load", "lib_path", "Schedule", "Denoiser", "Workspace", "SampleStats",
    "pd_init_schedule", "pd_denoiser_create", "pd_denoiser_forward",
    "pd_denoiser_forward_static", "pd_normals",
    "pd_workspace_create", "pd_sample_sequential", "pd_sample_picard",
    "PD_DDPM", "PD_DDIM", "PD_DDIM_HEUN", "PD_DDIM_DPM2M", "PD_STOP_RELAXED", "PD_STOP_PROP2",
    "PD_MODEL_GMM2D", "PD_MODEL_MLP", "PD_MODEL_CONV1X1",
    "PD_F32", "PD_BF16", "EXPORTED_SYMBOLS",
]

PD_OK, PD_ERR_INVALID_ARG, PD_ERR_OOM, PD_ERR_DEVICE, PD_ERR_NUMERIC, PD_ERR_UNSUPPORTED = range(6)
STATUS_NAMES = {0: "PD_OK", 1: "PD_ERR_INVALID_ARG", 2: "PD_ERR_OOM", 3: "PD_ERR_DEVICE",
                4: "PD_ERR_NUMERIC", 5: "PD_ERR_UNSUPPORTED"}
PD_DDPM, PD_DDIM, PD_DDIM_HEUN, PD_DDIM_DPM2M = 0, 1, 2, 3
PD_STOP_RELAXED, PD_STOP_PROP2 = 0, 1
STOP_RULES = {"relaxed": PD_STOP_RELAXED, "prop2": PD_STOP_PROP2}
PD_MODEL_GMM2D, PD_MODEL_MLP, PD_MODEL_CONV1X1 = 0, 1, 2
PD_F32, PD_BF16 = 0, 1

EXPORTED_SYMBOLS = [
    "pd_last_error", "pd_version", "pd_init_schedule", "pd_destroy_schedule",
    "pd_schedule_tables", "pd_schedule_multistep_tables", "pd_denoiser_create", "pd_denoiser_destroy",
    "pd_denoiser_forward", "pd_denoiser_forward_static",
    "pd_normals", "pd_workspace_create", "pd_workspace_destroy", "pd_sample_sequential",
    "pd_sample_picard",
]


class PdError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


class _ScheduleDesc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("T_train", ctypes.c_int32), ("T", ctypes.c_int32),
                ("tol_index_offset", ctypes.c_int32), ("stop_rule", ctypes.c_int32),
                ("beta_start", ctypes.c_double),
                ("beta_end", ctypes.c_double), ("eta", ctypes.c_double)]


class _ModelDesc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("dtype", ctypes.c_int32), ("width", ctypes.c_int32),
                ("cond_dim", ctypes.c_int32), ("n_components", ctypes.c_int32),
                ("guidance", ctypes.c_float)]


class _Stats(ctypes.Structure):
    _fields_ = [("iters", ctypes.c_int32), ("trace_cap", ctypes.c_int32),
                ("evals_per_sample", ctypes.c_int64), ("network_rows", ctypes.c_int64),
                ("stride_trace", ctypes.POINTER(ctypes.c_int32)),
                ("time_kernels", ctypes.c_int32), ("denoiser_launches", ctypes.c_int32),
                ("update_launches", ctypes.c_int32), ("finalize_launches", ctypes.c_int32),
                ("denoiser_ms", ctypes.c_double), ("update_ms", ctypes.c_double),
                ("finalize_ms", ctypes.c_double)]


_LIB: Optional[ctypes.CDLL] = None


def lib_path() -> str:
    return os.path.join(os.path.dirname(os.path.abspath(__file__)), "libparadigms.so")


def load() -> ctypes.CDLL:
    """Load libparadigms.so (raises if it has not been built)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = lib_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with "
                           "`python -m paper_2305_16317_amd.build` (no fallback exists)")
    L = ctypes.CDLL(path)
    vp, i32, i64, u64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
    P = ctypes.POINTER
    sig = {
        "pd_last_error": ([], ctypes.c_char_p),
        "pd_version": ([], ctypes.c_char_p),
        "pd_init_schedule": ([P(_ScheduleDesc), P(vp)], i32),
        "pd_destroy_schedule": ([vp], None),
        "pd_schedule_tables": ([vp, P(i32), P(f32), P(f32), P(f32), P(f32), P(i32)], i32),
        "pd_schedule_multistep_tables": ([vp, P(f32), P(f32)], i32),
        "pd_denoiser_create": ([P(_ModelDesc), P(i64), i32, P(P(f32)), i32, vp, P(vp)], i32),
        "pd_denoiser_destroy": ([vp], None),
        "pd_denoiser_forward": ([vp, vp, vp, i64, vp, vp], i32),
        "pd_denoiser_forward_static": ([vp, vp, vp, i64, vp, vp], i32),
        "pd_normals": ([u64, ctypes.c_uint32, i64, vp, vp], i32),
        "pd_workspace_create": ([vp, vp, i32, i32, P(vp)], i32),
        "pd_workspace_destroy": ([vp], None),
        "pd_sample_sequential": ([vp, vp, u64, i32, P(i64), i32, vp, P(_Stats), vp, vp], i32),
        "pd_sample_picard": ([vp, vp, i32, f32, u64, i32, P(i64), i32, vp, P(_Stats), vp, vp], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _LIB = L
    return L


def _check(code: int) -> None:
    if code != PD_OK:
        raise PdError(code, load().pd_last_error().decode())


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _ptr(t: Optional[torch.Tensor]) -> ctypes.c_void_p:
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def _shape(shape: Sequence[int]):
    arr = (ctypes.c_int64 * len(shape))(*[int(v) for v in shape])
    return arr, len(shape)


# --------------------------------------------------------------------- handles
class Schedule:
    def __init__(self, handle: ctypes.c_void_p, T: int, T_train: int):
        self._h = handle
        self.T = T
        self.T_train = T_train

    @property
    def handle(self):
        return self._h

    def tables(self) -> Dict[str, np.ndarray]:
        T = self.T
        A, B, zs, tv = (np.empty(T, np.float32) for _ in range(4))
        nt = np.empty(T, np.int32)
        Tout = ctypes.c_int32(0)
        fp = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
        _check(load().pd_schedule_tables(self._h, ctypes.byref(Tout), fp(A), fp(B), fp(zs), fp(tv),
                                          nt.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
        R, S = np.empty(T, np.float32), np.empty(T, np.float32)
        _check(load().pd_schedule_multistep_tables(self._h, fp(R), fp(S)))
        return {"A": A, "B": B, "noise_std": zs, "tol_var": tv, "model_t": nt, "R": R, "S": S}

    def __del__(self):
        if getattr(self, "_h", None) and _LIB is not None:
            _LIB.pd_destroy_schedule(self._h)
            self._h = None


class Denoiser:
    def __init__(self, handle, sample_shape, guided: bool):
        self._h = handle
        self.sample_shape = tuple(sample_shape)
        self.D = int(np.prod(sample_shape))
        self.guided = guided

    @property
    def handle(self):
        return self._h

    def __del__(self):
        if getattr(self, "_h", None) and _LIB is not None:
            _LIB.pd_denoiser_destroy(self._h)
            self._h = None


class Workspace:
    def __init__(self, handle):
        self._h = handle

    @property
    def handle(self):
        return self._h

    def __del__(self):
        if getattr(self, "_h", None) and _LIB is not None:
            _LIB.pd_workspace_destroy(self._h)
            self._h = None


@dataclasses.dataclass
class SampleStats:
    iters: int
    evals_per_sample: int
    network_rows: int
    trace: List[int]
    kernel_times: Optional[Dict[str, float]] = dataclasses.field(default=None, compare=False)


# ------------------------------------------------------------------ entry points
def pd_init_schedule(kind: int, T_train: int, T: int, beta_start: float = 1e-4,
                     beta_end: float = 0.02, eta: float = 0.0,
                     tol_index_offset: int = 0, stop_rule: int = PD_STOP_RELAXED) -> Schedule:
    d = _ScheduleDesc(kind, T_train, T, tol_index_offset, stop_rule, beta_start, beta_end, eta)
    h = ctypes.c_void_p()
    _check(load().pd_init_schedule(ctypes.byref(d), ctypes.byref(h)))
    return Schedule(h, T, T_train)


WEIGHT_ORDER = {
    PD_MODEL_GMM2D: ["means", "sigma0"],
    PD_MODEL_MLP: ["W1", "b1", "W2", "b2", "W3", "b3", "W4", "b4"],
    PD_MODEL_CONV1X1: ["W1", "b1", "W2", "b2", "W3", "b3", "W4", "b4"],
}


def pd_denoiser_create(kind: int, sample_shape: Sequence[int], weights: Dict[str, np.ndarray],
                       train: Schedule, width: int = 0, dtype: int = PD_F32,
                       cond_dim: int = 0, guidance: float = 1.0,
                       n_components: int = 0) -> Denoiser:
    names = list(WEIGHT_ORDER[kind]) + (["Wc", "c"] if cond_dim else [])
    arrs = [np.ascontiguousarray(weights[k], dtype=np.float32) for k in names]
    ptrs = (ctypes.POINTER(ctypes.c_float) * len(arrs))(
        *[a.ctypes.data_as(ctypes.POINTER(ctypes.c_float)) for a in arrs])
    if kind == PD_MODEL_GMM2D and not n_components:
        n_components = arrs[0].size // 2
    d = _ModelDesc(kind, dtype, width, cond_dim, n_components, guidance)
    shp, nd = _shape(sample_shape)
    h = ctypes.c_void_p()
    _check(load().pd_denoiser_create(ctypes.byref(d), shp, nd, ptrs, len(arrs), train.handle,
                                     ctypes.byref(h)))
    return Denoiser(h, sample_shape, cond_dim > 0)


def pd_denoiser_forward(den: Denoiser, x: torch.Tensor, model_t: torch.Tensor,
                        eps: torch.Tensor, stream=None) -> None:
    M = x.shape[0] if x.dim() else 0
    for t, dt in ((x, torch.float32), (eps, torch.float32), (model_t, torch.int32)):
        if t.dtype != dt or not t.is_contiguous() or not t.is_cuda:
            raise ValueError("x/eps must be contiguous float32 and model_t int32, on the GPU")
    _check(load().pd_denoiser_forward(den.handle, _ptr(x), _ptr(model_t), M, _ptr(eps),
                                      _stream(stream)))


def pd_denoiser_forward_static(den: Denoiser, x: torch.Tensor, model_t: torch.Tensor,
                               eps: torch.Tensor, stream=None) -> None:
    """pd_denoiser_forward without any allocation or synchronisation (the
    MLP's scratch is a static per-GPU array: M * 2 * width <= 2^20)."""
    M = x.shape[0] if x.dim() else 0
    for t, dt in ((x, torch.float32), (eps, torch.float32), (model_t, torch.int32)):
        if t.dtype != dt or not t.is_contiguous() or not t.is_cuda:
            raise ValueError("x/eps must be contiguous float32 and model_t int32, on the GPU")
    _check(load().pd_denoiser_forward_static(den.handle, _ptr(x), _ptr(model_t), M, _ptr(eps),
                                             _stream(stream)))


def pd_normals(seed: int, rng_stream: int, out: torch.Tensor, stream=None) -> None:
    if out.dtype != torch.float32 or not out.is_contiguous() or not out.is_cuda:
        raise ValueError("out must be a contiguous float32 GPU tensor")
    _check(load().pd_normals(seed, rng_stream, out.numel(), _ptr(out), _stream(stream)))


def pd_workspace_create(sched: Schedule, den: Denoiser, p: int, batch: int) -> Workspace:
    h = ctypes.c_void_p()
    _check(load().pd_workspace_create(sched.handle, den.handle, p, batch, ctypes.byref(h)))
    return Workspace(h)


def _stats(trace_cap: int, time_kernels: bool = False):
    buf = (ctypes.c_int32 * max(trace_cap, 1))()
    st = _Stats(0, trace_cap, 0, 0, ctypes.cast(buf, ctypes.POINTER(ctypes.c_int32)),
                int(time_kernels))
    return st, buf


def _out_stats(st, buf) -> SampleStats:
    n = min(st.iters, st.trace_cap)
    kt = None
    if st.time_kernels:
        kt = {"denoiser_ms": st.denoiser_ms, "denoiser_launches": st.denoiser_launches,
              "update_ms": st.update_ms, "update_launches": st.update_launches,
              "finalize_ms": st.finalize_ms, "finalize_launches": st.finalize_launches}
    return SampleStats(st.iters, st.evals_per_sample, st.network_rows, list(buf[:n]), kt)


def _check_out(x_out: torch.Tensor, batch: int, den: Denoiser):
    if (x_out.dtype != torch.float32 or not x_out.is_contiguous() or not x_out.is_cuda
            or x_out.numel() != batch * den.D):
        raise ValueError("x_out must be a contiguous float32 GPU tensor of batch * D elements")


def pd_sample_sequential(sched: Schedule, den: Denoiser, noise_seed: int, batch: int,
                         sample_shape: Sequence[int], x_out: torch.Tensor,
                         workspace: Optional[Workspace] = None, stream=None,
                         trace_cap: int = 0, time_kernels: bool = False) -> SampleStats:
    _check_out(x_out, batch, den)
    shp, nd = _shape(sample_shape)
    st, buf = _stats(trace_cap, time_kernels)
    _check(load().pd_sample_sequential(sched.handle, den.handle, noise_seed, batch, shp, nd,
                                       _ptr(x_out), ctypes.byref(st),
                                       workspace.handle if workspace else None, _stream(stream)))
    return _out_stats(st, buf)


def pd_sample_picard(sched: Schedule, den: Denoiser, p: int, tau: float, noise_seed: int,
                     batch: int, sample_shape: Sequence[int], x_out: torch.Tensor,
                     workspace: Optional[Workspace] = None, stream=None,
                     trace_cap: Optional[int] = None, time_kernels: bool = False) -> SampleStats:
    _check_out(x_out, batch, den)
    shp, nd = _shape(sample_shape)
    st, buf = _stats(sched.T if trace_cap is None else trace_cap, time_kernels)
    _check(load().pd_sample_picard(sched.handle, den.handle, p, float(tau), noise_seed, batch,
                                   shp, nd, _ptr(x_out), ctypes.byref(st),
                                   workspace.handle if workspace else None, _stream(stream)))
    return _out_stats(st, buf)


# ------------------------------------------------------------ workload helpers
def from_workload(w, weights: Dict[str, np.ndarray], tol_index_offset: int = 0,
                  rule: str = "relaxed"):
    """(schedule, denoiser) handles for a ``workloads.Workload``.  The schedule
    carries the training chain (T_train, abar) that the denoiser needs, and
    the stride test's reading (``tol_index_offset``) and rule ("relaxed" or
    "prop2")."""
    s = w.schedule
    if s.kind == "ddpm":
        kind = PD_DDPM
    else:
        kind = {"euler": PD_DDIM, "heun": PD_DDIM_HEUN,
                "dpm2m": PD_DDIM_DPM2M}[getattr(s, "solver", "euler")]
    sched = pd_init_schedule(kind, s.T_train, s.T, s.beta_start, s.beta_end, s.eta,
                             tol_index_offset, STOP_RULES[rule])
    m = w.model
    mk = {"gmm2d": PD_MODEL_GMM2D, "mlp": PD_MODEL_MLP, "conv1x1": PD_MODEL_CONV1X1}[m.kind]
    den = pd_denoiser_create(mk, m.sample_shape, weights, sched, width=m.width,
                             dtype=PD_BF16 if m.dtype == "bf16" else PD_F32,
                             cond_dim=m.cond_dim, guidance=m.guidance,
                             n_components=m.n_components if m.kind == "gmm2d" else 0)
    return sched, den
