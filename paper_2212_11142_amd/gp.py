"""Thin ctypes binding of libbaco_gp.so (the C-ABI in include/baco_gp.h).

Argument marshalling only: every step of fitting and scoring runs in the library's HIP
kernels. PyTorch supplies device memory (inputs, outputs, workspaces) and the current
HIP stream. There is no CPU fallback: if the library is missing or a call fails, an
exception is raised.
"""
from __future__ import annotations

import atexit
import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbaco_gp.so")

GP_REAL, GP_INT, GP_ORD, GP_CAT, GP_PERM = range(5)
PERM_DIST = {"spearman": 0, "kendall": 1, "hamming": 2, "naive": 3}
KIND = {"real": GP_REAL, "int": GP_INT, "ord": GP_ORD, "cat": GP_CAT, "perm": GP_PERM}
STATUS = {0: "GP_OK", 1: "GP_E_INVALID", 2: "GP_E_NOT_SPD", 3: "GP_E_HIP",
          4: "GP_E_UNSUPPORTED", 5: "GP_E_WORKSPACE", 6: "GP_E_NOT_CONVERGED"}
FIELDS = {"K": 0, "L": 1, "LINV": 2, "KINV": 3, "ALPHA": 4, "FEASIBLE_INDEX": 5,
          "CLS_F": 6, "CLS_GRAD": 7, "CLS_SQRTW": 8, "CLS_L": 9}
STAGES = ("encode", "xkernel", "contract", "epilogue", "refine", "argmax")


class GPError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class _Space(C.Structure):
    _fields_ = [("d", C.c_int32), ("type", C.POINTER(C.c_int32)), ("log2", C.POINTER(C.c_int32)),
                ("n_levels", C.POINTER(C.c_int32)), ("perm_dist", C.POINTER(C.c_int32)),
                ("lo", C.POINTER(C.c_double)), ("hi", C.POINTER(C.c_double)),
                ("ord_values", C.POINTER(C.POINTER(C.c_double)))]


class _Hyper(C.Structure):
    _fields_ = [("lengthscale", C.POINTER(C.c_double)), ("signal_var", C.c_double),
                ("noise_var", C.c_double)]


class _Prior(C.Structure):
    _fields_ = [("shape", C.c_double), ("rate", C.c_double)]


class _Info(C.Structure):
    _fields_ = [("n", C.c_int32), ("n_feasible", C.c_int32), ("d", C.c_int32),
                ("has_classifier", C.c_int32), ("cls_iterations", C.c_int32),
                ("code_words", C.c_int32), ("fstar", C.c_double), ("signal_var", C.c_double),
                ("noise_var", C.c_double), ("cls_signal_var", C.c_double)]


_lib = None

# (name, restype, argtypes) for every entry point of include/baco_gp.h
_VP = C.c_void_p
_SIGS = [
    ("gp_fit_workspace_bytes", C.c_size_t, [C.POINTER(_Space), C.c_int32, C.c_int32]),
    ("gp_fit", C.c_int, [C.POINTER(_Space), C.POINTER(_VP), C.c_int32, _VP, _VP,
                         C.POINTER(_Hyper), C.POINTER(_Hyper), _VP, C.c_size_t, _VP,
                         C.POINTER(_VP)]),
    ("gp_model_info", C.c_int, [_VP, C.POINTER(_Info)]),
    ("gp_model_export", C.c_int, [_VP, C.c_int32, C.POINTER(C.c_double), C.c_size_t]),
    ("gp_model_free", None, [_VP]),
    ("gp_score_workspace_bytes", C.c_size_t, [_VP, C.c_int64]),
    ("gp_score", C.c_int, [_VP, C.POINTER(_VP), C.c_int64, _VP, C.c_float, _VP, _VP, _VP, _VP,
                           _VP, _VP, _VP, C.c_size_t, _VP]),
    ("gp_score_noalloc", C.c_int, [_VP, C.POINTER(_VP), C.c_int64, _VP, C.c_float, _VP, _VP,
                                   _VP, _VP, _VP, _VP, _VP]),
    ("gp_score_noalloc_max_candidates", C.c_size_t, [_VP]),
    ("gp_fit_score_workspace_bytes", C.c_size_t, [C.POINTER(_Space), C.c_int32, C.c_int32,
                                                  C.c_int64]),
    ("gp_fit_score", C.c_int, [C.POINTER(_Space), C.POINTER(_VP), C.c_int32, _VP, _VP,
                               C.POINTER(_Hyper), C.POINTER(_Hyper), C.POINTER(_VP), C.c_int64,
                               _VP, C.c_float, _VP, _VP, _VP, _VP, _VP, _VP, _VP, C.c_size_t,
                               _VP, C.POINTER(_VP)]),
    ("gp_local_search_workspace_bytes", C.c_size_t, [_VP, C.c_int64, C.c_int32]),
    ("gp_local_search", C.c_int, [_VP, C.POINTER(_VP), C.c_int64, _VP, C.c_float, C.c_int32,
                                  C.c_int32, C.POINTER(_VP), _VP, _VP, _VP, _VP, C.c_size_t,
                                  _VP]),
    ("gp_hyper_workspace_bytes", C.c_size_t, [C.POINTER(_Space), C.c_int32, C.c_int32,
                                              C.c_int32]),
    ("gp_log_posterior", C.c_int, [C.POINTER(_Space), C.POINTER(_VP), C.c_int32, _VP, _VP, _VP,
                                   C.c_int32, C.POINTER(_Prior), C.c_double, _VP, _VP, _VP,
                                   C.c_size_t, _VP]),
    ("gp_hyperfit", C.c_int, [C.POINTER(_Space), C.POINTER(_VP), C.c_int32, _VP, _VP, _VP,
                              C.c_int32, C.c_int32, C.POINTER(_Prior), C.c_double, C.c_int32,
                              C.c_double, C.c_double, _VP, _VP, _VP, _VP, _VP, _VP, _VP,
                              C.c_size_t, _VP]),
    ("gp_cot_workspace_bytes", C.c_size_t, [C.POINTER(_Space), C.c_int32, _VP, _VP, _VP]),
    ("gp_cot_create", C.c_int, [C.POINTER(_Space), C.c_int32, _VP, _VP, _VP, C.POINTER(_VP), _VP,
                                C.c_size_t, _VP, C.POINTER(_VP)]),
    ("gp_cot_sample", C.c_int, [_VP, C.c_int64, C.c_uint64, C.c_uint64, C.POINTER(_VP), _VP]),
    ("gp_cot_member", C.c_int, [_VP, C.POINTER(_VP), C.c_int64, _VP, _VP]),
    ("gp_cot_free", None, [_VP]),
    ("gp_forest_workspace_bytes", C.c_size_t, [C.POINTER(_Space), C.c_int32, C.c_int32]),
    ("gp_forest_fit", C.c_int, [C.POINTER(_Space), C.POINTER(_VP), C.c_int32, _VP, C.c_int32,
                                C.c_int32, C.c_int32, C.c_uint64, _VP, C.c_size_t, _VP,
                                C.POINTER(_VP)]),
    ("gp_forest_predict", C.c_int, [_VP, C.POINTER(_VP), C.c_int64, _VP, _VP, C.c_float, _VP,
                                    _VP, _VP]),
    ("gp_forest_tree", C.c_int, [_VP, C.c_int32, C.c_int32, C.POINTER(C.c_int32), _VP, _VP, _VP,
                                 _VP]),
    ("gp_forest_free", None, [_VP]),
    ("gp_debug_workspace_bytes", C.c_size_t, [C.POINTER(_Space), _VP, C.c_int64]),
    ("gp_debug_encode", C.c_int, [C.POINTER(_Space), C.POINTER(_VP), C.c_int64, _VP, _VP, _VP,
                                  C.c_size_t, _VP]),
    ("gp_debug_terms", C.c_int, [_VP, C.POINTER(_VP), C.c_int64, _VP, _VP, C.c_size_t, _VP]),
    ("gp_debug_xkernel", C.c_int, [_VP, C.POINTER(_VP), C.c_int64, _VP, _VP, C.c_size_t, _VP]),
    ("gp_debug_pairs", C.c_int, [_VP, C.POINTER(_VP), C.c_int64, _VP, _VP,
                                 C.POINTER(C.c_uint64), C.POINTER(C.c_int32), _VP, C.c_size_t,
                                 _VP]),
    ("gp_debug_set_refine", C.c_int, [_VP, C.c_double, C.c_double]),
    ("gp_profile_start", C.c_int, []),
    ("gp_profile_stop", C.c_int, [C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
    ("gp_score_refined_count", C.c_int, [_VP, _VP, C.c_int64, _VP, C.POINTER(C.c_int64)]),
    ("gp_release", C.c_int, []),
    ("gp_last_error", C.c_char_p, []),
    ("gp_version", C.c_int32, []),
]


def load():
    """Load the built library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        lib = C.CDLL(LIB_PATH)
        for name, res, args in _SIGS:
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
        atexit.register(_release_at_exit)
    return _lib


def _release_at_exit():
    """Free the library's own streams and pinned host buffers before the interpreter
    (and with it the HIP runtime) shuts down."""
    if _lib is not None:
        _lib.gp_release()


def release():
    """gp_release: free the library's own streams and pinned host buffers now (they are
    recreated on demand by later calls)."""
    _check(load().gp_release())


def exported_names():
    return [s[0] for s in _SIGS]


def _check(status):
    if status != 0:
        raise GPError(status, load().gp_last_error().decode())


def _torch():
    import torch
    return torch


def _stream():
    torch = _torch()
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _workspace(nbytes):
    torch = _torch()
    # torch's caching allocator returns 512-byte aligned blocks
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")


# ------------------------------------------------------------------ space
class Space:
    """A search space (list of parameter descriptions) as a gp_space struct.

    Each parameter needs attributes ``kind`` ('real' | 'int' | 'ord' | 'cat' | 'perm'),
    ``log2``, ``lo``, ``hi``, ``values``, ``levels``, ``m`` and ``dist``."""

    def __init__(self, params: Sequence):
        self.params = list(params)
        d = len(self.params)
        self._type = (C.c_int32 * d)(*[KIND[p.kind] for p in self.params])
        self._log2 = (C.c_int32 * d)(*[1 if getattr(p, "log2", False) else 0 for p in self.params])
        lev = []
        for p in self.params:
            if p.kind == "cat":
                lev.append(p.levels)
            elif p.kind == "ord":
                lev.append(len(p.values))
            elif p.kind == "perm":
                lev.append(p.m)
            else:
                lev.append(0)
        self._lev = (C.c_int32 * d)(*lev)
        self._dist = (C.c_int32 * d)(*[PERM_DIST.get(getattr(p, "dist", "spearman"), 0)
                                       for p in self.params])
        self._lo = (C.c_double * d)(*[float(getattr(p, "lo", 0.0)) for p in self.params])
        self._hi = (C.c_double * d)(*[float(getattr(p, "hi", 1.0)) for p in self.params])
        self._vals = []
        ptrs = (C.POINTER(C.c_double) * d)()
        for i, p in enumerate(self.params):
            if p.kind == "ord":
                arr = (C.c_double * len(p.values))(*[float(v) for v in p.values])
                self._vals.append(arr)
                ptrs[i] = C.cast(arr, C.POINTER(C.c_double))
        self._ptrs = ptrs
        self.struct = _Space(d, self._type, self._log2, self._lev, self._dist, self._lo, self._hi,
                             self._ptrs)

    @property
    def d(self):
        return len(self.params)

    @property
    def n_numeric(self):
        return sum(1 for p in self.params if p.kind in ("real", "int", "ord"))

    def ref(self):
        return C.byref(self.struct)


def to_device_columns(space: Space, cols):
    """Raw numpy columns -> contiguous CUDA tensors of the C-ABI dtypes."""
    torch = _torch()
    out = []
    for p, c in zip(space.params, cols):
        a = np.ascontiguousarray(c)
        if p.kind == "real":
            a = a.astype(np.float64)
        else:
            a = a.astype(np.int32)
        out.append(torch.from_numpy(a).to("cuda"))
    return out


def _col_ptrs(cols):
    arr = (C.c_void_p * len(cols))()
    for i, c in enumerate(cols):
        if not c.is_contiguous():
            raise ValueError("columns must be contiguous")
        arr[i] = c.data_ptr()
    return arr


# ------------------------------------------------------------------ model
class Model:
    def __init__(self, handle, workspace, space):
        self.handle = handle
        self.workspace = workspace   # device memory the model refers to
        self.space = space

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.gp_model_free(self.handle)
            self.handle = None

    def info(self) -> dict:
        inf = _Info()
        _check(load().gp_model_info(self.handle, C.byref(inf)))
        return {k: getattr(inf, k) for k, _ in _Info._fields_}

    def export(self, field: str) -> np.ndarray:
        inf = self.info()
        n, nf = inf["n"], inf["n_feasible"]
        size = {"K": nf * nf, "L": nf * nf, "LINV": nf * nf, "KINV": nf * nf, "ALPHA": nf,
                "FEASIBLE_INDEX": n, "CLS_F": n, "CLS_GRAD": n, "CLS_SQRTW": n,
                "CLS_L": n * n}[field]
        buf = np.zeros(size, dtype=np.float64)
        _check(load().gp_model_export(self.handle, FIELDS[field],
                                      buf.ctypes.data_as(C.POINTER(C.c_double)), size))
        if size in (nf * nf,) and field in ("K", "L", "LINV", "KINV"):
            return buf.reshape(nf, nf)
        if field == "CLS_L":
            return buf.reshape(n, n)
        return buf


def fit(space: Space, X_cols, y, feasible, lengthscale, signal_var, noise_var,
        cls_signal_var: Optional[float] = None) -> Model:
    """gp_fit on CUDA tensors (X_cols: list of device columns; y: float64 [n];
    feasible: uint8 [n] or None)."""
    lib = load()
    n = int(y.shape[0])
    ls = np.ascontiguousarray(lengthscale, dtype=np.float64)
    ls_p = ls.ctypes.data_as(C.POINTER(C.c_double))
    reg = _Hyper(ls_p, float(signal_var), float(noise_var))
    cls = _Hyper(ls_p, float(cls_signal_var), 0.0) if cls_signal_var is not None else None
    nbytes = lib.gp_fit_workspace_bytes(space.ref(), n, 1 if cls is not None else 0)
    if nbytes == 0:
        raise GPError(1, "gp_fit_workspace_bytes rejected the space or n")
    ws = _workspace(nbytes)
    h = C.c_void_p()
    cols = _col_ptrs(X_cols)
    _check(lib.gp_fit(space.ref(), cols, n, _ptr(y), _ptr(feasible), C.byref(reg),
                      C.byref(cls) if cls is not None else None, _ptr(ws), ws.numel(), _stream(),
                      C.byref(h)))
    return Model(h, ws, space)


class ScoreBuffers:
    """Outputs + workspace of gp_score for M candidates (reusable across calls)."""

    def __init__(self, model: Model, M: int, want_p=True, want_argmax=False):
        torch = _torch()
        lib = load()
        self.M = int(M)
        dev = "cuda"
        self.mu = torch.empty(max(M, 1), dtype=torch.float32, device=dev)
        self.sigma = torch.empty_like(self.mu)
        self.ei = torch.empty_like(self.mu)
        self.acq = torch.empty_like(self.mu)
        self.p_feas = torch.empty_like(self.mu) if want_p else None
        self.argmax = torch.zeros(1, dtype=torch.int64, device=dev) if want_argmax else None
        nbytes = lib.gp_score_workspace_bytes(model.handle, self.M)
        if nbytes == 0:
            raise GPError(1, "gp_score_workspace_bytes rejected M")
        self.workspace = _workspace(nbytes)

    def result(self) -> dict:
        out = {"mu": self.mu[:self.M], "sigma": self.sigma[:self.M], "ei": self.ei[:self.M],
               "acq": self.acq[:self.M]}
        if self.p_feas is not None:
            out["p_feas"] = self.p_feas[:self.M]
        if self.argmax is not None:
            out["argmax"] = self.argmax
        return out


def score_into(model: Model, C_cols, bufs: ScoreBuffers, mask=None, eps_f: float = 0.0,
               stream=None):
    """gp_score into preallocated buffers (asynchronous on the current stream)."""
    lib = load()
    cols = _col_ptrs(C_cols)
    st = stream if stream is not None else _stream()
    _check(lib.gp_score(model.handle, cols, bufs.M, _ptr(mask), C.c_float(eps_f), _ptr(bufs.mu),
                        _ptr(bufs.sigma), _ptr(bufs.ei), _ptr(bufs.p_feas), _ptr(bufs.acq),
                        _ptr(bufs.argmax), _ptr(bufs.workspace), bufs.workspace.numel(), st))


def score(model: Model, C_cols, mask=None, eps_f: float = 0.0, want_p=True,
          want_argmax=False) -> dict:
    M = int(C_cols[0].shape[0])
    bufs = ScoreBuffers(model, M, want_p, want_argmax)
    score_into(model, C_cols, bufs, mask, eps_f)
    out = bufs.result()
    out["_buffers"] = bufs
    return out


def score_noalloc_max(model: Model) -> int:
    return int(load().gp_score_noalloc_max_candidates(model.handle))


def score_noalloc(model: Model, C_cols, mask=None, eps_f: float = 0.0, want_p=True,
                  want_argmax=False) -> dict:
    """gp_score_noalloc: gp_score with the library's fixed device scratch array in place
    of a workspace (the outputs are still allocated here, by the caller)."""
    torch = _torch()
    lib = load()
    M = int(C_cols[0].shape[0])
    out = {k: torch.empty(max(M, 1), dtype=torch.float32, device="cuda")
           for k in ("mu", "sigma", "ei", "acq")}
    if want_p:
        out["p_feas"] = torch.empty(max(M, 1), dtype=torch.float32, device="cuda")
    if want_argmax:
        out["argmax"] = torch.zeros(1, dtype=torch.int64, device="cuda")
    _check(lib.gp_score_noalloc(model.handle, _col_ptrs(C_cols), M, _ptr(mask), C.c_float(eps_f),
                                _ptr(out["mu"]), _ptr(out["sigma"]), _ptr(out["ei"]),
                                _ptr(out.get("p_feas")), _ptr(out["acq"]), _ptr(out.get("argmax")),
                                _stream()))
    return {k: (v if k == "argmax" else v[:M]) for k, v in out.items()}


class FitScoreBuffers:
    """Outputs + workspace of gp_fit_score for n observations and M candidates. The
    model a call returns lives in this workspace until the next call with it."""

    def __init__(self, space: Space, n: int, M: int, with_cls=True, want_p=True,
                 want_argmax=False):
        torch = _torch()
        lib = load()
        self.n, self.M, self.with_cls = int(n), int(M), bool(with_cls)
        self.mu = torch.empty(max(M, 1), dtype=torch.float32, device="cuda")
        self.sigma = torch.empty_like(self.mu)
        self.ei = torch.empty_like(self.mu)
        self.acq = torch.empty_like(self.mu)
        self.p_feas = torch.empty_like(self.mu) if want_p else None
        self.argmax = torch.zeros(1, dtype=torch.int64, device="cuda") if want_argmax else None
        total = lib.gp_fit_score_workspace_bytes(space.ref(), self.n, int(self.with_cls), self.M)
        fit = lib.gp_fit_workspace_bytes(space.ref(), self.n, int(self.with_cls))
        if total == 0 or fit == 0:
            raise GPError(1, "gp_fit_score_workspace_bytes rejected the space, n or M")
        self.fit_workspace = _workspace(total)
        # the scoring buffers (their first word: the count of fp64-recomputed candidates)
        self.workspace = self.fit_workspace[(fit + 255) // 256 * 256:]

    result = ScoreBuffers.result


def fit_score_into(space: Space, X_cols, y, feasible, lengthscale, signal_var, noise_var,
                   cls_signal_var, C_cols, bufs: FitScoreBuffers, mask=None,
                   eps_f: float = 0.0) -> Model:
    """gp_fit_score: fit on the observations and score the candidates into `bufs`
    (the scoring completes asynchronously on the current stream)."""
    lib = load()
    n = int(y.shape[0])
    if n != bufs.n or int(C_cols[0].shape[0]) != bufs.M or (cls_signal_var is not None) != bufs.with_cls:
        raise GPError(1, "buffers were made for another n, M or classifier setting")
    ls = np.ascontiguousarray(lengthscale, dtype=np.float64)
    ls_p = ls.ctypes.data_as(C.POINTER(C.c_double))
    reg = _Hyper(ls_p, float(signal_var), float(noise_var))
    cls = _Hyper(ls_p, float(cls_signal_var), 0.0) if cls_signal_var is not None else None
    h = C.c_void_p()
    ws = bufs.fit_workspace
    _check(lib.gp_fit_score(space.ref(), _col_ptrs(X_cols), n, _ptr(y), _ptr(feasible),
                            C.byref(reg), C.byref(cls) if cls is not None else None,
                            _col_ptrs(C_cols), bufs.M, _ptr(mask), C.c_float(eps_f),
                            _ptr(bufs.mu), _ptr(bufs.sigma), _ptr(bufs.ei), _ptr(bufs.p_feas),
                            _ptr(bufs.acq), _ptr(bufs.argmax), _ptr(ws), ws.numel(), _stream(),
                            C.byref(h)))
    return Model(h, ws, space)


def local_search(model: Model, C_cols, mask=None, eps_f: float = 0.0, n_starts: int = 8,
                 max_steps: int = 64) -> dict:
    """gp_local_search: start indices, final configurations (raw device columns), final
    acquisition values and moves per start (synchronous)."""
    torch = _torch()
    lib = load()
    M = int(C_cols[0].shape[0])
    k = min(int(n_starts), M)
    nbytes = lib.gp_local_search_workspace_bytes(model.handle, M, int(n_starts))
    if nbytes == 0:
        raise GPError(1, "gp_local_search_workspace_bytes rejected the arguments")
    ws = _workspace(nbytes)
    out_cols = []
    for p in model.space.params:
        if p.kind == "real":
            out_cols.append(torch.empty(k, dtype=torch.float64, device="cuda"))
        elif p.kind == "perm":
            out_cols.append(torch.empty((k, p.m), dtype=torch.int32, device="cuda"))
        else:
            out_cols.append(torch.empty(k, dtype=torch.int32, device="cuda"))
    acq = torch.empty(k, dtype=torch.float32, device="cuda")
    steps = torch.empty(k, dtype=torch.int32, device="cuda")
    start = torch.empty(k, dtype=torch.int64, device="cuda")
    _check(lib.gp_local_search(model.handle, _col_ptrs(C_cols), M, _ptr(mask), C.c_float(eps_f),
                               int(n_starts), int(max_steps), _col_ptrs(out_cols), _ptr(acq),
                               _ptr(steps), _ptr(start), _ptr(ws), ws.numel(), _stream()))
    return {"start_index": start, "cols": out_cols, "acq": acq, "steps": steps}


# ------------------------------------------------------------------ hyperparameters
def _prior(prior):
    return None if prior is None else C.byref(_Prior(float(prior[0]), float(prior[1])))


def log_posterior(space: Space, X_cols, y, feasible, theta, prior=None, noise_floor=1e-6,
                  want_grad=True) -> dict:
    """gp_log_posterior: objective (and gradient) of the settings theta (CUDA float64
    [count, d + 2]: log lengthscales, log signal_var, t with noise = floor + e^t)."""
    torch = _torch()
    lib = load()
    n, count = int(y.shape[0]), int(theta.shape[0])
    nbytes = lib.gp_hyper_workspace_bytes(space.ref(), n, count, 0)
    if nbytes == 0:
        raise GPError(1, "gp_hyper_workspace_bytes rejected the arguments")
    ws = _workspace(nbytes)
    theta = theta.contiguous()
    value = torch.empty(count, dtype=torch.float64, device="cuda")
    grad = torch.empty_like(theta) if want_grad else None
    _check(lib.gp_log_posterior(space.ref(), _col_ptrs(X_cols), n, _ptr(y), _ptr(feasible),
                                _ptr(theta), count, _prior(prior), float(noise_floor),
                                _ptr(value), _ptr(grad), _ptr(ws), ws.numel(), _stream()))
    return {"value": value, "grad": grad}


def hyperfit(space: Space, X_cols, y, feasible, theta0, n_keep, prior=None, noise_floor=1e-6,
             max_iter=100, gtol=1e-5, ftol=1e-10) -> dict:
    """gp_hyperfit: multistart L-BFGS fit from the sampled settings theta0 (CUDA float64
    [n_samples, d + 2]); returns the kept starts' final settings and objectives, every
    sample's objective, the kept indices, iterations and stop reasons."""
    torch = _torch()
    lib = load()
    n, S0, K = int(y.shape[0]), int(theta0.shape[0]), int(n_keep)
    nbytes = lib.gp_hyper_workspace_bytes(space.ref(), n, S0, K)
    if nbytes == 0:
        raise GPError(1, "gp_hyper_workspace_bytes rejected the arguments")
    ws = _workspace(nbytes)
    theta0 = theta0.contiguous()
    D = int(theta0.shape[1])
    dev = "cuda"
    theta = torch.empty((K, D), dtype=torch.float64, device=dev)
    value = torch.empty(K, dtype=torch.float64, device=dev)
    value0 = torch.empty(S0, dtype=torch.float64, device=dev)
    keep = torch.empty(K, dtype=torch.int32, device=dev)
    iters = torch.empty(K, dtype=torch.int32, device=dev)
    status = torch.empty(K, dtype=torch.int32, device=dev)
    _check(lib.gp_hyperfit(space.ref(), _col_ptrs(X_cols), n, _ptr(y), _ptr(feasible),
                           _ptr(theta0), S0, K, _prior(prior), float(noise_floor), int(max_iter),
                           float(gtol), float(ftol), _ptr(theta), _ptr(value), _ptr(value0),
                           _ptr(keep), _ptr(iters), _ptr(status), _ptr(ws), ws.numel(),
                           _stream()))
    return {"theta": theta, "value": value, "value0": value0, "keep": keep, "iters": iters,
            "status": status}


# ------------------------------------------------------------------ known constraints
class Chain:
    """A Chain-of-Trees on the device (gp_cot_create). trees: lists of parameter
    indices (level order); leaves: per tree an int array [n_leaves, k] of value indices
    in lexicographic order (numpy or a CUDA tensor)."""

    def __init__(self, space: Space, trees, leaves):
        torch = _torch()
        lib = load()
        self.space = space
        self.trees = [list(map(int, t)) for t in trees]
        nt = len(self.trees)
        self._size = np.array([len(t) for t in self.trees], dtype=np.int32)
        self._params = np.array([p for t in self.trees for p in t], dtype=np.int32)
        dev = []
        for lv in leaves:
            t = lv if isinstance(lv, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(lv))
            dev.append(t.to(device="cuda", dtype=torch.int32).contiguous())
        self._nleaves = np.array([int(t.shape[0]) for t in dev], dtype=np.int64)
        args = (space.ref(), nt, self._size.ctypes.data_as(_VP), self._params.ctypes.data_as(_VP),
                self._nleaves.ctypes.data_as(_VP))
        nbytes = lib.gp_cot_workspace_bytes(*args)
        if nbytes == 0:
            raise GPError(1, "gp_cot_workspace_bytes rejected the chain: " +
                          lib.gp_last_error().decode())
        self.workspace = _workspace(nbytes)
        ptrs = (_VP * max(nt, 1))(*[t.data_ptr() for t in dev])
        h = C.c_void_p()
        _check(lib.gp_cot_create(*args, ptrs, _ptr(self.workspace), self.workspace.numel(),
                                 _stream(), C.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.gp_cot_free(self.handle)
            self.handle = None

    def sample(self, M: int, seed: int, offset: int = 0):
        """gp_cot_sample: M configurations as CUDA raw columns."""
        torch = _torch()
        cols = []
        for p in self.space.params:
            if p.kind == "real":
                cols.append(torch.empty(M, dtype=torch.float64, device="cuda"))
            elif p.kind == "perm":
                cols.append(torch.empty((M, p.m), dtype=torch.int32, device="cuda"))
            else:
                cols.append(torch.empty(M, dtype=torch.int32, device="cuda"))
        _check(load().gp_cot_sample(self.handle, int(M), C.c_uint64(int(seed)),
                                    C.c_uint64(int(offset)), _col_ptrs(cols), _stream()))
        return cols

    def member(self, cols):
        """gp_cot_member: uint8 CUDA mask of the configurations in the chain."""
        torch = _torch()
        M = int(cols[0].shape[0])
        mask = torch.empty(max(M, 1), dtype=torch.uint8, device="cuda")
        _check(load().gp_cot_member(self.handle, _col_ptrs(cols), M, _ptr(mask), _stream()))
        return mask[:M]


# ------------------------------------------------------------------ hidden constraints
class Forest:
    """Random-forest feasibility model on the device (gp_forest_fit)."""

    def __init__(self, space: Space, X_cols, feasible, n_trees=64, max_depth=16, min_split=2,
                 seed=0):
        lib = load()
        n = int(feasible.shape[0])
        self.space, self.n, self.n_trees = space, n, int(n_trees)
        nbytes = lib.gp_forest_workspace_bytes(space.ref(), n, self.n_trees)
        if nbytes == 0:
            raise GPError(1, "gp_forest_workspace_bytes rejected the arguments: " +
                          lib.gp_last_error().decode())
        self.workspace = _workspace(nbytes)
        h = C.c_void_p()
        _check(lib.gp_forest_fit(space.ref(), _col_ptrs(X_cols), n, _ptr(feasible),
                                 self.n_trees, int(max_depth), int(min_split),
                                 C.c_uint64(int(seed)), _ptr(self.workspace),
                                 self.workspace.numel(), _stream(), C.byref(h)))
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.gp_forest_free(self.handle)
            self.handle = None

    def predict(self, C_cols, ei=None, mask=None, eps_f=0.0):
        """gp_forest_predict: (p_feas, acq or None) as CUDA float32 tensors."""
        torch = _torch()
        M = int(C_cols[0].shape[0])
        p = torch.empty(max(M, 1), dtype=torch.float32, device="cuda")
        acq = torch.empty_like(p) if ei is not None else None
        _check(load().gp_forest_predict(self.handle, _col_ptrs(C_cols), M, _ptr(ei), _ptr(mask),
                                        C.c_float(eps_f), _ptr(p), _ptr(acq), _stream()))
        return p[:M], (acq[:M] if acq is not None else None)

    def tree(self, t):
        """(feature, left, value) numpy arrays of tree t in breadth-first node order."""
        cap = 2 * self.n
        feat = np.empty(cap, np.int32)
        left = np.empty(cap, np.int32)
        val = np.empty(cap, np.float64)
        nn = C.c_int32()
        _check(load().gp_forest_tree(self.handle, int(t), cap, C.byref(nn),
                                     feat.ctypes.data_as(_VP), left.ctypes.data_as(_VP),
                                     val.ctypes.data_as(_VP), _stream()))
        k = nn.value
        return feat[:k], left[:k], val[:k]


def refined_count(model: Model, bufs: ScoreBuffers) -> int:
    c = C.c_int64()
    _check(load().gp_score_refined_count(model.handle, _ptr(bufs.workspace), bufs.M, _stream(),
                                         C.byref(c)))
    return int(c.value)


# ------------------------------------------------------------------ inspection
def debug_encode(space: Space, cols):
    torch = _torch()
    lib = load()
    count = int(cols[0].shape[0])
    out = torch.empty(max(count * space.n_numeric, 1), dtype=torch.float32, device="cuda")
    valid = torch.empty(max(count, 1), dtype=torch.uint8, device="cuda")
    ws = _workspace(lib.gp_debug_workspace_bytes(space.ref(), None, count))
    _check(lib.gp_debug_encode(space.ref(), _col_ptrs(cols), count, _ptr(out), _ptr(valid),
                               _ptr(ws), ws.numel(), _stream()))
    return out[:count * space.n_numeric].view(count, space.n_numeric), valid[:count]


def debug_terms(model: Model, cols):
    torch = _torch()
    lib = load()
    count = int(cols[0].shape[0])
    n, d = model.info()["n"], model.space.d
    out = torch.empty(max(count * n * d, 1), dtype=torch.float32, device="cuda")
    ws = _workspace(lib.gp_debug_workspace_bytes(None, model.handle, count))
    _check(lib.gp_debug_terms(model.handle, _col_ptrs(cols), count, _ptr(out), _ptr(ws),
                              ws.numel(), _stream()))
    return out[:count * n * d].view(count, n, d)


def debug_xkernel(model: Model, cols):
    torch = _torch()
    lib = load()
    count = int(cols[0].shape[0])
    n = model.info()["n"]
    out = torch.empty(max(count * n, 1), dtype=torch.float32, device="cuda")
    ws = _workspace(lib.gp_debug_workspace_bytes(None, model.handle, count))
    _check(lib.gp_debug_xkernel(model.handle, _col_ptrs(cols), count, _ptr(out), _ptr(ws),
                                ws.numel(), _stream()))
    return out[:count * n].view(count, n)


def debug_pairs(model: Model, cols):
    """gp_debug_pairs: the production cross-kernel's per-pair r2 [count, n] and integer
    word sums [count, n, W], with the bit masks of the parameters behind each word."""
    torch = _torch()
    lib = load()
    count = int(cols[0].shape[0])
    n = model.info()["n"]
    W = C.c_int32(0)
    masks = (C.c_uint64 * 256)()
    ws = _workspace(lib.gp_debug_workspace_bytes(None, model.handle, count))
    _check(lib.gp_debug_pairs(model.handle, _col_ptrs(cols), 0, None, None, masks,
                              C.byref(W), _ptr(ws), ws.numel(), _stream()))
    nw = W.value
    r2 = torch.empty(max(count * n, 1), dtype=torch.float32, device="cuda")
    cnt = torch.empty(max(count * n * nw, 1), dtype=torch.int32, device="cuda")
    _check(lib.gp_debug_pairs(model.handle, _col_ptrs(cols), count, _ptr(r2), _ptr(cnt), None,
                              None, _ptr(ws), ws.numel(), _stream()))
    return (r2[:count * n].view(count, n), cnt[:count * n * nw].view(count, n, nw),
            [int(masks[w]) for w in range(nw)])


def debug_set_refine(model: Model, var_frac: float, sens: float):
    """Set the fp64 recomputation thresholds of later gp_score calls with `model`
    (var_frac=inf or sens<0: every valid candidate)."""
    _check(load().gp_debug_set_refine(model.handle, float(var_frac), float(sens)))


# ------------------------------------------------------------------ profiling
def profile_start():
    _check(load().gp_profile_start())


def profile_stop() -> dict:
    ms = (C.c_double * len(STAGES))()
    calls = C.c_int64()
    _check(load().gp_profile_stop(ms, C.byref(calls)))
    out = {s: ms[i] for i, s in enumerate(STAGES)}
    out["calls"] = int(calls.value)
    return out
