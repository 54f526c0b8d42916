"""Exact large-sparse-target output layer on MI355X: Python binding.

Thin ctypes binding of the C ABI declared in include/lst.h.  The functions
below carry the same names as the C entry points and only marshal arguments:
torch tensors (device memory) become pointers, torch's current HIP stream
becomes the library's stream.  Every step of the computation runs in the HIP
kernels of liblst.so; there is no other code path.  If the library has not been
built, load_library() raises instead of falling back to anything.

Classes FactoredOutputLayer and NaiveOutputLayer wrap a state handle.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "liblst.so")

LST_OK = 0
LST_EINVAL = -1
LST_EINDEX = -2
LST_ESINGULAR = -3
LST_ENOMEM = -4
LST_EHIP = -5
LST_ENONFINITE = -6
LST_ESTATE = -7
LST_ENOSCRATCH = -8

LST_LOSS_SQUARED = 0
LST_LOSS_SPHERICAL = 1
LST_LOSS_SPHERICAL_SHIFTED = 2

_LOSS = {"squared": LST_LOSS_SQUARED, "spherical": LST_LOSS_SPHERICAL,
         "spherical_shifted": LST_LOSS_SPHERICAL_SHIFTED}


class lst_config(ctypes.Structure):
    _fields_ = [
        ("loss", ctypes.c_int32),
        ("sph_eps", ctypes.c_float),
        ("m_max", ctypes.c_int32),
        ("K_max", ctypes.c_int32),
        ("cond_max", ctypes.c_float),
    ]


class lst_stats_t(ctypes.Structure):
    _fields_ = [
        ("steps", ctypes.c_int64),
        ("restores", ctypes.c_int64),
        ("last_unique", ctypes.c_int32),
        ("last_nnz", ctypes.c_int32),
    ]


class lst_stab_config(ctypes.Structure):
    _fields_ = [
        ("sigma_low", ctypes.c_float),
        ("sigma_high", ctypes.c_float),
        ("squarings", ctypes.c_int32),
        ("max_fixes", ctypes.c_int32),
        ("reinvert", ctypes.c_int32),
    ]


class lst_stab_report(ctypes.Structure):
    _fields_ = [
        ("fixes_low", ctypes.c_int32),
        ("fixes_high", ctypes.c_int32),
        ("sigma_min", ctypes.c_float),
        ("sigma_max", ctypes.c_float),
    ]


class LstError(RuntimeError):
    def __init__(self, code: int, what: str = ""):
        self.code = code
        msg = _lib.lst_strerror(code).decode() if _lib is not None else str(code)
        super().__init__(f"{what}: {msg} ({code})" if what else f"{msg} ({code})")


_lib: Optional[ctypes.CDLL] = None

_P = ctypes.c_void_p
_SIGS = {
    "lst_init": (ctypes.c_int, [ctypes.POINTER(_P), ctypes.c_int64, ctypes.c_int32, _P, _P,
                                ctypes.POINTER(lst_config), _P]),
    "lst_step": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P, _P, _P, ctypes.c_float,
                                _P, _P]),
    "lst_step_solve": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P, _P, _P,
                                      ctypes.c_float, _P, _P]),
    "lst_materialize_W": (ctypes.c_int, [_P, _P]),
    "lst_get_state": (ctypes.c_int, [_P, _P, _P, _P]),
    "lst_get_V": (ctypes.c_int, [_P, _P]),
    "lst_get_shift": (ctypes.c_int, [_P, _P, _P]),
    "lst_touched_rows": (ctypes.c_int, [_P, _P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]),
    "lst_restore": (ctypes.c_int, [_P]),
    "lst_stabilize": (ctypes.c_int, [_P, ctypes.POINTER(lst_stab_config),
                                     ctypes.POINTER(lst_stab_report)]),
    "lst_stabilize_noalloc": (ctypes.c_int, [_P, ctypes.POINTER(lst_stab_config),
                                             ctypes.POINTER(lst_stab_report)]),
    "lst_set_stabilize": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.POINTER(lst_stab_config)]),
    "lst_naive_init": (ctypes.c_int, [ctypes.POINTER(_P), ctypes.c_int64, ctypes.c_int32, _P,
                                      ctypes.POINTER(lst_config), _P]),
    "lst_naive_step": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P, _P, _P,
                                      ctypes.c_float, _P, _P]),
    "lst_sync": (ctypes.c_int, [_P]),
    "lst_set_graphs": (ctypes.c_int, [_P, ctypes.c_int32]),
    "lst_set_split_tasks": (ctypes.c_int, [_P, ctypes.c_int32]),
    "lst_stats": (ctypes.c_int, [_P, ctypes.POINTER(lst_stats_t)]),
    "lst_profile_enable": (ctypes.c_int, [_P, ctypes.c_int32]),
    "lst_profile_read": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_double), ctypes.c_int32,
                                        ctypes.POINTER(ctypes.c_int32),
                                        ctypes.POINTER(ctypes.c_int64)]),
    "lst_profile_phase_name": (ctypes.c_char_p, [ctypes.c_int32]),
    "lst_input_init": (ctypes.c_int, [ctypes.POINTER(_P), ctypes.c_int64, ctypes.c_int32, _P, _P]),
    "lst_input_forward": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P, _P, _P]),
    "lst_input_update": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P, _P, _P,
                                        ctypes.c_float]),
    "lst_input_get_W": (ctypes.c_int, [_P, _P]),
    "lst_input_sync": (ctypes.c_int, [_P]),
    "lst_input_free": (None, [_P]),
    "lst_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "lst_free": (None, [_P]),
}

EXPORTED = tuple(_SIGS)


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load liblst.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} not found: build the HIP library first (python -m paper_1412_7091_amd.build)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(code: int, what: str) -> None:
    if code != LST_OK:
        raise LstError(code, what)


def _ptr(t, dtype, what: str):
    """Device pointer of a contiguous CUDA tensor of the given dtype (None -> NULL)."""
    import torch

    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{what} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream_handle(stream=None):
    import torch

    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _config(loss: str, sph_eps: float, m_max: int, K_max: int, cond_max: float) -> lst_config:
    if loss not in _LOSS:
        raise ValueError(f"loss must be one of {sorted(_LOSS)}")
    return lst_config(_LOSS[loss], float(sph_eps), int(m_max), int(K_max), float(cond_max))


# ----------------------------------------------------------- C-named wrappers
def lst_init(V, U=None, *, loss="squared", sph_eps=1e-3, m_max=128, K_max=16, cond_max=0.0,
             stream=None):
    """Create a factored state from device tensors V (D x d) and U (d x d or None)."""
    import torch

    lib = load_library()
    D, d = V.shape
    cfg = _config(loss, sph_eps, m_max, K_max, cond_max)
    h = _P()
    _check(lib.lst_init(ctypes.byref(h), D, d, _ptr(V, torch.float32, "V"),
                        _ptr(U, torch.float32, "U"), ctypes.byref(cfg), _stream_handle(stream)),
           "lst_init")
    return h


def lst_naive_init(W, *, loss="squared", sph_eps=1e-3, m_max=128, K_max=16, stream=None):
    import torch

    lib = load_library()
    D, d = W.shape
    cfg = _config(loss, sph_eps, m_max, K_max, 0.0)
    h = _P()
    _check(lib.lst_naive_init(ctypes.byref(h), D, d, _ptr(W, torch.float32, "W"),
                              ctypes.byref(cfg), _stream_handle(stream)), "lst_naive_init")
    return h


def _step(fn_name, h, H, Y_idx, Y_val, lr, loss_out, grad_out):
    import torch

    m, d = H.shape
    K = Y_idx.shape[1]
    if Y_idx.shape[0] != m or (Y_val is not None and tuple(Y_val.shape) != tuple(Y_idx.shape)):
        raise ValueError("H, Y_idx and Y_val disagree on m / K")
    if tuple(loss_out.shape) != (m,) or tuple(grad_out.shape) != (m, d):
        raise ValueError("loss must be (m,) and grad_H (m, d)")
    fn = getattr(load_library(), fn_name)
    _check(fn(h, m, K, _ptr(H, torch.float32, "H"), _ptr(Y_idx, torch.int32, "Y_idx"),
              _ptr(Y_val, torch.float32, "Y_val"), float(lr),
              _ptr(loss_out, torch.float32, "loss"), _ptr(grad_out, torch.float32, "grad_H")),
           fn_name)


def lst_step(h, H, Y_idx, Y_val, lr, loss_out, grad_out):
    _step("lst_step", h, H, Y_idx, Y_val, lr, loss_out, grad_out)


def lst_step_solve(h, H, Y_idx, Y_val, lr, loss_out, grad_out):
    _step("lst_step_solve", h, H, Y_idx, Y_val, lr, loss_out, grad_out)


def lst_naive_step(h, H, Y_idx, Y_val, lr, loss_out, grad_out):
    _step("lst_naive_step", h, H, Y_idx, Y_val, lr, loss_out, grad_out)


def lst_materialize_W(h, W_out):
    import torch

    _check(load_library().lst_materialize_W(h, _ptr(W_out, torch.float32, "W")),
           "lst_materialize_W")


def lst_get_state(h, Q=None, U=None, UinvT=None):
    import torch

    _check(load_library().lst_get_state(h, _ptr(Q, torch.float32, "Q"),
                                        _ptr(U, torch.float32, "U"),
                                        _ptr(UinvT, torch.float32, "UinvT")), "lst_get_state")


def lst_get_V(h, V_out):
    import torch

    _check(load_library().lst_get_V(h, _ptr(V_out, torch.float32, "V")), "lst_get_V")


def lst_get_shift(h, c_out=None, s_out=None):
    import torch

    _check(load_library().lst_get_shift(h, _ptr(c_out, torch.float32, "c"),
                                        _ptr(s_out, torch.float32, "s")), "lst_get_shift")


def lst_touched_rows(h, capacity: int):
    import numpy as np

    buf = (ctypes.c_int32 * max(1, capacity))()
    n = ctypes.c_int32(0)
    _check(load_library().lst_touched_rows(h, buf, capacity, ctypes.byref(n)), "lst_touched_rows")
    return np.frombuffer(buf, dtype=np.int32, count=n.value).copy()


def lst_restore(h):
    _check(load_library().lst_restore(h), "lst_restore")


def _stab_config(sigma_low, sigma_high, squarings, max_fixes, reinvert) -> lst_stab_config:
    return lst_stab_config(float(sigma_low), float(sigma_high), int(squarings), int(max_fixes),
                           int(reinvert))


def lst_stabilize(h, sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=2, reinvert=1,
                  report=True):
    """Appendix C correction of out-of-range singular values of U.  With report, synchronises
    and returns the lst_stab_report; else enqueues and returns None."""
    cfg = _stab_config(sigma_low, sigma_high, squarings, max_fixes, reinvert)
    rep = lst_stab_report() if report else None
    _check(load_library().lst_stabilize(h, ctypes.byref(cfg),
                                        ctypes.byref(rep) if rep is not None else None),
           "lst_stabilize")
    return rep


def lst_stabilize_noalloc(h, sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=2,
                          reinvert=1, report=True):
    """lst_stabilize on the library's static workspace (no device allocation)."""
    cfg = _stab_config(sigma_low, sigma_high, squarings, max_fixes, reinvert)
    rep = lst_stab_report() if report else None
    _check(load_library().lst_stabilize_noalloc(h, ctypes.byref(cfg),
                                                ctypes.byref(rep) if rep is not None else None),
           "lst_stabilize_noalloc")
    return rep


def lst_set_stabilize(h, every, sigma_low=1e-3, sigma_high=100.0, squarings=7, max_fixes=2,
                      reinvert=1):
    cfg = _stab_config(sigma_low, sigma_high, squarings, max_fixes, reinvert)
    _check(load_library().lst_set_stabilize(h, int(every), ctypes.byref(cfg)),
           "lst_set_stabilize")


def lst_sync(h) -> int:
    """Wait for the state's stream; returns (and clears) the sticky device status code."""
    return int(load_library().lst_sync(h))


def lst_set_graphs(h, enable: bool = True) -> None:
    _check(load_library().lst_set_graphs(h, 1 if enable else 0), "lst_set_graphs")


def lst_set_split_tasks(h, enable: bool = True) -> None:
    _check(load_library().lst_set_split_tasks(h, 1 if enable else 0), "lst_set_split_tasks")


def lst_stats(h) -> lst_stats_t:
    st = lst_stats_t()
    _check(load_library().lst_stats(h, ctypes.byref(st)), "lst_stats")
    return st


def lst_profile_enable(h, enable: bool = True) -> None:
    _check(load_library().lst_profile_enable(h, 1 if enable else 0), "lst_profile_enable")


def lst_profile_read(h):
    """{phase name: summed milliseconds} over the profiled steps, and the step count."""
    lib = load_library()
    buf = (ctypes.c_double * 64)()
    n = ctypes.c_int32(0)
    steps = ctypes.c_int64(0)
    _check(lib.lst_profile_read(h, buf, 64, ctypes.byref(n), ctypes.byref(steps)),
           "lst_profile_read")
    return {lib.lst_profile_phase_name(i).decode(): buf[i] for i in range(n.value)}, steps.value


def lst_profile_phase_name(i: int):
    r = load_library().lst_profile_phase_name(i)
    return None if r is None else r.decode()


def lst_strerror(code: int) -> str:
    return load_library().lst_strerror(code).decode()


def lst_free(h) -> None:
    if h is not None and h.value:
        load_library().lst_free(h)


# ------------------------------------------------------------------- classes
class _Layer:
    def __init__(self, handle, D: int, d: int, m_max: int, K_max: int, device):
        self._h = handle
        self.D, self.d = D, d
        self.m_max, self.K_max = m_max, K_max
        self.device = device

    def _alloc_outputs(self, m):
        import torch

        return (torch.empty(m, dtype=torch.float32, device=self.device),
                torch.empty((m, self.d), dtype=torch.float32, device=self.device))

    def materialize_W(self, out=None):
        import torch

        if out is None:
            out = torch.empty((self.D, self.d), dtype=torch.float32, device=self.device)
        lst_materialize_W(self._h, out)
        return out

    def sync(self) -> int:
        return lst_sync(self._h)

    def set_graphs(self, enable: bool = True) -> None:
        lst_set_graphs(self._h, enable)

    def profile(self, enable: bool = True) -> None:
        lst_profile_enable(self._h, enable)

    def profile_read(self):
        return lst_profile_read(self._h)

    def stats(self) -> lst_stats_t:
        return lst_stats(self._h)

    def close(self) -> None:
        if self._h is not None:
            lst_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class FactoredOutputLayer(_Layer):
    """W = V U with Q = W^T W and U^{-T} kept up to date (section 3 of the paper)."""

    def __init__(self, V, U=None, *, loss="squared", sph_eps=1e-3, m_max=128, K_max=16,
                 cond_max=0.0, stream=None):
        h = lst_init(V, U, loss=loss, sph_eps=sph_eps, m_max=m_max, K_max=K_max,
                     cond_max=cond_max, stream=stream)
        super().__init__(h, V.shape[0], V.shape[1], m_max, K_max, V.device)

    def step(self, H, Y_idx, Y_val, lr, out: Optional[Tuple] = None):
        loss, grad = out if out is not None else self._alloc_outputs(H.shape[0])
        lst_step(self._h, H, Y_idx, Y_val, lr, loss, grad)
        return loss, grad

    def step_solve(self, H, Y_idx, Y_val, lr, out: Optional[Tuple] = None):
        """The step with U_new^T Z = H solved from scratch (lst_step_solve)."""
        loss, grad = out if out is not None else self._alloc_outputs(H.shape[0])
        lst_step_solve(self._h, H, Y_idx, Y_val, lr, loss, grad)
        return loss, grad

    def get_state(self):
        import torch

        Q, U, Uit = (torch.empty((self.d, self.d), dtype=torch.float32, device=self.device)
                     for _ in range(3))
        lst_get_state(self._h, Q, U, Uit)
        return Q, U, Uit

    def get_V(self):
        import torch

        V = torch.empty((self.D, self.d), dtype=torch.float32, device=self.device)
        lst_get_V(self._h, V)
        return V

    def get_shift(self):
        """(c, s) of the shifted spherical loss: W = V U + 1 c^T, s = W^T 1."""
        import torch

        c, s = (torch.empty(self.d, dtype=torch.float32, device=self.device) for _ in range(2))
        lst_get_shift(self._h, c, s)
        return c, s

    def touched_rows(self):
        return lst_touched_rows(self._h, self.m_max * self.K_max)

    def restore(self):
        lst_restore(self._h)

    def set_split_tasks(self, enable: bool = True) -> None:
        lst_set_split_tasks(self._h, enable)

    def stabilize(self, **kw):
        return lst_stabilize(self._h, **kw)

    def stabilize_noalloc(self, **kw):
        return lst_stabilize_noalloc(self._h, **kw)

    def set_stabilize(self, every: int, **kw) -> None:
        lst_set_stabilize(self._h, every, **kw)


class SparseInputLayer:
    """Section 2.2 input layer: W_in (D_in x d) with K-sparse inputs."""

    def __init__(self, W_in, stream=None):
        import torch

        lib = load_library()
        self.D, self.d = W_in.shape
        self.device = W_in.device
        h = _P()
        _check(lib.lst_input_init(ctypes.byref(h), self.D, self.d,
                                  _ptr(W_in, torch.float32, "W_in"), _stream_handle(stream)),
               "lst_input_init")
        self._h = h

    def forward(self, idx, val, out=None):
        import torch

        m, K = idx.shape
        if out is None:
            out = torch.empty((m, self.d), dtype=torch.float32, device=self.device)
        _check(load_library().lst_input_forward(self._h, m, K, _ptr(idx, torch.int32, "idx"),
                                                _ptr(val, torch.float32, "val"),
                                                _ptr(out, torch.float32, "A")), "lst_input_forward")
        return out

    def update(self, idx, val, grad_A, lr):
        import torch

        m, K = idx.shape
        if tuple(grad_A.shape) != (m, self.d):
            raise ValueError("grad_A must be (m, d)")
        _check(load_library().lst_input_update(self._h, m, K, _ptr(idx, torch.int32, "idx"),
                                               _ptr(val, torch.float32, "val"),
                                               _ptr(grad_A, torch.float32, "grad_A"), float(lr)),
               "lst_input_update")

    def get_W(self):
        import torch

        W = torch.empty((self.D, self.d), dtype=torch.float32, device=self.device)
        _check(load_library().lst_input_get_W(self._h, _ptr(W, torch.float32, "W")),
               "lst_input_get_W")
        return W

    def sync(self) -> int:
        return int(load_library().lst_input_sync(self._h))

    def close(self) -> None:
        if self._h is not None:
            load_library().lst_input_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class NaiveOutputLayer(_Layer):
    """Explicit W (the O(D d) per example computation), same library and kernels."""

    def __init__(self, W, *, loss="squared", sph_eps=1e-3, m_max=128, K_max=16, stream=None):
        h = lst_naive_init(W, loss=loss, sph_eps=sph_eps, m_max=m_max, K_max=K_max, stream=stream)
        super().__init__(h, W.shape[0], W.shape[1], m_max, K_max, W.device)

    def step(self, H, Y_idx, Y_val, lr, out: Optional[Tuple] = None):
        loss, grad = out if out is not None else self._alloc_outputs(H.shape[0])
        lst_naive_step(self._h, H, Y_idx, Y_val, lr, loss, grad)
        return loss, grad
