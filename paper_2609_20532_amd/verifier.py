"""Python binding of the CPU verifier in ``include/dpsgd_verifier.h``
(argument marshalling only).

Every function has the name of the C entry point it calls. Tensors are host
numpy arrays: activations / output gradients as float32 or as bfloat16 bit
patterns (uint16), gradients as float32 (or float64 for the float64
recomputation), all C-contiguous. The library must be built
(``paper_2609_20532_amd.build``); loading fails loudly when it is missing.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

from .dpsgd import DPSGD_BF16, DPSGD_F32, dpsgd_layer

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdpsgd_verifier.so")

DPSGD_ERR_ABORTED = -5
DPSGD_VERIFY_ACCEPT, DPSGD_VERIFY_ABORT = 0, 1
(DPSGD_PATH_STRUCTURAL, DPSGD_PATH_UNCHECKED, DPSGD_PATH_BODY, DPSGD_PATH_AMBIGUITY,
 DPSGD_PATH_HARD) = range(5)

#: Every symbol the header declares (checked by the CPU test suite).
EXPORTED = ("dpsgd_verifier_init", "dpsgd_reference_mean_f32", "dpsgd_reference_mean_f64",
            "dpsgd_verify_step")


class VerifierError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed (status {status})")
        self.status = status


class dpsgd_verifier_params(ctypes.Structure):  # noqa: N801 - mirrors the C struct
    _fields_ = [("p", ctypes.c_double), ("tau_abs", ctypes.c_double),
                ("rho_amb", ctypes.c_double), ("rho_ill", ctypes.c_double),
                ("K_sub", ctypes.c_double), ("K_amb", ctypes.c_int64), ("C", ctypes.c_double),
                ("B", ctypes.c_int64), ("norm_slack", ctypes.c_double)]


class dpsgd_verifier_state(ctypes.Structure):  # noqa: N801
    _fields_ = [("Z_sub", ctypes.c_double), ("S_amb", ctypes.c_int64), ("steps", ctypes.c_int64),
                ("checked", ctypes.c_int64), ("aborted", ctypes.c_int32), ("pad", ctypes.c_int32)]


class dpsgd_verify_result(ctypes.Structure):  # noqa: N801
    _fields_ = [("decision", ctypes.c_int32), ("path", ctypes.c_int32), ("norm", ctypes.c_double),
                ("z32", ctypes.c_double), ("n_t", ctypes.c_double)]


_lib = None


def load(path: str | None = None):
    global _lib
    if _lib is not None:
        return _lib
    path = path or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_20532_amd.build`")
    lib = ctypes.CDLL(path)
    P, vp, i32, i64 = ctypes.POINTER, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    L = P(dpsgd_layer)
    sig = {
        "dpsgd_verifier_init": (ctypes.c_int, [P(dpsgd_verifier_params), P(dpsgd_verifier_state)]),
        "dpsgd_reference_mean_f32": (ctypes.c_int, [L, i32, ctypes.c_float, i64, P(vp), i32]),
        "dpsgd_reference_mean_f64": (ctypes.c_int, [L, i32, ctypes.c_double, i64, P(vp), i32]),
        "dpsgd_verify_step": (ctypes.c_int, [P(dpsgd_verifier_params), P(dpsgd_verifier_state),
                                             L, i32, P(vp), i32, i32, P(dpsgd_verify_result)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


@dataclass
class HostLayer:
    """Host copy of one layer (keeps the arrays the descriptor points at alive)."""

    A: np.ndarray
    G: np.ndarray
    desc: dpsgd_layer


def host_layer(A: np.ndarray, G: np.ndarray, tensor_id: int = 0) -> HostLayer:
    """Descriptor of a layer from host arrays A [B,T,d_in], G [B,T,d_out]:
    float32, or uint16 holding bfloat16 bit patterns."""
    if A.dtype != G.dtype or A.dtype not in (np.float32, np.uint16):
        raise ValueError("A and G must both be float32 or both uint16 (bfloat16 bits)")
    if A.ndim != 3 or G.ndim != 3 or A.shape[:2] != G.shape[:2]:
        raise ValueError("A and G must be [B, T, d] with the same B and T")
    A = np.ascontiguousarray(A)
    G = np.ascontiguousarray(G)
    B, T, d_in = A.shape
    desc = dpsgd_layer(A.ctypes.data, G.ctypes.data, B, T, d_in, G.shape[2],
                       DPSGD_BF16 if A.dtype == np.uint16 else DPSGD_F32, tensor_id)
    return HostLayer(A, G, desc)


def _descs(layers):
    arr = (dpsgd_layer * len(layers))(*[h.desc for h in layers])
    return arr, len(layers)


def _ptrs(arrays):
    return (ctypes.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])


def make_params(tau_abs, K_sub, K_amb, C, B, rho_amb=0.0, rho_ill=0.0, p=0.1,
                norm_slack=1e-4) -> dpsgd_verifier_params:
    return dpsgd_verifier_params(p=p, tau_abs=tau_abs, rho_amb=rho_amb, rho_ill=rho_ill,
                                 K_sub=K_sub, K_amb=K_amb, C=C, B=B, norm_slack=norm_slack)


def dpsgd_verifier_init(params: dpsgd_verifier_params) -> dpsgd_verifier_state:
    lib = load()
    st = dpsgd_verifier_state()
    s = lib.dpsgd_verifier_init(ctypes.byref(params), ctypes.byref(st))
    if s != 0:
        raise VerifierError("dpsgd_verifier_init", s)
    return st


def _reference(name, dtype, layers, C, B, threads):
    lib = load()
    arr, n = _descs(layers)
    outs = [np.empty((h.desc.d_out, h.desc.d_in), dtype=dtype) for h in layers]
    s = getattr(lib, name)(arr, n, C, B, _ptrs(outs), threads)
    if s != 0:
        raise VerifierError(name, s)
    return outs


def dpsgd_reference_mean_f32(layers, C, B, threads=0):
    return _reference("dpsgd_reference_mean_f32", np.float32, layers, C, B, threads)


def dpsgd_reference_mean_f64(layers, C, B, threads=0):
    return _reference("dpsgd_reference_mean_f64", np.float64, layers, C, B, threads)


def dpsgd_verify_step(params, state, layers, g_gpu, coin, threads=0) -> dpsgd_verify_result:
    """Raises VerifierError with status DPSGD_ERR_ABORTED once the run is aborted."""
    lib = load()
    arr, n = _descs(layers)
    g = [np.ascontiguousarray(x, dtype=np.float32) for x in g_gpu]
    for x, h in zip(g, layers):
        if x.shape != (h.desc.d_out, h.desc.d_in):
            raise ValueError("each submission array must be [d_out, d_in] of its layer")
    res = dpsgd_verify_result()
    s = lib.dpsgd_verify_step(ctypes.byref(params), ctypes.byref(state), arr, n, _ptrs(g),
                              int(bool(coin)), threads, ctypes.byref(res))
    if s != 0:
        raise VerifierError("dpsgd_verify_step", s)
    return res
