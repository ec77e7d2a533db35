"""Python binding of the C ABI in ``include/dpsgd.h`` (argument marshalling only).

Every function here has the name of the C entry point it calls and does no
arithmetic of the DP-SGD step: it converts torch tensors to device pointers,
fills ``dpsgd_layer`` descriptors, passes torch's current HIP stream, and
raises :class:`DpsgdError` on a non-zero status. torch supplies device memory
and streams only. The library must be built (``paper_2609_20532_amd.build``);
loading fails loudly when it is missing.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdpsgd.so")

DPSGD_F32 = 0
DPSGD_BF16 = 1
DPSGD_NORM_AUTO = 0
DPSGD_NORM_GHOST = 1
DPSGD_NORM_MATERIALIZE = 2
DPSGD_NORM_CLOSED_FORM = 3   # reported by dpsgd_select_norm_mode for T = 1 layers

DPSGD_OK = 0
DPSGD_ERR_INVALID_ARG = -1
DPSGD_ERR_UNSUPPORTED = -2
DPSGD_ERR_WORKSPACE = -3
DPSGD_ERR_HIP = -4

#: Every symbol the header declares (checked by the CPU test suite).
EXPORTED = (
    "dpsgd_norms_workspace_bytes", "dpsgd_select_norm_mode", "dpsgd_per_example_norms",
    "dpsgd_per_example_norms_multi", "dpsgd_per_example_norms_multi_noalloc",
    "dpsgd_clip_factors", "dpsgd_clip_workspace_bytes",
    "dpsgd_clip_accumulate", "dpsgd_clip_accumulate_multi", "dpsgd_clipped_sum_workspace_bytes",
    "dpsgd_clipped_sum_multi", "dpsgd_add_noise",
    "dpsgd_add_noise_multi", "dpsgd_noise_adamw", "dpsgd_noise_adamw_multi",
    "dpsgd_philox_u32", "dpsgd_gaussian", "dpsgd_status_string", "dpsgd_version",
)


class DpsgdError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__(f"{fn} failed: {text} (status {status})")
        self.status = status


class dpsgd_layer(ctypes.Structure):  # noqa: N801 - mirrors the C struct name
    _fields_ = [
        ("A", ctypes.c_void_p),
        ("G", ctypes.c_void_p),
        ("B", ctypes.c_int64),
        ("T", ctypes.c_int64),
        ("d_in", ctypes.c_int64),
        ("d_out", ctypes.c_int64),
        ("dtype", ctypes.c_int32),
        ("tensor_id", ctypes.c_uint32),
    ]


class dpsgd_adamw(ctypes.Structure):  # noqa: N801 - mirrors the C struct name
    _fields_ = [
        ("lr", ctypes.c_float),
        ("beta1", ctypes.c_float),
        ("beta2", ctypes.c_float),
        ("eps", ctypes.c_float),
        ("weight_decay", ctypes.c_float),
        ("t", ctypes.c_uint32),
    ]


_lib = None


def _declare(lib):
    P = ctypes.POINTER
    L = P(dpsgd_layer)
    vp, i32, i64, u32, u64, f32, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                       ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float,
                                       ctypes.c_size_t)
    sig = {
        "dpsgd_norms_workspace_bytes": (sz, [L, i32, i32]),
        "dpsgd_select_norm_mode": (i32, [L]),
        "dpsgd_per_example_norms": (ctypes.c_int, [L, i32, vp, i32, vp, sz, vp]),
        "dpsgd_per_example_norms_multi": (ctypes.c_int, [L, i32, i32, vp, i32, vp, sz, vp]),
        "dpsgd_per_example_norms_multi_noalloc": (ctypes.c_int, [L, i32, i32, vp, i32, vp]),
        "dpsgd_clip_factors": (ctypes.c_int, [vp, i64, f32, vp, vp, vp]),
        "dpsgd_clip_workspace_bytes": (sz, [L, i32]),
        "dpsgd_clip_accumulate": (ctypes.c_int, [L, vp, f32, vp, i32, vp, vp, vp, sz, vp]),
        "dpsgd_clip_accumulate_multi": (ctypes.c_int,
                                        [L, i32, vp, f32, P(vp), i32, vp, vp, vp, sz, vp]),
        "dpsgd_clipped_sum_workspace_bytes": (sz, [L, i32, i32]),
        "dpsgd_clipped_sum_multi": (ctypes.c_int, [L, i32, i32, f32, P(vp), i32, vp, vp, vp, vp,
                                                   sz, vp]),
        "dpsgd_add_noise": (ctypes.c_int, [L, vp, f32, f32, u64, u32, f32, vp]),
        "dpsgd_add_noise_multi": (ctypes.c_int, [L, i32, P(vp), f32, f32, u64, u32, f32, vp]),
        "dpsgd_noise_adamw": (ctypes.c_int, [L, vp, vp, vp, vp, vp, f32, f32, u64, u32, f32,
                                             P(dpsgd_adamw), vp]),
        "dpsgd_noise_adamw_multi": (ctypes.c_int, [L, i32, P(vp), P(vp), P(vp), P(vp), P(vp),
                                                   f32, f32, u64, u32, f32, P(dpsgd_adamw), vp]),
        "dpsgd_philox_u32": (ctypes.c_int, [vp, i64, i64, u64, u32, u32, vp]),
        "dpsgd_gaussian": (ctypes.c_int, [vp, i64, u64, u32, u32, vp]),
        "dpsgd_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "dpsgd_version": (ctypes.c_int, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args


def load(path: str | None = None):
    """Load ``libdpsgd.so`` (after torch, so both share one HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (loads the HIP runtime the library links against)

    path = path or LIB_PATH
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2609_20532_amd.build`")
    lib = ctypes.CDLL(path)
    _declare(lib)
    if lib.dpsgd_version() != 1:
        raise RuntimeError("libdpsgd version mismatch")
    _lib = lib
    return lib


def _check(fn: str, status: int):
    if status != DPSGD_OK:
        raise DpsgdError(fn, status, _lib.dpsgd_status_string(status).decode())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


# ----------------------------------------------------------------- descriptors


def make_layer(A, G, tensor_id: int) -> dpsgd_layer:
    """Descriptor of one layer from device tensors A [B,T,d_in] and G [B,T,d_out].

    ``tensor_id`` selects the layer's noise stream: the layers of one step
    need distinct ids (the noise calls reject repeats)."""
    import torch
    if A.dim() != 3 or G.dim() != 3 or A.shape[:2] != G.shape[:2]:
        raise ValueError("A must be [B,T,d_in] and G [B,T,d_out] with the same B, T")
    if A.dtype != G.dtype or A.dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("A and G must both be float32 or both bfloat16")
    if not (A.is_contiguous() and G.is_contiguous()):
        raise ValueError("A and G must be contiguous")
    if not (A.is_cuda and G.is_cuda):
        raise ValueError("A and G must be device tensors")
    B, T, d_in = A.shape
    return dpsgd_layer(A.data_ptr(), G.data_ptr(), B, T, d_in, G.shape[2],
                       DPSGD_BF16 if A.dtype == torch.bfloat16 else DPSGD_F32, tensor_id)


def shape_layer(B: int, T: int, d_in: int, d_out: int, dtype: int = DPSGD_BF16,
                tensor_id: int = 0) -> dpsgd_layer:
    """Descriptor with no data, for workspace queries and noise calls."""
    return dpsgd_layer(None, None, B, T, d_in, d_out, dtype, tensor_id)


def _array(layers):
    if isinstance(layers, dpsgd_layer):
        layers = [layers]
    arr = (dpsgd_layer * len(layers))(*layers)
    return arr, len(layers)


def _ptr_array(tensors):
    return (ctypes.c_void_p * len(tensors))(*[None if t is None else t.data_ptr() for t in tensors])


# ------------------------------------------------------------- entry points


def dpsgd_norms_workspace_bytes(layers, mode: int = DPSGD_NORM_AUTO) -> int:
    load()
    arr, n = _array(layers)
    return int(_lib.dpsgd_norms_workspace_bytes(arr, n, mode))


def dpsgd_select_norm_mode(layer: dpsgd_layer) -> int:
    load()
    r = int(_lib.dpsgd_select_norm_mode(ctypes.byref(layer)))
    if r < 0:
        _check("dpsgd_select_norm_mode", r)
    return r


def dpsgd_per_example_norms(layer, mode, norms_sq, accumulate=False, workspace=None,
                            stream=None):
    load()
    st = _lib.dpsgd_per_example_norms(ctypes.byref(layer), mode, _ptr(norms_sq), int(accumulate),
                                      _ptr(workspace),
                                      0 if workspace is None else workspace.numel(),
                                      _stream(stream))
    _check("dpsgd_per_example_norms", st)


def dpsgd_per_example_norms_multi(layers, mode, norms_sq, accumulate=False, workspace=None,
                                  stream=None):
    load()
    arr, n = _array(layers)
    st = _lib.dpsgd_per_example_norms_multi(arr, n, mode, _ptr(norms_sq), int(accumulate),
                                            _ptr(workspace),
                                            0 if workspace is None else workspace.numel(),
                                            _stream(stream))
    _check("dpsgd_per_example_norms_multi", st)


#: Bytes of the scratch array of dpsgd_per_example_norms_multi_noalloc.
DPSGD_NOALLOC_SCRATCH_BYTES = 8 << 20


def dpsgd_per_example_norms_multi_noalloc(layers, mode, norms_sq, accumulate=False, stream=None):
    load()
    arr, n = _array(layers)
    st = _lib.dpsgd_per_example_norms_multi_noalloc(arr, n, mode, _ptr(norms_sq), int(accumulate),
                                                    _stream(stream))
    _check("dpsgd_per_example_norms_multi_noalloc", st)


def dpsgd_clip_factors(norms_sq, C: float, factors=None, mask=None, stream=None):
    load()
    st = _lib.dpsgd_clip_factors(_ptr(norms_sq), norms_sq.numel(), C, _ptr(factors), _ptr(mask),
                                 _stream(stream))
    _check("dpsgd_clip_factors", st)


def dpsgd_clip_workspace_bytes(layers) -> int:
    load()
    arr, n = _array(layers)
    return int(_lib.dpsgd_clip_workspace_bytes(arr, n))


def dpsgd_clip_accumulate(layer, norms_sq, C, grad, accumulate=False, factors_out=None,
                          mask_out=None, workspace=None, stream=None):
    load()
    st = _lib.dpsgd_clip_accumulate(ctypes.byref(layer), _ptr(norms_sq), C, _ptr(grad),
                                    int(accumulate), _ptr(factors_out), _ptr(mask_out),
                                    _ptr(workspace), 0 if workspace is None else workspace.numel(),
                                    _stream(stream))
    _check("dpsgd_clip_accumulate", st)


def dpsgd_clip_accumulate_multi(layers, norms_sq, C, grads, accumulate=False, factors_out=None,
                                mask_out=None, workspace=None, stream=None):
    load()
    arr, n = _array(layers)
    st = _lib.dpsgd_clip_accumulate_multi(arr, n, _ptr(norms_sq), C, _ptr_array(grads),
                                          int(accumulate), _ptr(factors_out), _ptr(mask_out),
                                          _ptr(workspace),
                                          0 if workspace is None else workspace.numel(),
                                          _stream(stream))
    _check("dpsgd_clip_accumulate_multi", st)


def dpsgd_clipped_sum_workspace_bytes(layers, mode: int = DPSGD_NORM_AUTO) -> int:
    load()
    arr, n = _array(layers)
    return int(_lib.dpsgd_clipped_sum_workspace_bytes(arr, n, mode))


def dpsgd_clipped_sum_multi(layers, mode, C, grads, norms_sq, accumulate=False, factors_out=None,
                            mask_out=None, workspace=None, stream=None):
    load()
    arr, n = _array(layers)
    st = _lib.dpsgd_clipped_sum_multi(arr, n, mode, C, _ptr_array(grads), int(accumulate),
                                      _ptr(norms_sq), _ptr(factors_out), _ptr(mask_out),
                                      _ptr(workspace),
                                      0 if workspace is None else workspace.numel(),
                                      _stream(stream))
    _check("dpsgd_clipped_sum_multi", st)


def dpsgd_add_noise(layer, grad, sigma, C, seed, step, scale, stream=None):
    load()
    st = _lib.dpsgd_add_noise(ctypes.byref(layer), _ptr(grad), sigma, C, seed, step, scale,
                              _stream(stream))
    _check("dpsgd_add_noise", st)


def dpsgd_add_noise_multi(layers, grads, sigma, C, seed, step, scale, stream=None):
    load()
    arr, n = _array(layers)
    st = _lib.dpsgd_add_noise_multi(arr, n, _ptr_array(grads), sigma, C, seed, step, scale,
                                    _stream(stream))
    _check("dpsgd_add_noise_multi", st)


def make_adamw(lr, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, t=1) -> dpsgd_adamw:
    return dpsgd_adamw(lr=lr, beta1=beta1, beta2=beta2, eps=eps, weight_decay=weight_decay, t=t)


def dpsgd_noise_adamw(layer, grad, param, exp_avg, exp_avg_sq, sigma, C, seed, step, scale, opt,
                      noisy_out=None, stream=None):
    load()
    st = _lib.dpsgd_noise_adamw(ctypes.byref(layer), _ptr(grad), _ptr(param), _ptr(exp_avg),
                                _ptr(exp_avg_sq), _ptr(noisy_out), sigma, C, seed, step, scale,
                                ctypes.byref(opt), _stream(stream))
    _check("dpsgd_noise_adamw", st)


def dpsgd_noise_adamw_multi(layers, grads, params, exp_avgs, exp_avg_sqs, sigma, C, seed, step,
                            scale, opt, noisy_outs=None, stream=None):
    load()
    arr, n = _array(layers)
    st = _lib.dpsgd_noise_adamw_multi(arr, n, _ptr_array(grads), _ptr_array(params),
                                      _ptr_array(exp_avgs), _ptr_array(exp_avg_sqs),
                                      None if noisy_outs is None else _ptr_array(noisy_outs),
                                      sigma, C, seed, step, scale, ctypes.byref(opt),
                                      _stream(stream))
    _check("dpsgd_noise_adamw_multi", st)


def dpsgd_philox_u32(out, first_block, n_blocks, seed, tensor_id, step, stream=None):
    load()
    st = _lib.dpsgd_philox_u32(_ptr(out), first_block, n_blocks, seed, tensor_id, step,
                               _stream(stream))
    _check("dpsgd_philox_u32", st)


def dpsgd_gaussian(out, n, seed, tensor_id, step, stream=None):
    load()
    st = _lib.dpsgd_gaussian(_ptr(out), n, seed, tensor_id, step, _stream(stream))
    _check("dpsgd_gaussian", st)


# ------------------------------------------------------------ whole step


@dataclass
class StepBuffers:
    """Device buffers of one step: norms, factors, mask, workspaces, grads."""

    norms_sq: object
    factors: object
    mask: object
    norms_ws: object
    clip_ws: object
    grads: list
    fused_ws: object = None   # workspace of dpsgd_clipped_sum_multi (alloc_step(fused=True))


def alloc_step(layers, mode: int = DPSGD_NORM_AUTO, device="cuda", fused: bool = False) -> StepBuffers:
    """Allocate (with torch) every buffer a step over ``layers`` needs; with
    ``fused`` also the workspace of the one-call form (run_step(fused=True))."""
    import torch
    B = layers[0].B
    nb = dpsgd_norms_workspace_bytes(layers, mode)
    cb = dpsgd_clip_workspace_bytes(layers)
    fb = dpsgd_clipped_sum_workspace_bytes(layers, mode) if fused else 0
    return StepBuffers(
        norms_sq=torch.empty(B, dtype=torch.float32, device=device),
        factors=torch.empty(B, dtype=torch.float32, device=device),
        mask=torch.empty(B, dtype=torch.uint8, device=device),
        norms_ws=torch.empty(max(nb, 1), dtype=torch.uint8, device=device),
        clip_ws=torch.empty(max(cb, 1), dtype=torch.uint8, device=device),
        grads=[torch.empty((L.d_out, L.d_in), dtype=torch.float32, device=device)
               for L in layers],
        fused_ws=torch.empty(max(fb, 1), dtype=torch.uint8, device=device) if fused else None,
    )


def run_clipped_sum(layers, buf: StepBuffers, C: float, mode: int = DPSGD_NORM_AUTO, stream=None,
                    fused: bool = False):
    """The step up to its commit point: global norms, clip factors and the
    clipped sums in ``buf.grads`` (two ABI calls, or one with ``fused``)."""
    if fused:
        dpsgd_clipped_sum_multi(layers, mode, C, buf.grads, buf.norms_sq, accumulate=False,
                                factors_out=buf.factors, mask_out=buf.mask,
                                workspace=buf.fused_ws, stream=stream)
    else:
        dpsgd_per_example_norms_multi(layers, mode, buf.norms_sq, accumulate=False,
                                      workspace=buf.norms_ws, stream=stream)
        dpsgd_clip_accumulate_multi(layers, buf.norms_sq, C, buf.grads, accumulate=False,
                                    factors_out=buf.factors, mask_out=buf.mask,
                                    workspace=buf.clip_ws, stream=stream)


def run_step(layers, buf: StepBuffers, C: float, sigma: float, seed: int, step: int = 0,
             scale: float = 1.0, mode: int = DPSGD_NORM_AUTO, stream=None, fused: bool = False):
    """One DP-SGD gradient step: global norms, clip + sum, noise (three ABI
    calls, or two with ``fused``: dpsgd_clipped_sum_multi, then the noise)."""
    run_clipped_sum(layers, buf, C, mode, stream, fused)
    dpsgd_add_noise_multi(layers, buf.grads, sigma, C, seed, step, scale, stream=stream)


class StepGraph:
    """The clipped-sum part of a step captured as a HIP graph (torch.cuda.CUDAGraph),
    replayed once per step, followed by the noise call.

    The library makes no allocation, memset or synchronising call while it
    enqueues, so the norms, factors and clipped sums (two ABI calls, or one
    with ``fused``) can be captured. A replay re-runs them with the arguments
    of the capture: the same input and output buffers (refill the inputs in
    place between replays) and the same C. The noise is not captured: it is
    enqueued after each replay with the seed and step that ``replay`` is
    given, because a captured noise kernel would add the same normals at
    every replay. A (seed, step) pair that this object has already released
    is refused: the noise of every release must be fresh."""

    def __init__(self, layers, buf: StepBuffers, C: float, sigma: float, scale: float = 1.0,
                 mode: int = DPSGD_NORM_AUTO, fused: bool = False):
        import torch
        load()
        self._keep = (layers, buf)
        self._noise = (sigma, C, scale)
        self._used = set()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):   # one eager pass first, outside the capture
            run_clipped_sum(layers, buf, C, mode, fused=fused)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            run_clipped_sum(layers, buf, C, mode, fused=fused)

    def replay(self, seed: int, step: int):
        """One step: the captured clipped sums, then noise keyed by (seed, step)."""
        key = (int(seed), int(step))
        if key in self._used:
            raise ValueError(f"noise (seed, step) = {key} was already released by this graph")
        self._used.add(key)
        layers, buf = self._keep
        sigma, C, scale = self._noise
        self.graph.replay()
        dpsgd_add_noise_multi(layers, buf.grads, sigma, C, seed, step, scale)
