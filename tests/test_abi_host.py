"""Host-side checks of the C ABI library (CPU only: no kernel is launched).

The library loads, exports every function ``include/dpsgd.h`` declares, and
rejects bad arguments before enqueuing anything.
"""

import ctypes
import os
import re

import pytest

from paper_2609_20532_amd import dpsgd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return dpsgd.load()


def _declared_functions():
    text = open(os.path.join(ROOT, "include", "dpsgd.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dpsgd_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_function_is_exported(lib):
    names = _declared_functions()
    assert len(names) >= 14
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(dpsgd.EXPORTED)


def test_status_strings(lib):
    for st in (0, -1, -2, -3, -4, 99):
        assert isinstance(lib.dpsgd_status_string(st), bytes)
    assert lib.dpsgd_status_string(-3) == b"workspace missing or too small"


def test_layer_struct_layout():
    assert ctypes.sizeof(dpsgd.dpsgd_layer) == 56
    assert dpsgd.dpsgd_layer.dtype.offset == 48


def test_workspace_queries_and_mode_selection(lib):
    c3 = dpsgd.shape_layer(64, 512, 768, 3072)
    assert dpsgd.dpsgd_select_norm_mode(c3) == dpsgd.DPSGD_NORM_GHOST
    lora = dpsgd.shape_layer(16, 1024, 4096, 16)
    assert dpsgd.dpsgd_select_norm_mode(lora) == dpsgd.DPSGD_NORM_MATERIALIZE
    # T = 512 bf16 runs the Gram form on 256-row tiles: 2 row blocks, so 4
    # partials per example (one per diagonal tile, two per off-diagonal tile;
    # 64 x 4 floats), and the 192 tiles become 256 jobs (the off-diagonal
    # tiles as two row halves), each workgroup with a 256 KB float32 park slot.
    assert dpsgd.dpsgd_norms_workspace_bytes(c3, dpsgd.DPSGD_NORM_GHOST) == 1024 + 256 * 262144
    # More than 512 jobs: the grid (and the park area) stays at 512 workgroups.
    big = dpsgd.shape_layer(200, 520, 64, 64)    # 3 row blocks, 6 tiles, 1200 jobs
    assert dpsgd.dpsgd_norms_workspace_bytes(big, dpsgd.DPSGD_NORM_GHOST) == 7424 + 512 * 262144
    # c4's 11008-wide layer: 160 tiles of 236 column slices; splitting their
    # columns would need a second round on 256 CUs, while 4 + 2 x 6 = 16 jobs
    # per example (256) fill exactly one.
    c4 = dpsgd.shape_layer(16, 1024, 4096, 11008)
    assert dpsgd.dpsgd_norms_workspace_bytes(c4, dpsgd.DPSGD_NORM_GHOST) == 1024 + 256 * 262144
    # At B = 8 (80 tiles) each tile is split into 3 column parts (240 jobs, one
    # round) that park their partial Gram tiles: two 256 KB slots per part.
    c4b8 = dpsgd.shape_layer(8, 1024, 4096, 11008)
    assert dpsgd.dpsgd_norms_workspace_bytes(c4b8, dpsgd.DPSGD_NORM_GHOST) == 512 + 80 * 3 * 2 * 262144
    # float32 keeps the 128-row tiles (4 T-tiles -> 10 pairs) and no park area.
    c3f = dpsgd.shape_layer(64, 512, 768, 3072, dpsgd.DPSGD_F32)
    assert dpsgd.dpsgd_norms_workspace_bytes(c3f, dpsgd.DPSGD_NORM_GHOST) == 2560
    t1 = dpsgd.shape_layer(32, 1, 256, 128, dpsgd.DPSGD_F32)
    assert dpsgd.dpsgd_norms_workspace_bytes(t1) == 256   # one partial per example, rounded
    assert dpsgd.dpsgd_clip_workspace_bytes(t1) > 0
    bad = dpsgd.shape_layer(0, 1, 4, 4)
    assert dpsgd.dpsgd_norms_workspace_bytes(bad) == 0
    with pytest.raises(dpsgd.DpsgdError):
        dpsgd.dpsgd_select_norm_mode(bad)


def _lay(**kw):
    base = dict(A=16, G=32, B=2, T=3, d_in=4, d_out=5, dtype=1, tensor_id=0)
    base.update(kw)
    return dpsgd.dpsgd_layer(base["A"], base["G"], base["B"], base["T"], base["d_in"],
                             base["d_out"], base["dtype"], base["tensor_id"])


@pytest.mark.parametrize("kw,status", [
    (dict(B=0), -1), (dict(T=0), -1), (dict(d_in=-3), -1), (dict(d_out=0), -1),
    (dict(A=None), -1), (dict(G=None), -1), (dict(dtype=7), -2),
    (dict(B=1 << 40), -1), (dict(d_in=1 << 31, d_out=1 << 31), -1),
    (dict(A=24), -1), (dict(G=40), -1),   # not 16-byte aligned
])
def test_norms_rejects_bad_layers(lib, kw, status):
    L = _lay(**kw)
    st = lib.dpsgd_per_example_norms(ctypes.byref(L), 0, ctypes.c_void_p(64), 0,
                                     ctypes.c_void_p(128), 1 << 20, None)
    assert st == status


def test_norms_rejects_bad_mode_and_workspace(lib):
    L = _lay()
    assert lib.dpsgd_per_example_norms(ctypes.byref(L), 5, ctypes.c_void_p(64), 0,
                                       ctypes.c_void_p(128), 1 << 20, None) == -2
    assert lib.dpsgd_per_example_norms(ctypes.byref(L), 0, None, 0,
                                       ctypes.c_void_p(128), 1 << 20, None) == -1
    assert lib.dpsgd_per_example_norms(ctypes.byref(L), 0, ctypes.c_void_p(64), 0,
                                       ctypes.c_void_p(128), 0, None) == -3
    assert lib.dpsgd_per_example_norms(ctypes.byref(L), 0, ctypes.c_void_p(64), 0,
                                       None, 1 << 20, None) == -3


def test_multi_rejects_mixed_batches_and_dtypes(lib):
    arr = (dpsgd.dpsgd_layer * 2)(_lay(), _lay(B=3))
    assert lib.dpsgd_per_example_norms_multi(arr, 2, 0, ctypes.c_void_p(64), 0,
                                             ctypes.c_void_p(128), 1 << 20, None) == -1
    arr = (dpsgd.dpsgd_layer * 2)(_lay(), _lay(dtype=0))
    assert lib.dpsgd_per_example_norms_multi(arr, 2, 0, ctypes.c_void_p(64), 0,
                                             ctypes.c_void_p(128), 1 << 20, None) == -2
    assert lib.dpsgd_per_example_norms_multi(arr, 0, 0, ctypes.c_void_p(64), 0,
                                             ctypes.c_void_p(128), 1 << 20, None) == -1


@pytest.mark.parametrize("C", [0.0, -1.0, float("nan")])
def test_clip_rejects_bad_C(lib, C):
    L = _lay()
    st = lib.dpsgd_clip_accumulate(ctypes.byref(L), ctypes.c_void_p(64), C, ctypes.c_void_p(256),
                                   0, None, None, ctypes.c_void_p(512), 1 << 20, None)
    assert st == -1
    assert lib.dpsgd_clip_factors(ctypes.c_void_p(64), 4, C, None, None, None) == -1


def test_clip_rejects_null_grad_and_small_workspace(lib):
    L = _lay()
    assert lib.dpsgd_clip_accumulate(ctypes.byref(L), ctypes.c_void_p(64), 1.0, None, 0, None,
                                     None, ctypes.c_void_p(512), 1 << 20, None) == -1
    assert lib.dpsgd_clip_accumulate(ctypes.byref(L), ctypes.c_void_p(64), 1.0,
                                     ctypes.c_void_p(256), 0, None, None, ctypes.c_void_p(512),
                                     8, None) == -3


@pytest.mark.parametrize("sigma,C,scale", [(-1.0, 1.0, 1.0), (float("nan"), 1.0, 1.0),
                                           (1.0, 0.0, 1.0), (1.0, float("inf"), 1.0),
                                           (1.0, 1.0, float("inf")), (float("inf"), 1.0, 1.0)])
def test_noise_rejects_bad_scalars(lib, sigma, C, scale):
    L = _lay()
    assert lib.dpsgd_add_noise(ctypes.byref(L), ctypes.c_void_p(256), sigma, C, 1, 0, scale,
                               None) == -1


def test_hooks_reject_bad_args_and_accept_empty(lib):
    assert lib.dpsgd_philox_u32(None, 0, 4, 1, 0, 0, None) == -1
    assert lib.dpsgd_philox_u32(ctypes.c_void_p(64), -1, 4, 1, 0, 0, None) == -1
    assert lib.dpsgd_philox_u32(ctypes.c_void_p(64), 0, 0, 1, 0, 0, None) == 0
    assert lib.dpsgd_gaussian(ctypes.c_void_p(64), -5, 1, 0, 0, None) == -1
    assert lib.dpsgd_gaussian(ctypes.c_void_p(64), 0, 1, 0, 0, None) == 0


def test_adamw_struct_layout():
    assert ctypes.sizeof(dpsgd.dpsgd_adamw) == 24
    assert dpsgd.dpsgd_adamw.t.offset == 20


_GOOD_ADAMW = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01, t=1)


@pytest.mark.parametrize("bad", [dict(lr=-1.0), dict(lr=float("inf")), dict(beta1=1.0),
                                 dict(beta1=-0.1), dict(beta2=1.0), dict(beta2=float("nan")),
                                 dict(eps=0.0), dict(eps=float("inf")), dict(weight_decay=-1e-3),
                                 dict(weight_decay=float("nan")), dict(t=0)])
def test_noise_adamw_rejects_bad_hyperparameters(lib, bad):
    L = _lay()
    opt = dpsgd.make_adamw(**{**_GOOD_ADAMW, **bad})
    p = [ctypes.c_void_p(256 * (k + 1)) for k in range(4)]
    assert lib.dpsgd_noise_adamw(ctypes.byref(L), *p, None, 1.0, 1.0, 1, 0, 1.0,
                                 ctypes.byref(opt), None) == -1


def test_noise_adamw_rejects_null_and_misaligned_buffers(lib):
    L = _lay()
    opt = dpsgd.make_adamw(**_GOOD_ADAMW)
    good = [ctypes.c_void_p(256 * (k + 1)) for k in range(4)]
    for k in range(4):
        for bad in (None, ctypes.c_void_p(256 * (k + 1) + 4)):
            p = list(good)
            p[k] = bad
            assert lib.dpsgd_noise_adamw(ctypes.byref(L), *p, None, 1.0, 1.0, 1, 0, 1.0,
                                         ctypes.byref(opt), None) == -1
    # misaligned optional output, NULL optimizer config, bad noise scalars
    assert lib.dpsgd_noise_adamw(ctypes.byref(L), *good, ctypes.c_void_p(2052), 1.0, 1.0, 1, 0,
                                 1.0, ctypes.byref(opt), None) == -1
    assert lib.dpsgd_noise_adamw(ctypes.byref(L), *good, None, 1.0, 1.0, 1, 0, 1.0, None,
                                 None) == -1
    assert lib.dpsgd_noise_adamw(ctypes.byref(L), *good, None, -1.0, 1.0, 1, 0, 1.0,
                                 ctypes.byref(opt), None) == -1


def _fused(lib, layers, mode=0, C=1.0, grads=(256,), norms=64, ws=512, ws_bytes=1 << 30):
    arr = (dpsgd.dpsgd_layer * len(layers))(*layers)
    g = (ctypes.c_void_p * len(grads))(*[ctypes.c_void_p(x) if x else None for x in grads])
    return lib.dpsgd_clipped_sum_multi(arr, len(layers), mode, C, g, 0,
                                       ctypes.c_void_p(norms) if norms else None, None, None,
                                       ctypes.c_void_p(ws) if ws else None, ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(B=0), -1), (dict(T=0), -1), (dict(d_out=0), -1), (dict(A=None), -1),
    (dict(dtype=7), -2), (dict(A=24), -1),
])
def test_fused_rejects_bad_layers(lib, kw, status):
    assert _fused(lib, [_lay(**kw)]) == status


def test_fused_rejects_bad_arguments(lib):
    L = _lay()
    assert _fused(lib, [L], mode=5) == -2
    assert _fused(lib, [L], norms=None) == -1
    assert _fused(lib, [L], grads=(None,)) == -1
    assert _fused(lib, [L], grads=(264,)) == -1          # grad not 16-byte aligned
    for C in (0.0, -1.0, float("nan")):
        assert _fused(lib, [L], C=C) == -1
    assert _fused(lib, [L], ws=None) == -3
    assert _fused(lib, [L], ws_bytes=8) == -3
    assert _fused(lib, [L], ws=520) == -1                # workspace not 16-byte aligned
    assert _fused(lib, [L, _lay(B=3)], grads=(256, 512)) == -1


def test_fused_workspace_holds_the_stored_gradients(lib):
    """Adapter matrices (narrow side <= 16) take the stored form: the fused
    call's workspace holds B * d_in * d_out float32 per row range for each of
    them; with mode = GHOST it holds none and is smaller."""
    B, T = 16, 1024
    lora_a = dpsgd.shape_layer(B, T, 4096, 16)
    lora_b = dpsgd.shape_layer(B, T, 16, 4096)
    both = [lora_a, lora_b]
    fused = dpsgd.dpsgd_clipped_sum_workspace_bytes(both)
    ghost = dpsgd.dpsgd_clipped_sum_workspace_bytes(both, dpsgd.DPSGD_NORM_GHOST)
    # At least one row range of per-example gradients per adapter matrix (the
    # other workspace parts differ between the two plans).
    assert fused >= 2 * B * 4096 * 16 * 4
    assert fused > ghost
    # A layer without a narrow side stores nothing: same size in both modes.
    wide = [dpsgd.shape_layer(64, 512, 768, 3072)]
    assert dpsgd.dpsgd_clipped_sum_workspace_bytes(wide, dpsgd.DPSGD_NORM_GHOST) == \
        dpsgd.dpsgd_clipped_sum_workspace_bytes(wide)
    assert dpsgd.dpsgd_clipped_sum_workspace_bytes([dpsgd.shape_layer(0, 1, 4, 4)]) == 0


def test_select_norm_mode_reports_the_closed_form_for_T1(lib):
    """T = 1 layers run ||a||^2 ||g||^2 under every mode, and the query says so."""
    for d_in, d_out in ((256, 128), (784, 512), (4096, 16)):
        L = dpsgd.shape_layer(32, 1, d_in, d_out, dpsgd.DPSGD_F32)
        assert dpsgd.dpsgd_select_norm_mode(L) == dpsgd.DPSGD_NORM_CLOSED_FORM
    # The reported value is not a mode argument.
    L = _lay()
    assert lib.dpsgd_per_example_norms(ctypes.byref(L), dpsgd.DPSGD_NORM_CLOSED_FORM,
                                       ctypes.c_void_p(64), 0, ctypes.c_void_p(128), 1 << 20,
                                       None) == -2
    assert dpsgd.dpsgd_norms_workspace_bytes(L, dpsgd.DPSGD_NORM_CLOSED_FORM) == 0


def test_norms_and_clip_reject_misaligned_workspace(lib):
    L = _lay()
    assert lib.dpsgd_per_example_norms(ctypes.byref(L), 0, ctypes.c_void_p(64), 0,
                                       ctypes.c_void_p(136), 1 << 20, None) == -1
    arr = (dpsgd.dpsgd_layer * 2)(_lay(), _lay(tensor_id=1))
    assert lib.dpsgd_per_example_norms_multi(arr, 2, 0, ctypes.c_void_p(64), 0,
                                             ctypes.c_void_p(520), 1 << 20, None) == -1
    assert lib.dpsgd_clip_accumulate(ctypes.byref(L), ctypes.c_void_p(64), 1.0,
                                     ctypes.c_void_p(256), 0, None, None, ctypes.c_void_p(516),
                                     1 << 20, None) == -1
    g = (ctypes.c_void_p * 2)(ctypes.c_void_p(256), ctypes.c_void_p(512))
    assert lib.dpsgd_clip_accumulate_multi(arr, 2, ctypes.c_void_p(64), 1.0, g, 0, None, None,
                                           ctypes.c_void_p(1032), 1 << 20, None) == -1


def test_noise_calls_reject_repeated_tensor_ids(lib):
    """Two layers of one noise call with the same tensor_id would receive the
    same normals; the call refuses them before enqueuing anything."""
    dup = (dpsgd.dpsgd_layer * 3)(_lay(tensor_id=0), _lay(tensor_id=5), _lay(tensor_id=0))
    ok = (dpsgd.dpsgd_layer * 3)(_lay(tensor_id=0), _lay(tensor_id=5), _lay(tensor_id=1))
    g = (ctypes.c_void_p * 3)(*[ctypes.c_void_p(256 * (k + 1)) for k in range(3)])
    assert lib.dpsgd_add_noise_multi(dup, 3, g, 1.0, 1.0, 1, 0, 1.0, None) == -1
    opt = dpsgd.make_adamw(**_GOOD_ADAMW)
    arrs = [(ctypes.c_void_p * 3)(*[ctypes.c_void_p(4096 * (j + 1) + 256 * k) for k in range(3)])
            for j in range(4)]
    assert lib.dpsgd_noise_adamw_multi(dup, 3, *arrs, None, 1.0, 1.0, 1, 0, 1.0,
                                       ctypes.byref(opt), None) == -1
    # The same arrays with distinct ids pass the checks (a NULL stream would
    # then launch, so only the argument checks are exercised here: sigma < 0).
    assert lib.dpsgd_add_noise_multi(ok, 3, g, -1.0, 1.0, 1, 0, 1.0, None) == -1


def test_make_layer_requires_a_tensor_id():
    import inspect
    p = inspect.signature(dpsgd.make_layer).parameters["tensor_id"]
    assert p.default is inspect.Parameter.empty


def test_noalloc_norms_reject_sizes_beyond_the_scratch(lib):
    """More partials than the allocation-free call's scratch array holds:
    refused before the device is touched."""
    assert dpsgd.DPSGD_NOALLOC_SCRATCH_BYTES == 8 << 20
    B = (8 << 20) // 4 + 1           # T = 1: one partial per example
    L = _lay(B=B, T=1, d_in=4, d_out=4)
    assert dpsgd.dpsgd_norms_workspace_bytes(L, 0) > dpsgd.DPSGD_NOALLOC_SCRATCH_BYTES
    assert lib.dpsgd_per_example_norms_multi_noalloc(ctypes.byref(L), 1, 0, ctypes.c_void_p(64),
                                                     0, None) == -3
    # The usual argument checks come first.
    assert lib.dpsgd_per_example_norms_multi_noalloc(ctypes.byref(_lay(B=0)), 1, 0,
                                                     ctypes.c_void_p(64), 0, None) == -1
    assert lib.dpsgd_per_example_norms_multi_noalloc(ctypes.byref(_lay()), 1, 7,
                                                     ctypes.c_void_p(64), 0, None) == -2
    assert lib.dpsgd_per_example_norms_multi_noalloc(ctypes.byref(_lay()), 1, 0, None, 0,
                                                     None) == -1
