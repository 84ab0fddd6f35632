"""The C ABI on the host: the library loads, exports what include/xpress.h
declares, and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

from paper_2608_02438_amd import xpress as X

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "xpress.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(xp_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(X.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = X.load_library()
    for name in declared_functions():
        assert hasattr(L, name), name


def _weights(**kw):
    w = X._Weights(H=4096, r=256, V=151936, B=16, dtype=X.XP_BF16)
    for n in X.WEIGHT_NAMES:
        setattr(w, n, 0x1000)          # never dereferenced: validation fails first
    for k, v in kw.items():
        setattr(w, k, v)
    return w


@pytest.mark.parametrize("change,status", [
    (dict(r=128), X.XP_EUNSUPPORTED),
    (dict(B=33), X.XP_EUNSUPPORTED),
    (dict(H=4000), X.XP_EUNSUPPORTED),
    (dict(H=16384), X.XP_EUNSUPPORTED),
    (dict(dtype=7), X.XP_EINVAL),
    (dict(V=0), X.XP_EINVAL),
    (dict(W_r=None), X.XP_EINVAL),
    (dict(W_lm=None), X.XP_EINVAL),
])
def test_create_rejects_bad_arguments_without_a_gpu(change, status):
    L = X.load_library()
    h = ctypes.c_void_p(0)
    w = _weights(**change)
    assert L.xp_create(ctypes.byref(w), 1, ctypes.byref(h)) == status
    assert not h.value
    assert L.xp_last_error(None)


def test_create_rejects_bad_batch():
    L = X.load_library()
    h = ctypes.c_void_p(0)
    assert L.xp_create(ctypes.byref(_weights()), 0, ctypes.byref(h)) == X.XP_EINVAL
    assert L.xp_create(ctypes.byref(_weights()), 5000, ctypes.byref(h)) == X.XP_EINVAL
    assert L.xp_create(None, 1, ctypes.byref(h)) == X.XP_EINVAL
    assert L.xp_create(ctypes.byref(_weights()), 1, None) == X.XP_EINVAL


def test_calls_on_a_null_handle_are_rejected():
    L = X.load_library()
    assert L.xp_refine_block(None, 1, 1, 1, None, None, None, None, None, None, 6, 0, 1, None, None,
                             None, None) == X.XP_EINVAL
    assert L.xp_verify_block(None, 1, 1, None, 1, None, None, None, 1, 1, None) == X.XP_EINVAL
    assert L.xp_device_errors(None, None, None) == X.XP_EINVAL
    L.xp_destroy(None)


def test_status_strings():
    L = X.load_library()
    assert L.xp_status_string(X.XP_EHIP) == b"XP_EHIP"
    assert L.xp_status_string(X.XP_OK) == b"XP_OK"


def test_probes_reject_bad_arguments_without_a_gpu():
    L = X.load_library()
    assert L.xp_probe_hbm_read(None, 16, 0x1000, 1, None) == X.XP_EINVAL
    assert L.xp_probe_hbm_read(0x1000, 24, 0x1000, 1, None) == X.XP_EINVAL
    assert L.xp_probe_hbm_read(0x1008, 16, 0x1000, 1, None) == X.XP_EINVAL
    assert L.xp_probe_hbm_read(0x1000, 16, None, 1, None) == X.XP_EINVAL
    assert L.xp_probe_hbm_read(0x1000, 16, 0x1000, 0, None) == X.XP_EINVAL
    assert L.xp_probe_mfma_bf16(None, 1, 1, 0x1000, None) == X.XP_EINVAL
    assert L.xp_probe_mfma_bf16(0x1000, 0, 1, 0x1000, None) == X.XP_EINVAL
    assert L.xp_probe_mfma_bf16(0x1000, 1, -1, 0x1000, None) == X.XP_EINVAL
    assert L.xp_probe_mfma_bf16(0x1000, 1, 1, None, None) == X.XP_EINVAL


def test_toeplitz_mixer_rejects_bad_arguments_without_a_gpu():
    L = X.load_library()
    p = ctypes.c_void_p(0x1000)         # never dereferenced: validation fails first
    assert L.xp_toeplitz_mixer(None, 256, 16, X.XP_BF16, p, None) == X.XP_EINVAL
    assert L.xp_toeplitz_mixer(p, 256, 16, X.XP_BF16, None, None) == X.XP_EINVAL
    assert L.xp_toeplitz_mixer(p, 0, 16, X.XP_BF16, p, None) == X.XP_EINVAL
    assert L.xp_toeplitz_mixer(p, 256, 0, X.XP_F32, p, None) == X.XP_EINVAL
    assert L.xp_toeplitz_mixer(p, 256, 33, X.XP_F32, p, None) == X.XP_EINVAL
    assert L.xp_toeplitz_mixer(p, 256, 16, 7, p, None) == X.XP_EINVAL


def _layer_weights(**kw):
    w = X._LayerWeights(H=4096, n_heads=32, n_kv=8, head_dim=128, ffn=12288, eps=1e-6,
                        rope_theta=1e6)
    for n in X.LAYER_WEIGHT_NAMES:
        setattr(w, n, 0x1000)          # never dereferenced: validation fails first
    for k, v in kw.items():
        setattr(w, k, v)
    return w


@pytest.mark.parametrize("change,status", [
    (dict(head_dim=64), X.XP_EUNSUPPORTED),
    (dict(n_kv=3), X.XP_EUNSUPPORTED),            # 32 heads not a multiple of 3
    (dict(n_kv=2), X.XP_EUNSUPPORTED),            # group of 16
    (dict(H=4000), X.XP_EUNSUPPORTED),
    (dict(H=16384), X.XP_EUNSUPPORTED),
    (dict(ffn=1000), X.XP_EUNSUPPORTED),
    (dict(H=0), X.XP_EINVAL),
    (dict(rope_theta=0.0), X.XP_EINVAL),
    (dict(eps=-1.0), X.XP_EINVAL),
    (dict(Wd=None), X.XP_EINVAL),
    (dict(g_q=None), X.XP_EINVAL),
    (dict(Wo=0x1008), X.XP_EINVAL),               # not 16-byte aligned
])
def test_layer_create_rejects_bad_arguments_without_a_gpu(change, status):
    L = X.load_library()
    h = ctypes.c_void_p(0)
    w = _layer_weights(**change)
    assert L.xp_layer_create(ctypes.byref(w), 1, 16, 2048, ctypes.byref(h)) == status
    assert not h.value


def test_layer_create_and_forward_reject_bad_sizes_and_null_handles():
    L = X.load_library()
    h = ctypes.c_void_p(0)
    w = _layer_weights()
    for mb, mB, mc in ((0, 16, 2048), (1, 0, 2048), (1, 33, 2048), (1, 16, -1)):
        assert L.xp_layer_create(ctypes.byref(w), mb, mB, mc, ctypes.byref(h)) == X.XP_EINVAL
    assert L.xp_layer_create(None, 1, 16, 2048, ctypes.byref(h)) == X.XP_EINVAL
    assert L.xp_layer_create(ctypes.byref(w), 1, 16, 2048, None) == X.XP_EINVAL
    p = 0x1000
    assert L.xp_layer_forward(None, 1, 16, 1, p, p, p, 64, p, p, p, None) == X.XP_EINVAL
    L.xp_layer_destroy(None)


def _layer_weights(**kw):
    w = X._LayerWeights(H=4096, n_heads=32, n_kv=8, head_dim=128, ffn=12288, eps=1e-6,
                        rope_theta=1e6)
    for n in X.LAYER_WEIGHT_NAMES:
        setattr(w, n, 0x1000)          # never dereferenced: validation fails first
    for k, v in kw.items():
        setattr(w, k, v)
    return w


@pytest.mark.parametrize("change,call,status", [
    ({}, dict(batch=64, B=32), X.XP_EINVAL),              # 2048 positions: beyond the scratch
    ({}, dict(batch=1, B=33), X.XP_EINVAL),
    ({}, dict(batch=0, B=16), X.XP_EINVAL),
    ({}, dict(C_max=0), X.XP_EINVAL),
    ({}, dict(causal=2), X.XP_EINVAL),
    ({}, dict(x=0x1008), X.XP_EINVAL),                    # not 16-byte aligned
    (dict(Wd=None), {}, X.XP_EINVAL),
    (dict(head_dim=64), {}, X.XP_EUNSUPPORTED),
    (dict(n_heads=24), {}, X.XP_EUNSUPPORTED),            # group 3
])
def test_layer_forward_noalloc_rejects_without_a_gpu(change, call, status):
    """The allocation-free forward checks the weights, the call and whether
    the call's buffers fit its static scratch before any HIP call."""
    L = X.load_library()
    w = _layer_weights(**change)
    a = dict(batch=1, B=16, causal=1, x=0x1000, C_max=100)
    a.update(call)
    st = L.xp_layer_forward_noalloc(ctypes.byref(w), a["batch"], a["B"], a["causal"], a["x"],
                                    0x1000, 0x1000, a["C_max"], 0x1000, 0x1000, 0x1000, None)
    assert st == status
    assert L.xp_layer_last_error(None)
