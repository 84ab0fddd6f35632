"""Python binding of libxpress.so (the C ABI in include/xpress.h).

Argument marshalling only: every step of the refine + verify path runs in the
HIP kernels of the library.  PyTorch is used for device memory and streams.
The library must have been built (``python -m paper_2608_02438_amd.build``);
there is no fallback implementation, and loading fails loudly without it.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Dict, Optional

import numpy as np

# the library this process loads; XPRESS_LIB names another build of it (the
# host-ASan one of build.py --asan)
LIB_PATH = os.environ.get("XPRESS_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libxpress.so")

XP_OK, XP_EINVAL, XP_EUNSUPPORTED, XP_EHIP, XP_ENOMEM = 0, -1, -2, -3, -4
XP_F32, XP_BF16 = 0, 1
XP_EARLY_EXIT, XP_WRITE_LOGITS = 1, 2
XP_DEVERR_TOKEN, XP_DEVERR_TEMPERATURE, XP_DEVERR_FILTER = 1, 2, 4

EXPORTS = ("xp_create", "xp_destroy", "xp_last_error", "xp_status_string",
           "xp_refine_block", "xp_verify_block", "xp_device_errors", "xp_timing_enable",
           "xp_timing_read", "xp_probe_hbm_read", "xp_probe_mfma_bf16", "xp_toeplitz_mixer",
           "xp_layer_create", "xp_layer_forward", "xp_layer_destroy", "xp_layer_last_error",
           "xp_layer_forward_noalloc")
LAYER_WEIGHT_NAMES = ("g_attn", "Wq", "Wk", "Wv", "g_q", "g_k", "Wo", "g_mlp", "Wg", "Wu", "Wd")
STAGES = ("prep", "lmhead", "select", "rspace", "read", "verify")


class XpError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_status_name(status)}: {msg}")
        self.status = status


class _Weights(ctypes.Structure):
    _fields_ = [("H", ctypes.c_int32), ("r", ctypes.c_int32), ("V", ctypes.c_int32),
                ("B", ctypes.c_int32), ("dtype", ctypes.c_int32)] + [
        (n, ctypes.c_void_p) for n in ("W_lm", "W_h", "W_g", "W_e", "W_in", "L", "W_1", "W_2", "W_r")]


WEIGHT_NAMES = ("W_lm", "W_h", "W_g", "W_e", "W_in", "L", "W_1", "W_2", "W_r")

class _LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("H", "n_heads", "n_kv", "head_dim", "ffn")] + [
        ("eps", ctypes.c_float), ("rope_theta", ctypes.c_float)] + [
        (n, ctypes.c_void_p) for n in ("g_attn", "Wq", "Wk", "Wv", "g_q", "g_k", "Wo", "g_mlp",
                                       "Wg", "Wu", "Wd")]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libxpress.so and declare its signatures (no GPU work)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2608_02438_amd.build`")
    L = ctypes.CDLL(path)
    vp, i32, u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32
    L.xp_create.argtypes = [ctypes.POINTER(_Weights), i32, ctypes.POINTER(vp)]
    L.xp_create.restype = i32
    L.xp_destroy.argtypes = [vp]
    L.xp_destroy.restype = None
    L.xp_last_error.argtypes = [vp]
    L.xp_last_error.restype = ctypes.c_char_p
    L.xp_status_string.argtypes = [i32]
    L.xp_status_string.restype = ctypes.c_char_p
    L.xp_refine_block.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, i32, u32, vp, vp, vp,
                                  vp, vp]
    L.xp_refine_block.restype = i32
    L.xp_verify_block.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.xp_verify_block.restype = i32
    L.xp_device_errors.argtypes = [vp, ctypes.POINTER(u32), vp]
    L.xp_device_errors.restype = i32
    L.xp_timing_enable.argtypes = [vp, u32, i32]
    L.xp_timing_enable.restype = i32
    L.xp_timing_read.argtypes = [vp, ctypes.POINTER(ctypes.c_float), ctypes.POINTER(i32)]
    L.xp_timing_read.restype = i32
    L.xp_probe_hbm_read.argtypes = [vp, ctypes.c_size_t, vp, i32, vp]
    L.xp_probe_hbm_read.restype = i32
    L.xp_probe_mfma_bf16.argtypes = [vp, i32, i32, vp, vp]
    L.xp_probe_mfma_bf16.restype = i32
    L.xp_toeplitz_mixer.argtypes = [vp, i32, i32, i32, vp, vp]
    L.xp_toeplitz_mixer.restype = i32
    L.xp_layer_create.argtypes = [ctypes.POINTER(_LayerWeights), i32, i32, i32, ctypes.POINTER(vp)]
    L.xp_layer_create.restype = i32
    L.xp_layer_forward.argtypes = [vp, i32, i32, i32, vp, vp, vp, i32, vp, vp, vp, vp]
    L.xp_layer_forward.restype = i32
    L.xp_layer_destroy.argtypes = [vp]
    L.xp_layer_destroy.restype = None
    L.xp_layer_last_error.argtypes = [vp]
    L.xp_layer_last_error.restype = ctypes.c_char_p
    L.xp_layer_forward_noalloc.argtypes = [ctypes.POINTER(_LayerWeights), i32, i32, i32, vp, vp,
                                           vp, i32, vp, vp, vp, vp]
    L.xp_layer_forward_noalloc.restype = i32
    _lib = L
    return L


def _status_name(s: int) -> str:
    try:
        return load_library().xp_status_string(s).decode()
    except Exception:  # pragma: no cover
        return str(s)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return int(t.data_ptr())


def _stream(stream) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def bf16_tensor(bits: np.ndarray, device="cuda"):
    """Device bf16 tensor from bf16 bit patterns (uint16)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def device_tensor(x: np.ndarray, device="cuda"):
    """Device tensor of a stored input: uint16 -> bf16, float32 -> float32, ints as is."""
    import torch
    if x.dtype == np.uint16:
        return bf16_tensor(x, device)
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


@dataclass
class RefineOut:
    ids: object
    iters: object
    logits: Optional[object]
    traj: Optional[object]


class Refiner:
    """One xp_handle: weights on the device plus the workspace for max_batch sequences."""

    def __init__(self, weights: Dict[str, object], H: int, r: int, V: int, B: int,
                 max_batch: int):
        import torch
        L = load_library()
        w0 = weights["W_lm"]
        self.dtype = XP_BF16 if w0.dtype == torch.bfloat16 else XP_F32
        tdt = torch.bfloat16 if self.dtype == XP_BF16 else torch.float32
        self.tdtype = tdt
        self.H, self.r, self.V, self.B, self.max_batch = H, r, V, B, max_batch
        self.device = w0.device
        self._keep = {}
        st = _Weights(H=H, r=r, V=V, B=B, dtype=self.dtype)
        for n in WEIGHT_NAMES:
            t = weights[n]
            if t.dtype != tdt or not t.is_contiguous() or t.device != self.device:
                raise ValueError(f"{n}: expected a contiguous {tdt} tensor on {self.device}")
            self._keep[n] = t
            setattr(st, n, t.data_ptr())
        h = ctypes.c_void_p()
        with torch.cuda.device(self.device):
            s = L.xp_create(ctypes.byref(st), max_batch, ctypes.byref(h))
        if s != XP_OK:
            raise XpError(s, L.xp_last_error(None).decode())
        self._h = h
        self._L = L

    # ------------------------------------------------------------------
    def _check(self, s: int):
        if s != XP_OK:
            raise XpError(s, self._L.xp_last_error(self._h).decode())

    def refine_block(self, hidden, anchor, seed_ids=None, temp=None, u_draft=None, K: int = 6,
                     early_exit: bool = False, write_logits: bool = False,
                     want_traj: bool = False, out: Optional[RefineOut] = None,
                     stream=None, temperature=None, top_k=None, top_p=None) -> RefineOut:
        import torch
        batch = hidden.shape[0]
        if (tuple(hidden.shape) != (batch, self.B, self.H) or hidden.dtype != self.tdtype
                or not hidden.is_contiguous() or hidden.device != self.device):
            raise ValueError(f"hidden must be a contiguous [{batch}][{self.B}][{self.H}] "
                             f"{self.tdtype} tensor on {self.device}")
        for name, t, dt in (("anchor", anchor, torch.int32), ("seed_ids", seed_ids, torch.int32),
                            ("temp", temp, torch.uint8), ("u_draft", u_draft, torch.float32),
                            ("temperature", temperature, torch.float32),
                            ("top_k", top_k, torch.int32), ("top_p", top_p, torch.float32)):
            if t is not None and (t.dtype != dt or not t.is_contiguous() or t.device != self.device):
                raise ValueError(f"{name}: expected a contiguous {dt} tensor on {self.device}")
        if out is None:
            dev = self.device
            out = RefineOut(
                ids=torch.empty((batch, self.B), dtype=torch.int32, device=dev),
                iters=torch.empty((batch,), dtype=torch.int32, device=dev),
                logits=(torch.empty((batch, self.B, self.V), dtype=torch.float32, device=dev)
                        if write_logits else None),
                traj=(torch.empty((K + 1, batch, self.B), dtype=torch.int32, device=dev)
                      if want_traj else None))
        flags = (XP_EARLY_EXIT if early_exit else 0) | (XP_WRITE_LOGITS if write_logits else 0)
        s = self._L.xp_refine_block(
            self._h, batch, _ptr(hidden), _ptr(anchor), _ptr(seed_ids), _ptr(temp),
            _ptr(temperature), _ptr(top_k), _ptr(top_p), _ptr(u_draft), K, flags, _ptr(out.ids),
            _ptr(out.iters),
            _ptr(out.logits) if write_logits else None, _ptr(out.traj), _stream(stream))
        self._check(s)
        return out

    def verify_block(self, draft_ids, target_ids, temp=None, target_logits=None, r_accept=None,
                     u_resample=None, out=None, stream=None):
        import torch
        batch = draft_ids.shape[0]
        if out is None:
            out = (torch.empty((batch,), dtype=torch.int32, device=self.device),
                   torch.empty((batch,), dtype=torch.int32, device=self.device))
        s = self._L.xp_verify_block(
            self._h, batch, _ptr(draft_ids), _ptr(temp), _ptr(target_ids), _ptr(target_logits),
            _ptr(r_accept), _ptr(u_resample), _ptr(out[0]), _ptr(out[1]), _stream(stream))
        self._check(s)
        return out

    def device_errors(self, stream=None) -> int:
        v = ctypes.c_uint32(0)
        self._check(self._L.xp_device_errors(self._h, ctypes.byref(v), _stream(stream)))
        return int(v.value)

    def timing_enable(self, stages=("lmhead",), capacity: int = 4096):
        """Record HIP events around the named stages of every following call."""
        mask = 0
        for n in stages:
            mask |= 1 << STAGES.index(n)
        self._check(self._L.xp_timing_enable(self._h, mask, capacity))

    def timing_read(self):
        """{stage: (total ms, recorded launches)} since the last read; synchronizes."""
        ms = (ctypes.c_float * len(STAGES))()
        n = (ctypes.c_int32 * len(STAGES))()
        self._check(self._L.xp_timing_read(self._h, ms, n))
        return {s: (float(ms[i]), int(n[i])) for i, s in enumerate(STAGES)}

    def close(self):
        if getattr(self, "_h", None):
            self._L.xp_destroy(self._h)
            self._h = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass


def refiner_from_arrays(weights: Dict[str, np.ndarray], H, r, V, B, max_batch, device="cuda"):
    """Upload stored weights (bf16 bits or float32) and create a Refiner."""
    return Refiner({n: device_tensor(weights[n], device) for n in WEIGHT_NAMES}, H, r, V, B,
                   max_batch)


def _check(st: int, what: str):
    if st != XP_OK:
        raise XpError(st, what)


def probe_hbm_read(buf, out_sum, workgroups: int, stream=None):
    """Launch the HBM read probe over the whole of `buf` (a contiguous device
    tensor); `out_sum` (a device int32/uint32 tensor of one element) receives
    the sum of its 32-bit words modulo 2^32."""
    L = load_library()
    nbytes = buf.numel() * buf.element_size()
    _check(L.xp_probe_hbm_read(_ptr(buf), nbytes, _ptr(out_sum), workgroups, _stream(stream)),
           "xp_probe_hbm_read")


def probe_mfma_bf16(operands, workgroups: int, iters: int, out, stream=None):
    """Launch the bf16 MFMA probe; `operands` holds 8 x 64 x 2 x 16 bytes
    (8 x 64 x 2 x 8 bf16), `out` workgroups x 4 x 64 x 16 floats."""
    L = load_library()
    assert operands.numel() * operands.element_size() == 8 * 64 * 2 * 16
    assert out.numel() >= workgroups * 4 * 64 * 16
    _check(L.xp_probe_mfma_bf16(_ptr(operands), workgroups, iters, _ptr(out), _stream(stream)),
           "xp_probe_mfma_bf16")


def toeplitz_mixer(kappa, out=None, stream=None):
    """The full mixer L [r][B][B] of the Toeplitz form of Mix from its kernel
    taps kappa [r][B] (a device tensor, bf16 or float32; kappa[:, 0] unused),
    written by the device into `out` (allocated when None) for use as the
    weight "L"."""
    import torch
    L = load_library()
    assert kappa.dim() == 2 and kappa.is_contiguous()
    r, B = kappa.shape
    dt = {torch.float32: XP_F32, torch.bfloat16: XP_BF16}[kappa.dtype]
    if out is None:
        out = torch.empty((r, B, B), dtype=kappa.dtype, device=kappa.device)
    assert out.shape == (r, B, B) and out.dtype == kappa.dtype and out.is_contiguous()
    _check(L.xp_toeplitz_mixer(_ptr(kappa), r, B, dt, _ptr(out), _stream(stream)),
           "xp_toeplitz_mixer")
    return out


def layer_weights_struct(weights: Dict[str, object], H: int, n_heads: int, n_kv: int, ffn: int,
                         eps: float = 1e-6, theta: float = 1e6, head_dim: int = 128):
    """The xp_layer_weights record of a weight dict (LAYER_WEIGHT_NAMES to bf16
    device tensors)."""
    w = _LayerWeights(H=H, n_heads=n_heads, n_kv=n_kv, head_dim=head_dim, ffn=ffn, eps=eps,
                      rope_theta=theta)
    for n in LAYER_WEIGHT_NAMES:
        setattr(w, n, _ptr(weights[n]))
    return w


def layer_forward_noalloc(w, x, k_cache, v_cache, ctx_len, h_f32, h_bf16, causal=True,
                          stream=None):
    """xp_layer_forward_noalloc: one forward with the library's static
    scratch; `w` from layer_weights_struct, outputs preallocated by the
    caller (no allocation happens here or in the library)."""
    L = load_library()
    batch, B, _ = x.shape
    for t in (x, k_cache, v_cache, ctx_len, h_f32, h_bf16):
        assert t.is_contiguous()
    st = L.xp_layer_forward_noalloc(ctypes.byref(w), batch, B, 1 if causal else 0, _ptr(x),
                                    _ptr(k_cache), _ptr(v_cache), k_cache.shape[1],
                                    _ptr(ctx_len), _ptr(h_f32), _ptr(h_bf16), _stream(stream))
    if st != XP_OK:
        raise XpError(st, "xp_layer_forward_noalloc: " + L.xp_layer_last_error(None).decode())


class Layer:
    """The context layer (xp_layer_*): `weights` maps LAYER_WEIGHT_NAMES to
    bf16 device tensors, which must outlive the layer."""

    def __init__(self, weights: Dict[str, object], H: int, n_heads: int, n_kv: int, ffn: int,
                 max_batch: int, max_B: int, max_ctx: int, eps: float = 1e-6,
                 theta: float = 1e6, head_dim: int = 128):
        L = load_library()
        self._keep = dict(weights)
        w = _LayerWeights(H=H, n_heads=n_heads, n_kv=n_kv, head_dim=head_dim, ffn=ffn, eps=eps,
                          rope_theta=theta)
        for n in LAYER_WEIGHT_NAMES:
            setattr(w, n, _ptr(weights[n]))
        h = ctypes.c_void_p(0)
        st = L.xp_layer_create(ctypes.byref(w), max_batch, max_B, max_ctx, ctypes.byref(h))
        if st != XP_OK:
            raise XpError(st, "xp_layer_create: " + L.xp_layer_last_error(None).decode())
        self._h = h
        self.H = H

    def forward(self, x, k_cache, v_cache, ctx_len, causal=True, h_f32=None, h_bf16=None,
                stream=None):
        """x [batch][B][H] bf16; k_cache, v_cache [batch][C_max][n_kv][128] bf16;
        ctx_len [batch] int32 (device tensors).  Returns (h_f32, h_bf16)."""
        import torch
        L = load_library()
        batch, B, H = x.shape
        C_max = k_cache.shape[1]
        if h_f32 is None:
            h_f32 = torch.empty((batch, B, H), dtype=torch.float32, device=x.device)
        if h_bf16 is None:
            h_bf16 = torch.empty((batch, B, H), dtype=torch.bfloat16, device=x.device)
        for t in (x, k_cache, v_cache, ctx_len, h_f32, h_bf16):
            assert t.is_contiguous()
        st = L.xp_layer_forward(self._h, batch, B, 1 if causal else 0, _ptr(x), _ptr(k_cache),
                                _ptr(v_cache), C_max, _ptr(ctx_len), _ptr(h_f32), _ptr(h_bf16),
                                _stream(stream))
        if st != XP_OK:
            raise XpError(st, "xp_layer_forward: " + L.xp_layer_last_error(self._h).decode())
        return h_f32, h_bf16

    def close(self):
        if getattr(self, "_h", None):
            load_library().xp_layer_destroy(self._h)
            self._h = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass
