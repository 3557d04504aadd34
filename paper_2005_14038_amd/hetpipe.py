"""Thin ctypes binding of libhetpipe.so (include/hetpipe.h).

Argument marshalling only: every step of the stage step and of the WSP update
runs in the library's HIP kernels.  Tensors are PyTorch device tensors (used
for device memory and streams); their ``data_ptr()`` is handed to the C ABI.
There is no fallback: if the library is missing or fails to load, importing
this module raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhetpipe.so")

HP_OK, HP_WOULD_BLOCK = 0, 1
HP_ERR_ARG, HP_ERR_STATE, HP_ERR_HIP, HP_ERR_NOMEM = -1, -2, -3, -4
HP_CONV, HP_FC, HP_RELU, HP_MAXPOOL, HP_BN, HP_ADD, HP_GAP, HP_SOFTMAX_CE = range(1, 9)
HP_FP32, HP_BF16 = 0, 1

EXPORTS = [
    "hp_stage_create", "hp_stage_destroy", "hp_stage_param_count", "hp_stage_param_layout",
    "hp_stage_output_shape", "hp_stage_device_bytes", "hp_stage_layer_bytes",
    "hp_stage_set_timing",
    "hp_stage_read_timing", "hp_stage_read_layer_timing", "hp_stage_forward",
    "hp_stage_backward", "hp_stage_backward_noalloc", "hp_stage_layer_buffers",
    "hp_ps_create", "hp_ps_destroy", "hp_ps_weights", "hp_ps_clock", "hp_ps_set_timing",
    "hp_ps_read_timing",
    "hp_vw_create", "hp_vw_destroy", "hp_vw_set_momentum", "hp_wsp_weights",
    "hp_wsp_local_update",
    "hp_wsp_push_wave", "hp_wsp_pull", "hp_wsp_wave_end", "hp_wsp_state", "hp_wsp_version",
    "hp_wsp_buffers", "hp_last_error",
]


class HPError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"hetpipe error {code}: {msg}")
        self.code = code


class hp_layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("in0", ctypes.c_int32), ("in1", ctypes.c_int32),
                ("C", ctypes.c_int32), ("K", ctypes.c_int32), ("R", ctypes.c_int32),
                ("S", ctypes.c_int32), ("stride", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("bias", ctypes.c_int32), ("eps", ctypes.c_float)]


class hp_wsp_state_t(ctypes.Structure):
    _fields_ = [("p", ctypes.c_int64), ("W", ctypes.c_int32), ("c", ctypes.c_int32),
                ("g", ctypes.c_int32), ("push_due", ctypes.c_int32), ("gated", ctypes.c_int32),
                ("next_slot", ctypes.c_int32), ("n_vw", ctypes.c_int32),
                ("in_flight", ctypes.c_int32)]


_lib = None
_vp = ctypes.c_void_p
_pp = ctypes.POINTER(ctypes.c_void_p)


def lib():
    """Load libhetpipe.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2005_14038_amd.build` (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    i32, sz = ctypes.c_int, ctypes.c_size_t
    L.hp_stage_create.argtypes = [ctypes.POINTER(hp_layer), i32, i32, i32, i32, i32, i32, _vp, _pp]
    L.hp_stage_destroy.argtypes = [_vp]
    L.hp_stage_param_count.argtypes = [_vp, ctypes.POINTER(sz)]
    L.hp_stage_param_layout.argtypes = [_vp, i32, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    L.hp_stage_output_shape.argtypes = [_vp, i32, ctypes.POINTER(ctypes.c_int * 3)]
    L.hp_stage_device_bytes.argtypes = [_vp, ctypes.POINTER(sz)]
    L.hp_stage_set_timing.argtypes = [_vp, i32]
    L.hp_stage_read_timing.argtypes = [_vp, ctypes.POINTER(ctypes.c_double * 2),
                                       ctypes.POINTER(ctypes.c_int64 * 2)]
    L.hp_stage_read_layer_timing.argtypes = [_vp, _vp, _vp, i32]
    L.hp_stage_layer_bytes.argtypes = [_vp, _vp, i32]
    L.hp_stage_forward.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp]
    L.hp_stage_backward.argtypes = [_vp, _vp, _vp, _vp, _vp]
    L.hp_stage_layer_buffers.argtypes = [_vp, i32, _pp, _pp]
    L.hp_stage_backward_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp]
    L.hp_ps_create.argtypes = [sz, _vp, i32, i32, _vp, _pp]
    L.hp_ps_destroy.argtypes = [_vp]
    L.hp_ps_weights.argtypes = [_vp, _pp]
    L.hp_ps_clock.argtypes = [_vp, ctypes.POINTER(i32)]
    L.hp_ps_set_timing.argtypes = [_vp, i32]
    L.hp_ps_read_timing.argtypes = [_vp, ctypes.POINTER(ctypes.c_double * 6),
                                    ctypes.POINTER(ctypes.c_int64 * 6)]
    L.hp_vw_create.argtypes = [_vp, i32, i32, _pp]
    L.hp_vw_destroy.argtypes = [_vp]
    L.hp_vw_set_momentum.argtypes = [_vp, ctypes.c_float]
    L.hp_wsp_weights.argtypes = [_vp, _pp]
    L.hp_wsp_local_update.argtypes = [_vp, _vp, ctypes.c_float]
    L.hp_wsp_push_wave.argtypes = [_vp, _vp]
    L.hp_wsp_pull.argtypes = [_vp, _vp]
    L.hp_wsp_wave_end.argtypes = [_vp, _vp, _vp, ctypes.c_float]
    L.hp_wsp_state.argtypes = [_vp, ctypes.POINTER(hp_wsp_state_t)]
    L.hp_wsp_version.argtypes = [_vp, ctypes.POINTER(ctypes.c_int64)]
    L.hp_wsp_buffers.argtypes = [_vp, _pp, ctypes.POINTER(sz), _pp]
    L.hp_last_error.restype = ctypes.c_char_p
    for name in EXPORTS:
        if name != "hp_last_error":
            getattr(L, name).restype = ctypes.c_int
    _lib = L
    return L


def _check(rc, allow=(HP_OK,)):
    if rc in allow:
        return rc
    raise HPError(rc, lib().hp_last_error().decode())


def _ptr(t):
    """Device pointer of a torch tensor (or an int address, or None)."""
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream_ptr(stream):
    if stream is None:
        return None
    return int(stream.cuda_stream) if hasattr(stream, "cuda_stream") else int(stream)


def make_layers(layers):
    """Convert a list of layer dicts into a ctypes hp_layer array."""
    arr = (hp_layer * len(layers))()
    for i, d in enumerate(layers):
        L = arr[i]
        L.kind = d["kind"]
        L.in0 = d.get("in0", i - 1)
        L.in1 = d.get("in1", -1)
        L.C = d.get("C", 0)
        L.K = d.get("K", 0)
        L.R = d.get("R", 1)
        L.S = d.get("S", d.get("R", 1))
        L.stride = d.get("stride", 1)
        L.pad = d.get("pad", 0)
        L.bias = 1 if d.get("bias", False) else 0
        L.eps = d.get("eps", 1e-5)
    return arr


class Stage:
    """One pipeline stage (hp_stage)."""

    def __init__(self, layers, batch, H, W, C, dtype="fp32", stream=None):
        self._L = lib()
        self.layers = layers
        self._arr = make_layers(layers)
        self.batch, self.H, self.W, self.C = batch, H, W, C
        self.dtype = dtype
        mode = HP_BF16 if dtype == "bf16" else HP_FP32
        h = ctypes.c_void_p()
        _check(self._L.hp_stage_create(self._arr, len(layers), batch, H, W, C, mode,
                                       _stream_ptr(stream), ctypes.byref(h)))
        self.h = h
        n = ctypes.c_size_t()
        _check(self._L.hp_stage_param_count(self.h, ctypes.byref(n)))
        self.P = n.value
        self.has_loss = layers[-1]["kind"] == HP_SOFTMAX_CE

    def close(self):
        if getattr(self, "h", None):
            self._L.hp_stage_destroy(self.h)
            self.h = None

    __del__ = close

    def param_layout(self, layer):
        o, n = ctypes.c_size_t(), ctypes.c_size_t()
        _check(self._L.hp_stage_param_layout(self.h, layer, ctypes.byref(o), ctypes.byref(n)))
        return o.value, n.value

    def output_shape(self, layer=-1):
        d = (ctypes.c_int * 3)()
        _check(self._L.hp_stage_output_shape(self.h, layer, ctypes.byref(d)))
        return tuple(d)

    def device_bytes(self):
        n = ctypes.c_size_t()
        _check(self._L.hp_stage_device_bytes(self.h, ctypes.byref(n)))
        return n.value

    def set_timing(self, on=True):
        _check(self._L.hp_stage_set_timing(self.h, 1 if on else 0))

    def read_timing(self):
        """({'contraction': ms, 'other': ms}, {'contraction': n, 'other': n}); resets."""
        ms = (ctypes.c_double * 2)()
        n = (ctypes.c_int64 * 2)()
        _check(self._L.hp_stage_read_timing(self.h, ctypes.byref(ms), ctypes.byref(n)))
        return ({"contraction": ms[0], "other": ms[1]},
                {"contraction": int(n[0]), "other": int(n[1])})

    def layer_bytes(self):
        """(per-layer device bytes, stage-level bytes)."""
        n = len(self.layers) + 1
        b = (ctypes.c_size_t * n)()
        _check(self._L.hp_stage_layer_bytes(self.h, ctypes.byref(b), n))
        return list(b)[:-1], b[n - 1]

    def read_layer_timing(self):
        """(fwd_ms, bwd_ms): per-layer device time of the timed passes since the
        last read, lists of n_layers + 1 (the last entry: stage-level work such
        as the bf16 weight copies); resets."""
        n = len(self.layers) + 1
        f = (ctypes.c_double * n)()
        b = (ctypes.c_double * n)()
        _check(self._L.hp_stage_read_layer_timing(self.h, ctypes.byref(f), ctypes.byref(b), n))
        return list(f), list(b)

    def forward(self, w, x, y=None, labels=None, loss=None):
        _check(self._L.hp_stage_forward(self.h, _ptr(w), _ptr(x), _ptr(y), _ptr(labels),
                                        _ptr(loss)))

    def layer_buffers(self, layer):
        """(value_ptr, grad_ptr) of layer `layer` after the last forward and
        backward passes (hp_stage_layer_buffers); None where the stage holds
        no such buffer."""
        v, g = ctypes.c_void_p(), ctypes.c_void_p()
        _check(self._L.hp_stage_layer_buffers(self.h, layer, ctypes.byref(v), ctypes.byref(g)))
        return v.value, g.value

    def backward(self, w, dy, dx, grad):
        _check(self._L.hp_stage_backward(self.h, _ptr(w), _ptr(dy), _ptr(dx), _ptr(grad)))

    def backward_noalloc(self, w, dy, dx, grad):
        """hp_stage_backward_noalloc: the backward pass with the library's
        static workspace (no device allocation)."""
        _check(self._L.hp_stage_backward_noalloc(self.h, _ptr(w), _ptr(dy), _ptr(dx), _ptr(grad)))


class ParameterServer:
    """hp_ps: global weights w_g and clock c_g in device memory."""

    def __init__(self, P, w0, N, D, stream=None):
        self._L = lib()
        h = ctypes.c_void_p()
        _check(self._L.hp_ps_create(P, _ptr(w0), N, D, _stream_ptr(stream), ctypes.byref(h)))
        self.h = h
        self.P, self.N, self.D = P, N, D

    def close(self):
        if getattr(self, "h", None):
            self._L.hp_ps_destroy(self.h)
            self.h = None

    __del__ = close

    def weights_ptr(self):
        p = ctypes.c_void_p()
        _check(self._L.hp_ps_weights(self.h, ctypes.byref(p)))
        return p.value

    def clock(self):
        c = ctypes.c_int()
        _check(self._L.hp_ps_clock(self.h, ctypes.byref(c)))
        return c.value

    TIMING_CLASSES = ("update_first", "update", "push", "pull", "wave_end_pull", "wave_end")

    def set_timing(self, on=True):
        _check(self._L.hp_ps_set_timing(self.h, 1 if on else 0))

    def read_timing(self):
        """({class: ms}, {class: launches}) of the WSP update kernels for the
        classes in TIMING_CLASSES; resets the sums."""
        ms = (ctypes.c_double * 6)()
        n = (ctypes.c_int64 * 6)()
        _check(self._L.hp_ps_read_timing(self.h, ctypes.byref(ms), ctypes.byref(n)))
        return ({k: ms[i] for i, k in enumerate(self.TIMING_CLASSES)},
                {k: int(n[i]) for i, k in enumerate(self.TIMING_CLASSES)})


class VirtualWorker:
    """hp_vw: one virtual worker's WSP state."""

    def __init__(self, ps: ParameterServer, vw_id, s_local):
        self._L = lib()
        self.ps = ps
        h = ctypes.c_void_p()
        _check(self._L.hp_vw_create(ps.h, vw_id, s_local, ctypes.byref(h)))
        self.h = h
        self.id = vw_id
        self.W = s_local + 1

    def close(self):
        if getattr(self, "h", None):
            self._L.hp_vw_destroy(self.h)
            self.h = None

    __del__ = close

    def set_momentum(self, mu):
        _check(self._L.hp_vw_set_momentum(self.h, ctypes.c_float(mu)))

    def weights(self):
        p = ctypes.c_void_p()
        _check(self._L.hp_wsp_weights(self.h, ctypes.byref(p)))
        return p.value

    def local_update(self, grad, lr):
        _check(self._L.hp_wsp_local_update(self.h, _ptr(grad), ctypes.c_float(lr)))

    def push_wave(self):
        _check(self._L.hp_wsp_push_wave(self.h, self.ps.h))

    def wave_end(self, grad, lr):
        """Local update + push + gate of a wave's last minibatch in one call
        (hp_wsp_wave_end).  Returns True if the VW may proceed, False if the
        clock bound blocks it (then pull() until it returns True)."""
        rc = _check(self._L.hp_wsp_wave_end(self.h, self.ps.h, _ptr(grad), ctypes.c_float(lr)),
                    allow=(HP_OK, HP_WOULD_BLOCK))
        return rc == HP_OK

    def pull(self):
        """Returns True if the VW may proceed, False if the clock bound blocks it."""
        rc = _check(self._L.hp_wsp_pull(self.h, self.ps.h), allow=(HP_OK, HP_WOULD_BLOCK))
        return rc == HP_OK

    def state(self):
        s = hp_wsp_state_t()
        _check(self._L.hp_wsp_state(self.h, ctypes.byref(s)))
        return {f: getattr(s, f) for f, _ in hp_wsp_state_t._fields_}

    def version(self):
        n = self.ps.N
        arr = (ctypes.c_int64 * n)()
        _check(self._L.hp_wsp_version(self.h, arr))
        return tuple(int(v) for v in arr)

    def buffers(self):
        r, u = ctypes.c_void_p(), ctypes.c_void_p()
        st = ctypes.c_size_t()
        _check(self._L.hp_wsp_buffers(self.h, ctypes.byref(r), ctypes.byref(st), ctypes.byref(u)))
        return r.value, st.value, u.value


# ---- device-to-device copies of raw library buffers (inspection only) ----
_hip = None


def _hiprt():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [_vp, _vp, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
        _hip.hipDeviceSynchronize.restype = ctypes.c_int
    return _hip


def copy_device(src_ptr: int, dst_tensor):
    """Copy dst_tensor.numel() elements from the device address src_ptr into dst_tensor."""
    h = _hiprt()
    rc = h.hipDeviceSynchronize()
    if rc != 0:
        raise RuntimeError(f"hipDeviceSynchronize failed ({rc})")
    rc = h.hipMemcpy(dst_tensor.data_ptr(), src_ptr,
                     dst_tensor.numel() * dst_tensor.element_size(), 3)
    if rc != 0:
        raise RuntimeError(f"hipMemcpy failed ({rc})")
    return dst_tensor


def read_vector(src_ptr: int, n: int) -> np.ndarray:
    """Read n fp32 values at a device address into a host array."""
    import torch
    t = torch.empty(n, dtype=torch.float32, device="cuda")
    copy_device(src_ptr, t)
    return t.cpu().numpy()
