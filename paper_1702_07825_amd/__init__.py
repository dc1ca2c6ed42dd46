"""Autoregressive WaveNet sample generation on AMD MI355X (gfx950).

Thin ctypes binding over ``libwn.so`` (the C ABI declared in ``include/wn.h``).
Every step of generation runs in the library's HIP kernels; this module only
checks tensor shapes and passes device pointers and the current HIP stream.
PyTorch provides device memory and streams.  There is no CPU fallback: without a
built ``libwn.so`` every entry point raises.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libwn.so")

WN_OK, WN_EINVAL, WN_EUNSUPPORTED, WN_ENOMEM, WN_EHIP, WN_ETIMEOUT, WN_EABORTED = 0, -1, -2, -3, -4, -5, -6
WN_F32, WN_BF16, WN_I8 = 0, 1, 2
WN_NONLIN_EXACT, WN_NONLIN_PAPER = 0, 1
A_CLASSES = 256
EXPORTED = ("wn_create", "wn_workspace_bytes", "wn_generate", "wn_generate_sampled", "wn_teacher_force", "wn_status",
            "wn_abort", "wn_kernel_variant", "wn_launch_info", "wn_destroy", "wn_error_string", "wn_last_error",
            "wn_cond_create", "wn_cond_workspace_bytes", "wn_condition", "wn_condition_static", "wn_cond_destroy")
# WN_COND_SCRATCH_BYTES of include/wn_cond.h: the largest scratch wn_condition_static takes
COND_SCRATCH_BYTES = 64 << 20
# wn_sample_mode_t: how a step's distribution becomes its sample
SAMPLE_DIRECT, SAMPLE_TEMPERATURE, SAMPLE_TOPK, SAMPLE_MODE, SAMPLE_MEAN = 0, 1, 2, 3, 4

_lib = None
_lock = threading.Lock()


class WnError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str = ""):
        self.code = code
        super().__init__("%s failed: %s (%d)%s" % (where, error_string(code), code, (": " + detail) if detail else ""))


class Config(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("r", ctypes.c_int32), ("s", ctypes.c_int32), ("a", ctypes.c_int32),
                ("dilations", ctypes.POINTER(ctypes.c_int32)), ("embed_taps", ctypes.c_int32),
                ("initial_sample", ctypes.c_int32), ("weight_dtype", ctypes.c_int32), ("nonlinearity", ctypes.c_int32)]


class Sampler(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("temperature", ctypes.c_float), ("top_k", ctypes.c_int32)]


class CondConfig(ctypes.Structure):
    _fields_ = [("n_features", ctypes.c_int32), ("h1", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("r", ctypes.c_int32), ("frame_rate", ctypes.c_int32), ("audio_rate", ctypes.c_int32)]


class CondWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.POINTER(ctypes.c_float)) for n in ("w1", "b1", "w2", "b2")]


WEIGHT_FIELDS = ("embed", "b_embed", "w_prev", "w_cur", "b_gate", "w_res", "b_res", "w_skip", "b_skip",
                 "w_relu", "b_relu", "w_out", "b_out")


class Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.POINTER(ctypes.c_float)) for n in WEIGHT_FIELDS]


def load_library(path: str = LIB_PATH):
    """Load libwn.so (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(path):
            raise RuntimeError("libwn.so is not built (%s); run __graft_entry__.build()" % path)
        L = ctypes.CDLL(path)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        L.wn_create.restype = ctypes.c_int
        L.wn_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Weights), ctypes.POINTER(vp)]
        L.wn_workspace_bytes.restype = sz
        L.wn_workspace_bytes.argtypes = [vp, i32]
        L.wn_generate.restype = ctypes.c_int
        L.wn_generate.argtypes = [vp, i32, i32, vp, vp, vp, vp, sz, i32, vp]
        L.wn_generate_sampled.restype = ctypes.c_int
        L.wn_generate_sampled.argtypes = [vp, i32, i32, vp, vp, vp, vp, sz, i32, ctypes.POINTER(Sampler), vp]
        L.wn_cond_create.restype = ctypes.c_int
        L.wn_cond_create.argtypes = [ctypes.POINTER(CondConfig), ctypes.POINTER(CondWeights), ctypes.POINTER(vp)]
        L.wn_cond_workspace_bytes.restype = sz
        L.wn_cond_workspace_bytes.argtypes = [vp, i32, i32]
        L.wn_condition.restype = ctypes.c_int
        L.wn_condition.argtypes = [vp, i32, i32, vp, i32, vp, vp, sz, vp]
        L.wn_condition_static.restype = ctypes.c_int
        L.wn_condition_static.argtypes = [vp, i32, i32, vp, i32, vp, vp]
        L.wn_cond_destroy.restype = None
        L.wn_cond_destroy.argtypes = [vp]
        L.wn_teacher_force.restype = ctypes.c_int
        L.wn_teacher_force.argtypes = [vp, i32, i32, vp, vp, vp, vp, sz, i32, vp]
        L.wn_status.restype = ctypes.c_int
        L.wn_status.argtypes = [vp, vp, vp]
        L.wn_abort.restype = ctypes.c_int
        L.wn_abort.argtypes = [vp, i32]
        L.wn_kernel_variant.restype = ctypes.c_char_p
        L.wn_kernel_variant.argtypes = [vp, i32]
        L.wn_launch_info.restype = ctypes.c_int
        L.wn_launch_info.argtypes = [vp, i32, ctypes.POINTER(i32), ctypes.POINTER(i32)]
        L.wn_destroy.restype = None
        L.wn_destroy.argtypes = [vp]
        L.wn_error_string.restype = ctypes.c_char_p
        L.wn_error_string.argtypes = [ctypes.c_int]
        L.wn_last_error.restype = ctypes.c_char_p
        L.wn_last_error.argtypes = []
        _lib = L
        return L


def error_string(code: int) -> str:
    return load_library().wn_error_string(code).decode()


def _check(rc: int, where: str):
    if rc != WN_OK:
        raise WnError(rc, where, load_library().wn_last_error().decode())


def _stream_handle(stream) -> Optional[int]:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dev_ptr(t, dtype, shape, name):
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch tensor" % name)
    if t.device.type != "cuda":
        raise ValueError("%s must be on a GPU device" % name)
    if t.dtype != dtype:
        raise ValueError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, got %s" % (name, tuple(shape), tuple(t.shape)))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t.data_ptr()


class WaveNet:
    """A WaveNet model resident on one GPU (wraps wn_create / wn_destroy).

    ``weights``: dict of fp32 host arrays with the row-major shapes of include/wn.h; ``embed`` is
    [a, r] (one tap) or [2, a, r] (two taps: tap 0 embeds y_{t-2}, tap 1 y_{t-1}).
    """

    def __init__(self, weights: Dict[str, np.ndarray], dilations: Sequence[int], initial_sample: int = 128,
                 weight_dtype: str = "f32", embed_taps: Optional[int] = None, approx_nonlin: bool = False):
        self._lib = load_library()
        self._h = None
        w = {k: np.ascontiguousarray(weights[k], dtype=np.float32) for k in WEIGHT_FIELDS}
        taps = 1 if w["embed"].ndim == 2 else int(w["embed"].shape[0])
        if embed_taps is not None and int(embed_taps) != taps:
            raise ValueError("embed_taps=%d but the embedding has %d tables" % (embed_taps, taps))
        self.embed_taps = taps
        embed_taps = taps
        L, two_r, r = w["w_prev"].shape
        self.n_layers, self.r, self.s, self.a = int(L), int(r), int(w["w_skip"].shape[1]), int(w["w_out"].shape[0])
        self.dilations = np.ascontiguousarray(dilations, dtype=np.int32)
        self.initial_sample = int(initial_sample)
        self.weight_dtype = weight_dtype
        cfg = Config(self.n_layers, self.r, self.s, self.a,
                     self.dilations.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), int(embed_taps),
                     self.initial_sample, {"f32": WN_F32, "bf16": WN_BF16, "i8": WN_I8}[weight_dtype],
                     WN_NONLIN_PAPER if approx_nonlin else WN_NONLIN_EXACT)
        self.approx_nonlin = bool(approx_nonlin)
        ws = Weights(*[w[k].ctypes.data_as(ctypes.POINTER(ctypes.c_float)) for k in WEIGHT_FIELDS])
        h = ctypes.c_void_p()
        _check(self._lib.wn_create(ctypes.byref(cfg), ctypes.byref(ws), ctypes.byref(h)), "wn_create")
        self._h = h

    def close(self):
        if self._h is not None:
            self._lib.wn_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_bytes(self, B: int) -> int:
        return int(self._lib.wn_workspace_bytes(self._h, int(B)))

    def new_workspace(self, B: int, device="cuda"):
        import torch
        return torch.empty(self.workspace_bytes(B), dtype=torch.uint8, device=device)

    def kernel_variant(self, B: int) -> str:
        return self._lib.wn_kernel_variant(self._h, int(B)).decode()

    def launch_info(self, B: int):
        """(workgroups, replicas) a call with B streams launches (see wn_launch_info)."""
        wg, rep = ctypes.c_int32(0), ctypes.c_int32(0)
        _check(self._lib.wn_launch_info(self._h, int(B), ctypes.byref(wg), ctypes.byref(rep)), "wn_launch_info")
        return int(wg.value), int(rep.value)

    def generate(self, cond, uniforms, samples=None, workspace=None, reset: bool = True, stream=None, sampler=None):
        """cond fp32 [B,T,l,2r], uniforms fp32 [B,T] (device) -> samples int32 [B,T].

        ``sampler``: None (direct sampling) or (mode, temperature, top_k) with mode one of the
        SAMPLE_* values (include/wn.h, wn_sampler)."""
        import torch
        B, T = int(cond.shape[0]), int(cond.shape[1])
        cp = _dev_ptr(cond, torch.float32, (B, T, self.n_layers, 2 * self.r), "cond")
        up = _dev_ptr(uniforms, torch.float32, (B, T), "uniforms")
        if samples is None:
            samples = torch.empty((B, T), dtype=torch.int32, device=cond.device)
        sp = _dev_ptr(samples, torch.int32, (B, T), "samples")
        if workspace is None:
            workspace = self.new_workspace(B, cond.device)
        if sampler is None:
            _check(self._lib.wn_generate(self._h, B, T, cp, up, sp, workspace.data_ptr(), workspace.numel(),
                                         1 if reset else 0, _stream_handle(stream)), "wn_generate")
        else:
            smp = Sampler(int(sampler[0]), float(sampler[1]), int(sampler[2]))
            _check(self._lib.wn_generate_sampled(self._h, B, T, cp, up, sp, workspace.data_ptr(), workspace.numel(),
                                                 1 if reset else 0, ctypes.byref(smp), _stream_handle(stream)),
                   "wn_generate_sampled")
        return samples

    def teacher_force(self, cond, y, logits=None, workspace=None, reset: bool = True, stream=None):
        """cond fp32 [B,T,l,2r], y int32 [B,T] (device) -> logits fp32 [B,T,a]."""
        import torch
        B, T = int(cond.shape[0]), int(cond.shape[1])
        cp = _dev_ptr(cond, torch.float32, (B, T, self.n_layers, 2 * self.r), "cond")
        yp = _dev_ptr(y, torch.int32, (B, T), "y")
        if logits is None:
            logits = torch.empty((B, T, self.a), dtype=torch.float32, device=cond.device)
        lp = _dev_ptr(logits, torch.float32, (B, T, self.a), "logits")
        if workspace is None:
            workspace = self.new_workspace(B, cond.device)
        _check(self._lib.wn_teacher_force(self._h, B, T, cp, yp, lp, workspace.data_ptr(), workspace.numel(),
                                          1 if reset else 0, _stream_handle(stream)), "wn_teacher_force")
        return logits

    def abort(self, on: bool = True):
        """wn_abort: ask this model's running and later calls to stop early (on=False withdraws it)."""
        _check(self._lib.wn_abort(self._h, 1 if on else 0), "wn_abort")

    def status(self, workspace, stream=None) -> int:
        """Synchronise the stream and return the kernel status word (0 = ok)."""
        return int(self._lib.wn_status(self._h, workspace.data_ptr(), _stream_handle(stream)))


class Conditioner:
    """The conditioning network on one GPU (wraps wn_cond_create / wn_cond_destroy, include/wn_cond.h).

    ``weights``: fp32 host arrays w1 [2, 3 h1, 2, F], b1 [2, 3 h1], w2 [2, 3 h2, 2, 2 h1], b2 [2, 3 h2]
    with h2 = n_layers * r.
    """

    def __init__(self, weights: Dict[str, np.ndarray], n_layers: int, r: int, frame_rate: int, audio_rate: int):
        self._lib = load_library()
        self._h = None
        w = {k: np.ascontiguousarray(weights[k], dtype=np.float32) for k in ("w1", "b1", "w2", "b2")}
        _, three_h1, _, F = w["w1"].shape
        self.n_features, self.h1 = int(F), int(three_h1 // 3)
        self.n_layers, self.r = int(n_layers), int(r)
        cfg = CondConfig(self.n_features, self.h1, self.n_layers, self.r, int(frame_rate), int(audio_rate))
        ws = CondWeights(*[w[k].ctypes.data_as(ctypes.POINTER(ctypes.c_float)) for k in ("w1", "b1", "w2", "b2")])
        h = ctypes.c_void_p()
        _check(self._lib.wn_cond_create(ctypes.byref(cfg), ctypes.byref(ws), ctypes.byref(h)), "wn_cond_create")
        self._h = h

    def close(self):
        if self._h is not None:
            self._lib.wn_cond_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_bytes(self, B: int, n_frames: int) -> int:
        return int(self._lib.wn_cond_workspace_bytes(self._h, int(B), int(n_frames)))

    def __call__(self, features, T: int, cond=None, workspace=None, stream=None):
        """features fp32 [B, n_frames, F] (device) -> cond fp32 [B, T, n_layers, 2r]."""
        import torch
        B, Tf = int(features.shape[0]), int(features.shape[1])
        fp = _dev_ptr(features, torch.float32, (B, Tf, self.n_features), "features")
        if cond is None:
            cond = torch.empty((B, T, self.n_layers, 2 * self.r), dtype=torch.float32, device=features.device)
        cp = _dev_ptr(cond, torch.float32, (B, T, self.n_layers, 2 * self.r), "cond")
        if workspace is None:
            workspace = torch.empty(max(self.workspace_bytes(B, Tf), 1), dtype=torch.uint8, device=features.device)
        _check(self._lib.wn_condition(self._h, B, Tf, fp, int(T), cp, workspace.data_ptr(), workspace.numel(),
                                      _stream_handle(stream)), "wn_condition")
        return cond

    def condition_static(self, features, T: int, cond, stream=None):
        """wn_condition_static: as __call__, with the library's static scratch instead of a workspace.
        ``cond`` (fp32 [B, T, n_layers, 2r], device) is required: this path allocates nothing."""
        import torch
        B, Tf = int(features.shape[0]), int(features.shape[1])
        fp = _dev_ptr(features, torch.float32, (B, Tf, self.n_features), "features")
        cp = _dev_ptr(cond, torch.float32, (B, T, self.n_layers, 2 * self.r), "cond")
        _check(self._lib.wn_condition_static(self._h, B, Tf, fp, int(T), cp, _stream_handle(stream)),
               "wn_condition_static")
        return cond
