"""CPU oracle for autoregressive WaveNet generation (Deep Voice, arXiv 1702.07825).

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package; the GPU library
(``paper_1702_07825_amd``) never does, and this package imports nothing from it.

The arithmetic lives in ``wn_oracle.c`` (plain sequential C, double precision),
built with gcc into ``liboracle.so`` next to it.  This module only marshals numpy
arrays into that library, plus the mu-law companding closed form (``mulaw``).

Pins of this oracle (tests/test_oracle_pins.py): a whole-sequence dilated
causal convolution written with torch's conv1d, the no-recurrence special case
as numpy matmuls, the head-and-sampler special case against numpy's
searchsorted, receptive field and causality, chunked == one-shot, the skip
concatenation identity, the paper's model-size and FLOP figures, and the other
sampling rules (temperature, top k, mode, mean) on a known distribution and
through their identities with direct sampling and the argmax.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Optional, Sequence

import numpy as np

from . import mulaw  # noqa: F401  (re-exported)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wn_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None
_lock = threading.Lock()


def build(force: bool = True) -> str:
    """Compile wn_oracle.c with gcc -O2 into liboracle.so (no intrinsics, no threads)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Model(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int), ("r", ctypes.c_int), ("s", ctypes.c_int), ("a", ctypes.c_int),
                ("dilations", ctypes.POINTER(ctypes.c_int)), ("initial_sample", ctypes.c_int),
                ("weight_format", ctypes.c_int), ("embed_taps", ctypes.c_int), ("approx_nonlin", ctypes.c_int)] + [
        (n, ctypes.POINTER(ctypes.c_float)) for n in
        ("embed", "b_embed", "w_prev", "w_cur", "b_gate", "w_res", "b_res", "w_skip", "b_skip",
         "w_relu", "b_relu", "w_out", "b_out")]


class _State(ctypes.Structure):
    _fields_ = [("t", ctypes.c_longlong), ("last_sample", ctypes.c_int), ("prev_sample", ctypes.c_int),
                ("hist", ctypes.POINTER(ctypes.c_double))]


def lib():
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                build(force=True)
            L = ctypes.CDLL(_LIB_PATH)
            L.oracle_run.restype = ctypes.c_int
            L.oracle_run.argtypes = [ctypes.POINTER(_Model), ctypes.POINTER(_State), ctypes.c_int, ctypes.c_longlong,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_void_p, ctypes.c_void_p]
            L.oracle_run_sampled.restype = ctypes.c_int
            L.oracle_run_sampled.argtypes = L.oracle_run.argtypes + [ctypes.c_int, ctypes.c_double, ctypes.c_int]
            L.oracle_approx_nonlin.restype = None
            L.oracle_approx_nonlin.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_longlong]
            L.oracle_sample_nl.restype = ctypes.c_int
            L.oracle_sample_nl.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_float, ctypes.c_int,
                                           ctypes.c_double, ctypes.c_int, ctypes.c_void_p]
            L.oracle_sample.restype = ctypes.c_int
            L.oracle_sample.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_float, ctypes.c_int, ctypes.c_double,
                                        ctypes.c_int, ctypes.c_void_p]
            L.oracle_condition.restype = ctypes.c_int
            L.oracle_condition.argtypes = [ctypes.POINTER(_CondModel), ctypes.c_longlong, ctypes.c_void_p,
                                           ctypes.c_longlong, ctypes.c_int, ctypes.c_int, ctypes.c_void_p]
            L.oracle_draw_nl.restype = ctypes.c_int
            L.oracle_draw_nl.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_float, ctypes.c_void_p,
                                         ctypes.c_void_p]
            L.oracle_draw.restype = ctypes.c_int
            L.oracle_draw.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p]
            L.oracle_history_len.restype = ctypes.c_longlong
            L.oracle_history_len.argtypes = [ctypes.POINTER(_Model)]
            L.oracle_reset.restype = None
            L.oracle_reset.argtypes = [ctypes.POINTER(_Model), ctypes.POINTER(_State)]
            L.oracle_param_count.restype = ctypes.c_longlong
            L.oracle_param_count.argtypes = [ctypes.c_int] * 4
            L.oracle_flops_per_sample.restype = ctypes.c_double
            L.oracle_flops_per_sample.argtypes = [ctypes.c_int] * 4 + [ctypes.c_double] * 2
            L.oracle_quantize_rows_i8.restype = None
            L.oracle_quantize_rows_i8.argtypes = [ctypes.c_void_p, ctypes.c_longlong, ctypes.c_longlong,
                                                  ctypes.c_void_p, ctypes.c_void_p]
            L.oracle_round_bf16_array.restype = None
            L.oracle_round_bf16_array.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_longlong]
            _lib = L
    return _lib


class _CondModel(ctypes.Structure):
    _fields_ = [("n_features", ctypes.c_int), ("h1", ctypes.c_int), ("h2", ctypes.c_int),
                ("w1", ctypes.POINTER(ctypes.c_float)), ("b1", ctypes.POINTER(ctypes.c_float)),
                ("w2", ctypes.POINTER(ctypes.c_float)), ("b2", ctypes.POINTER(ctypes.c_float))]


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Model:
    """A WaveNet parameter set as the oracle sees it (fp32 arrays, row-major [out][in]).

    ``embed`` is [a, r] (one tap: x0 = E[y_{t-1}] + B_embed) or [2, a, r] (two taps: tap 0
    embeds y_{t-2}, tap 1 y_{t-1})."""

    def __init__(self, weights: Dict[str, np.ndarray], dilations: Sequence[int], initial_sample: int = 128,
                 bf16_weights: bool = False, approx_nonlin: bool = False, int8_weights: bool = False):
        self.w = {k: np.ascontiguousarray(v, dtype=np.float32) for k, v in weights.items()}
        L, two_r, r = self.w["w_prev"].shape
        s = self.w["w_skip"].shape[1]
        a = self.w["w_out"].shape[0]
        assert two_r == 2 * r and len(dilations) == L and min(dilations) >= 1
        self.n_layers, self.r, self.s, self.a = L, r, s, a
        self.dilations = np.ascontiguousarray(dilations, dtype=np.int32)
        self.initial_sample = int(initial_sample)
        assert not (bf16_weights and int8_weights)
        self.bf16 = bool(bf16_weights)
        self.int8 = bool(int8_weights)
        e = self.w["embed"]
        assert e.shape[-2:] == (a, r) and (e.ndim == 2 or (e.ndim == 3 and e.shape[0] == 2)), e.shape
        self.embed_taps = 1 if e.ndim == 2 else 2
        m = _Model()
        m.n_layers, m.r, m.s, m.a = L, r, s, a
        m.dilations = self.dilations.ctypes.data_as(ctypes.POINTER(ctypes.c_int))
        m.initial_sample = self.initial_sample
        m.weight_format = 2 if self.int8 else (1 if self.bf16 else 0)
        m.embed_taps = self.embed_taps
        self.approx_nonlin = bool(approx_nonlin)
        m.approx_nonlin = int(self.approx_nonlin)
        for name in ("embed", "b_embed", "w_prev", "w_cur", "b_gate", "w_res", "b_res", "w_skip", "b_skip",
                     "w_relu", "b_relu", "w_out", "b_out"):
            setattr(m, name, self.w[name].ctypes.data_as(ctypes.POINTER(ctypes.c_float)))
        self._m = m

    @property
    def receptive_field(self) -> int:
        return receptive_field(self.dilations, self.embed_taps)


class State:
    """Per-stream generator state (histories + last sample) for chunked runs."""

    def __init__(self, model: Model):
        self.model = model
        n = int(lib().oracle_history_len(ctypes.byref(model._m)))
        self.hist = np.zeros(max(n, 1), np.float64)
        self._s = _State()
        self._s.hist = self.hist.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
        lib().oracle_reset(ctypes.byref(model._m), ctypes.byref(self._s))

    @property
    def t(self) -> int:
        return int(self._s.t)

    @property
    def last_sample(self) -> int:
        return int(self._s.last_sample)

    @property
    def prev_sample(self) -> int:
        return int(self._s.prev_sample)


# Ways of using the output distribution (Appendix "Sampling from Output Distribution"):
# (mode, temperature, top_k) with mode 0 direct, 1 temperature, 2 top k, 3 mode (argmax), 4 mean.
DIRECT = (0, 1.0, 256)
SAMPLE_MODES = {"direct": 0, "temperature": 1, "top_k": 2, "mode": 3, "mean": 4}


def run(model: Model, cond: np.ndarray, u: Optional[np.ndarray] = None, y_in: Optional[np.ndarray] = None,
        state: Optional[State] = None, want_logits: bool = True, sampler=DIRECT):
    """Run one stream for T = cond.shape[0] steps.

    Generation if ``y_in`` is None (needs ``u``), else teacher forcing on ``y_in``.  Draws use
    ``sampler`` = (mode, temperature, top_k).
    Returns (samples int32 [T] or None, logits float64 [T, a] or None, margins float64 [T] or None).
    """
    cond = np.ascontiguousarray(cond, dtype=np.float32)
    T = cond.shape[0]
    assert cond.shape[1:] == (model.n_layers, 2 * model.r), cond.shape
    mode = 0 if y_in is None else 1
    if u is not None:
        u = np.ascontiguousarray(u, dtype=np.float32)
        assert u.shape == (T,)
    if y_in is not None:
        y_in = np.ascontiguousarray(y_in, dtype=np.int32)
        assert y_in.shape == (T,)
        assert T == 0 or (y_in.min() >= 0 and y_in.max() < model.a)
    samples = np.zeros(T, np.int32) if (mode == 0 or u is not None) else None
    logits = np.zeros((T, model.a), np.float64) if want_logits else None
    margins = np.zeros(T, np.float64) if u is not None else None
    smode, temp, top_k = sampler
    rc = lib().oracle_run_sampled(ctypes.byref(model._m), None if state is None else ctypes.byref(state._s), mode, T,
                                  _ptr(cond), _ptr(u), _ptr(y_in), _ptr(samples), _ptr(logits), _ptr(margins),
                                  int(smode), float(temp), int(top_k))
    if rc != 0:
        raise RuntimeError("oracle_run failed with %d" % rc)
    return samples, logits, margins


def run_streams(model: Model, cond: np.ndarray, u: Optional[np.ndarray] = None, y_in: Optional[np.ndarray] = None,
                want_logits: bool = True, threads: int = 1, sampler=DIRECT):
    """``run`` over the leading stream axis of cond [B, T, l, 2r]; streams go to ``threads`` host threads."""
    B = cond.shape[0]

    def one(b):
        return run(model, cond[b], None if u is None else u[b], None if y_in is None else y_in[b],
                   want_logits=want_logits, sampler=sampler)

    if threads <= 1:
        res = [one(b) for b in range(B)]
    else:
        with ThreadPoolExecutor(max_workers=threads) as ex:
            res = list(ex.map(one, range(B)))

    def stack(i):
        return None if res[0][i] is None else np.stack([x[i] for x in res])

    return stack(0), stack(1), stack(2)


def draw(logits: np.ndarray, u: float, approx_nonlin: bool = False):
    """Direct sampling of one step: returns (index, probabilities, margin)."""
    lg = np.ascontiguousarray(logits, dtype=np.float64)
    p = np.zeros_like(lg)
    mg = ctypes.c_double(0.0)
    y = lib().oracle_draw_nl(int(bool(approx_nonlin)), lg.shape[0], _ptr(lg), ctypes.c_float(float(u)), _ptr(p),
                             ctypes.byref(mg))
    return int(y), p, float(mg.value)


def sample(logits: np.ndarray, u: float, sampler=DIRECT, approx_nonlin: bool = False):
    """One step's result under ``sampler`` = (mode, temperature, top_k): returns (index, margin)."""
    lg = np.ascontiguousarray(logits, dtype=np.float64)
    mg = ctypes.c_double(0.0)
    smode, temp, top_k = sampler
    y = lib().oracle_sample_nl(int(bool(approx_nonlin)), lg.shape[0], _ptr(lg), ctypes.c_float(float(u)), int(smode),
                               float(temp), int(top_k), ctypes.byref(mg))
    if y < 0:
        raise ValueError("invalid sampler %r" % (sampler,))
    return int(y), float(mg.value)


def condition(weights: Dict[str, np.ndarray], features: np.ndarray, n_audio: int, frame_rate: int,
              audio_rate: int) -> np.ndarray:
    """Conditioning network (Appendix A.2): features [Tf, F] -> cond [n_audio, 2 h2] (float64).

    ``weights``: w1 [2, 3 h1, 2, F], b1 [2, 3 h1], w2 [2, 3 h2, 2, 2 h1], b2 [2, 3 h2] (fp32)."""
    w = {k: np.ascontiguousarray(weights[k], dtype=np.float32) for k in ("w1", "b1", "w2", "b2")}
    x = np.ascontiguousarray(features, dtype=np.float32)
    Tf, F = x.shape
    h1, h2 = w["b1"].shape[1] // 3, w["b2"].shape[1] // 3
    assert w["w1"].shape == (2, 3 * h1, 2, F) and w["w2"].shape == (2, 3 * h2, 2, 2 * h1)
    m = _CondModel(F, h1, h2, *[w[k].ctypes.data_as(ctypes.POINTER(ctypes.c_float)) for k in ("w1", "b1", "w2", "b2")])
    out = np.zeros((n_audio, 2 * h2), np.float64)
    rc = lib().oracle_condition(ctypes.byref(m), Tf, _ptr(x), n_audio, int(frame_rate), int(audio_rate), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_condition failed with %d" % rc)
    return out


def round_bf16(x: np.ndarray) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    lib().oracle_round_bf16_array(_ptr(x), _ptr(out), x.size)
    return out


APPROX = {"tanh": 0, "sigmoid": 1, "exp": 2}


def approx_nonlin(which: str, x: np.ndarray) -> np.ndarray:
    """The approximate tanh, sigmoid or exp of Appendix C at every element of x (float64)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty_like(x)
    lib().oracle_approx_nonlin(APPROX[which], _ptr(x), _ptr(out), x.size)
    return out


def receptive_field(dilations: Sequence[int], embed_taps: int = 1) -> int:
    """R = taps + sum of dilations: samples y_{t-1-k}, k = 0..taps-1+sum(d), reach step t's distribution."""
    return int(embed_taps) + int(sum(int(d) for d in dilations))


def param_count(n_layers: int, r: int, s: int, a: int = 256) -> int:
    return int(lib().oracle_param_count(n_layers, r, s, a))


def flops_per_sample(n_layers: int, r: int, s: int, a: int = 256, f_div: float = 10.0, f_exp: float = 10.0) -> float:
    return float(lib().oracle_flops_per_sample(n_layers, r, s, a, f_div, f_exp))


def quantize_rows_i8(w: np.ndarray):
    """int8 weight storage of a matrix (the oracle's rule): returns (codes int8 [rows, cols],
    scales float32 [rows]) for the rows of w reshaped to [-1, w.shape[-1]]."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    cols = w.shape[-1]
    flat = w.reshape(-1, cols)
    codes = np.zeros(flat.shape, np.float32)
    scale = np.zeros(flat.shape[0], np.float32)
    lib().oracle_quantize_rows_i8(_ptr(flat), flat.shape[0], cols, _ptr(codes), _ptr(scale))
    return codes.astype(np.int8), scale
