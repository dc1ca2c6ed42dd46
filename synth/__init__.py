"""Seeded synthetic workloads for the autoregressive WaveNet generator.

This module serves both the GPU path and the CPU oracle, so it holds no
arithmetic of the method itself: only model sizes, dilation schedules and
seeded random inputs (weights, per-layer conditioning, per-step uniforms).

Model hyper-parameters follow the paper's notation (Appendix A.1,
"Auto-regressive WaveNet"): ``n_layers`` = l, ``r`` residual channels,
``s`` skip channels, ``a`` = 256 mu-law classes.  The paper never states
its dilation schedule; the workloads here use d_i = 2^(i mod 10), the
usual WaveNet cycle, and 1,2,4,8 for the tiny model.

Weight initialisation (the paper trains its weights; none ship with it):
every matrix is N(0, 1/fan_in), biases are zero unless ``bias_scale`` > 0.
fan_in per matrix: W_prev and W_cur 2r (the width-2 conv sees
[x_{t-d}; x_t]), W_res r, W_skip l*r (one projection of the concatenated
hidden states), W_relu s, W_out a, the embedding table 1 (its input is a
one-hot vector, so exactly one weight per output is active).

Conditioning [B, T, l, 2r] ~ N(0,1) fp32 and uniforms [B, T] ~ U[0,1) fp32
are drawn per stream from sub-seeds (seed+1, b) and (seed+2, b), so any
subset of streams can be regenerated alone.  Conditioning can be generated
on a GPU (torch's device generator) for the large batched workloads; the
oracle then consumes bytes copied back from that same device tensor.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Sequence

import numpy as np

A_CLASSES = 256
INITIAL_SAMPLE = 128  # y_{-1}: the mu-law code of silence (0.0)
SAMPLE_RATE_HZ = 16000
PAPER_SAMPLE_RATE_HZ = 16384


def dilation_cycle(n_layers: int, cycle: int = 10) -> List[int]:
    """d_i = 2^(i mod cycle), i = 0..n_layers-1."""
    return [1 << (i % cycle) for i in range(n_layers)]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_layers: int
    r: int
    s: int
    a: int
    dilations: tuple
    B: int
    T: int
    weight_dtype: str  # "f32", "bf16" or "i8" (storage); arithmetic is fp32 on the GPU
    description: str
    embed_taps: int = 1          # 2: the width-2 input convolution of Section 5.1
    sample_rate: int = 16000     # Hz of the audio the workload stands for

    @property
    def receptive_field(self) -> int:
        return self.embed_taps + sum(self.dilations)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 4, 16, 32, A_CLASSES, (1, 2, 4, 8), 1, 1600, "f32",
                     "l=4 (d=1,2,4,8), r=16, s=32, a=256, B=1, T=1600, fp32"),
    "l20_r64_b1": Workload("l20_r64_b1", 20, 64, 256, A_CLASSES, tuple(dilation_cycle(20)), 1, 16000, "f32",
                           "l=20 (d=2^(i mod 10)), r=64, s=256, a=256, B=1, T=16000, fp32"),
    "l40_r64_b1": Workload("l40_r64_b1", 40, 64, 256, A_CLASSES, tuple(dilation_cycle(40)), 1, 16000, "f32",
                           "l=40 (d=2^(i mod 10)), r=64, s=256, a=256, B=1, T=16000, fp32"),
    "l20_r128_b32": Workload("l20_r128_b32", 20, 128, 256, A_CLASSES, tuple(dilation_cycle(20)), 32, 16000, "f32",
                             "l=20 (d=2^(i mod 10)), r=128, s=256, a=256, B=32, T=16000, fp32"),
    "l20_r64_b256_bf16": Workload("l20_r64_b256_bf16", 20, 64, 256, A_CLASSES, tuple(dilation_cycle(20)), 256, 32000,
                                  "bf16",
                                  "l=20 (d=2^(i mod 10)), r=64, s=256, a=256, B=256, T=32000, "
                                  "bf16 weights, fp32 accumulate and activations"),
    "l20_r64_b1_i8": Workload("l20_r64_b1_i8", 20, 64, 256, A_CLASSES, tuple(dilation_cycle(20)), 1, 16000, "i8",
                              "l=20 (d=2^(i mod 10)), r=64, s=256, a=256, B=1, T=16000, "
                              "int8 weights (per-row scale), fp32 accumulate and activations"),
    "l20_r64_b256_i8": Workload("l20_r64_b256_i8", 20, 64, 256, A_CLASSES, tuple(dilation_cycle(20)), 256, 32000,
                                "i8",
                                "l=20 (d=2^(i mod 10)), r=64, s=256, a=256, B=256, T=32000, "
                                "int8 weights (per-row scale), fp32 accumulate and activations"),
    "l20_r64_b1_2tap_48k": Workload("l20_r64_b1_2tap_48k", 20, 64, 256, A_CLASSES, tuple(dilation_cycle(20)), 1,
                                    48000, "f32",
                                    "l=20 (d=2^(i mod 10)), r=64, s=256, a=256, two-tap input embedding, B=1, "
                                    "T=48000 (1 s at 48 kHz), fp32", embed_taps=2, sample_rate=48000),
}

WEIGHT_NAMES = ("embed", "b_embed", "w_prev", "w_cur", "b_gate", "w_res", "b_res",
                "w_skip", "b_skip", "w_relu", "b_relu", "w_out", "b_out")


def weight_shapes(n_layers: int, r: int, s: int, a: int, embed_taps: int = 1) -> Dict[str, tuple]:
    """Row-major [out][in] shapes of every parameter array (a two-tap embedding is [2, a, r]:
    tap 0 embeds y_{t-2}, tap 1 y_{t-1})."""
    L = n_layers
    return {
        "embed": (a, r) if embed_taps == 1 else (embed_taps, a, r), "b_embed": (r,),
        "w_prev": (L, 2 * r, r), "w_cur": (L, 2 * r, r), "b_gate": (L, 2 * r),
        "w_res": (L, r, r), "b_res": (L, r),
        "w_skip": (L, s, r), "b_skip": (s,),
        "w_relu": (a, s), "b_relu": (a,),
        "w_out": (a, a), "b_out": (a,),
    }


def fan_in(name: str, n_layers: int, r: int, s: int, a: int, embed_taps: int = 1) -> Optional[int]:
    return {"embed": embed_taps, "w_prev": 2 * r, "w_cur": 2 * r, "w_res": r,
            "w_skip": n_layers * r, "w_relu": s, "w_out": a}.get(name)


def make_weights(n_layers: int, r: int, s: int, a: int = A_CLASSES, seed: int = 0,
                 bias_scale: float = 0.0, weight_scale: float = 1.0, embed_taps: int = 1) -> Dict[str, np.ndarray]:
    """fp32 host weights; matrices N(0, weight_scale^2/fan_in), biases N(0, bias_scale^2) (zero by default)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = {}
    for name, shape in weight_shapes(n_layers, r, s, a, embed_taps).items():
        fi = fan_in(name, n_layers, r, s, a, embed_taps)
        if fi is None:
            if bias_scale > 0:
                out[name] = (rng.standard_normal(shape) * bias_scale).astype(np.float32)
            else:
                out[name] = np.zeros(shape, np.float32)
        else:
            out[name] = (rng.standard_normal(shape) * (weight_scale / np.sqrt(fi))).astype(np.float32)
    return out


def _stream_seed(seed: int, salt: int, b: int) -> int:
    return (seed * 1000003 + salt * 7919 + b * 104729) & 0x7FFFFFFF


def make_uniforms(B: int, T: int, seed: int = 0, streams: Optional[Sequence[int]] = None) -> np.ndarray:
    """fp32 U[0,1) per step, [len(streams), T]; stream b uses sub-seed (seed+2, b)."""
    streams = range(B) if streams is None else streams
    rows = []
    for b in streams:
        rng = np.random.Generator(np.random.PCG64(_stream_seed(seed, 2, b)))
        rows.append(rng.random(T, dtype=np.float32))
    return np.stack(rows) if rows else np.zeros((0, T), np.float32)


def make_cond(n_layers: int, r: int, B: int, T: int, seed: int = 0, device: str = "cpu",
              streams: Optional[Sequence[int]] = None, out=None):
    """fp32 N(0,1) conditioning [len(streams), T, l, 2r] as a torch tensor on ``device``.

    Stream b draws from its own torch generator seeded (seed+1, b) on that device, so a
    CPU-generated and a GPU-generated workload differ; the oracle always consumes the
    bytes of whichever tensor the GPU path used.
    """
    import torch
    streams = list(range(B)) if streams is None else list(streams)
    if out is None:
        out = torch.empty((len(streams), T, n_layers, 2 * r), dtype=torch.float32, device=device)
    dev = torch.device(device)
    for i, b in enumerate(streams):
        g = torch.Generator(device=dev)
        g.manual_seed(_stream_seed(seed, 1, b))
        torch.randn((T, n_layers, 2 * r), generator=g, dtype=torch.float32, device=dev, out=out[i])
    return out


def make_samples(B: int, T: int, a: int = A_CLASSES, seed: int = 0) -> np.ndarray:
    """int32 sample indices in [0, a) for teacher-forced runs (any sequence is valid input)."""
    rng = np.random.Generator(np.random.PCG64(_stream_seed(seed, 3, 0)))
    return rng.integers(0, a, size=(B, T), dtype=np.int32)


# ---------------------------------------------------------------------------------------------
# Conditioning network inputs (Appendix A.2 "Conditioning Network" and "Input Featurization")
# ---------------------------------------------------------------------------------------------
N_PHONEMES = 40      # 39 ARPABET phonemes + silence
N_STRESS = 5         # no, primary, secondary, tertiary, quaternary stress
N_FEATURES = 5 * (N_PHONEMES + N_STRESS) + 2  # 227: five phonemes in context, voiced flag, log F0
FRAME_RATE_HZ = 256
COND_H1 = 256        # channels per direction of the first QRNN layer (the paper gives no size)


def make_features(B: int, n_frames: int, seed: int, min_dur: int = 8, max_dur: int = 40) -> np.ndarray:
    """Seeded features [B, n_frames, 227] with the paper's layout: for the current phoneme, the two
    before it and the two after it, a 40-way identity one-hot and a 5-way stress one-hot (the last
    two stress levels never occur, as in datasets without them), then a voiced flag and a
    normalised log F0 in [-1, 1] (0 when unvoiced).  Phonemes last min_dur..max_dur frames."""
    out = np.zeros((B, n_frames, N_FEATURES), np.float32)
    for b in range(B):
        rng = np.random.default_rng((seed, b))
        ids, stress, voiced, durs = [], [], [], []
        while sum(durs) < n_frames + 2 * max_dur:
            ids.append(int(rng.integers(N_PHONEMES)))
            stress.append(int(rng.integers(3)))
            voiced.append(bool(rng.random() < 0.6))
            durs.append(int(rng.integers(min_dur, max_dur + 1)))
        starts = np.cumsum([0] + durs)
        f0 = np.clip(np.cumsum(rng.normal(0.0, 0.05, n_frames)) * 0.5 + rng.uniform(-0.5, 0.5), -1.0, 1.0)
        for t in range(n_frames):
            p = int(np.searchsorted(starts, t, side="right")) - 1
            for c, q in enumerate(range(p - 2, p + 3)):
                if 0 <= q < len(ids):
                    out[b, t, c * N_PHONEMES + ids[q]] = 1.0
                    out[b, t, 5 * N_PHONEMES + c * N_STRESS + stress[q]] = 1.0
            if voiced[p]:
                out[b, t, N_FEATURES - 2] = 1.0
                out[b, t, N_FEATURES - 1] = f0[t]
    return out


def make_cond_weights(n_features: int, h1: int, h2: int, seed: int, bias_scale: float = 0.0) -> Dict[str, np.ndarray]:
    """Seeded conditioning-network weights: w1 [2, 3 h1, 2, F], b1 [2, 3 h1], w2 [2, 3 h2, 2, 2 h1],
    b2 [2, 3 h2] (direction, gate rows h~ / o / f, convolution tap, input); matrices N(0, 1/fan_in)
    with fan_in = 2 x inputs (the width-2 convolution), biases 0 unless bias_scale > 0."""
    rng = np.random.default_rng((seed, 77))
    w = {}
    for name, h, cin in (("1", h1, n_features), ("2", h2, 2 * h1)):
        w["w" + name] = (rng.standard_normal((2, 3 * h, 2, cin)) / np.sqrt(2 * cin)).astype(np.float32)
        w["b" + name] = (rng.standard_normal((2, 3 * h)) * bias_scale).astype(np.float32)
    return w


@dataclasses.dataclass(frozen=True)
class CondWorkload:
    name: str
    n_features: int
    h1: int
    n_layers: int
    r: int
    B: int
    n_frames: int
    frame_rate: int
    audio_rate: int
    description: str

    @property
    def T(self) -> int:
        return self.n_frames * self.audio_rate // self.frame_rate


def _cond_wl(name, n_layers, r, B, seconds):
    fr, ar = FRAME_RATE_HZ, SAMPLE_RATE_HZ
    return CondWorkload(name, N_FEATURES, COND_H1, n_layers, r, B, seconds * fr, fr, ar,
                        "conditioning network: %d features at %d Hz -> l=%d x 2r=%d at %d Hz, h1=%d, B=%d, %d s"
                        % (N_FEATURES, fr, n_layers, 2 * r, ar, COND_H1, B, seconds))


COND_WORKLOADS = {
    "cond_l20_r64_b1": _cond_wl("cond_l20_r64_b1", 20, 64, 1, 1),
    "cond_l20_r64_b256": _cond_wl("cond_l20_r64_b256", 20, 64, 256, 2),
}
