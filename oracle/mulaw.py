"""mu-law companding for a = 256 classes (Appendix A.1 uses 8-bit mu-law audio and
defers to WaveNet's Section 2.2 for the transform f(x) = sign(x) ln(1 + mu|x|) / ln(1 + mu),
mu = 255).  TEST INFRASTRUCTURE ONLY; the GPU path works on integer sample codes.

Quantisation reading: code = clamp(floor((f(x) + 1) / 2 * 255 + 1/2), 0, 255);
decoding maps a code to g = 2 code / 255 - 1 and inverts f exactly.
"""
import numpy as np

MU = 255.0


def compress(x):
    x = np.asarray(x, dtype=np.float64)
    return np.sign(x) * np.log1p(MU * np.abs(x)) / np.log1p(MU)


def expand(g):
    g = np.asarray(g, dtype=np.float64)
    return np.sign(g) * ((1.0 + MU) ** np.abs(g) - 1.0) / MU


def encode(x):
    f = compress(np.clip(np.asarray(x, dtype=np.float64), -1.0, 1.0))
    return np.clip(np.floor((f + 1.0) / 2.0 * 255.0 + 0.5), 0, 255).astype(np.int32)


def decode(code):
    g = 2.0 * np.asarray(code, dtype=np.float64) / 255.0 - 1.0
    return expand(g)
