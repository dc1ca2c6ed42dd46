"""GPU parity of int8 weight storage (WN_I8: int8 codes with one fp32 scale per row) through the C
ABI, against the oracle's int8 mode, which quantizes with the same rule and uses code * scale
exactly.  Bars as for fp32 weights: teacher-forced logits within 1e-3, sample indices bit-exact at
every step whose oracle CDF margin exceeds 1e-4.  The logits' distance from the unquantized fp32
model is reported (it measures the quantization, not the kernels).  Cases cover every (r, s) pair,
one and several streams, nonzero biases, a zero weight row, and calls split at odd steps.
"""
import zlib

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

MARGIN = 1e-4
# the kernel the library picks for int8 models: the multi-CU kernel (which converts the codes to
# fp32 once, as it loads its resident weights) wherever it serves the shape, else the per-stream one
I8_KERNEL = {16: "stream_l2", 32: "multi_cu_chain", 64: "multi_cu_chain", 128: "multi_cu_chain"}

CASES = [
    # name, L, r, s, dilations, B, T, bias
    ("tiny_r16", 4, 16, 32, (1, 2, 4, 8), 2, 400, 0.3),
    ("r32_s128", 6, 32, 128, (1, 2, 4, 8, 16, 32), 2, 200, 0.2),
    ("l20_r64_b1", 20, 64, 256, tuple(synth.dilation_cycle(20)), 1, 300, 0.1),
    ("l9_r64_s128_b3", 9, 64, 128, (1, 1, 2, 1, 8, 1, 3, 1, 2), 3, 200, 0.3),
    ("l40_r64_b2", 40, 64, 256, tuple(synth.dilation_cycle(40)), 2, 120, 0.1),
    ("l20_r128_b3", 20, 128, 256, tuple(synth.dilation_cycle(20)), 3, 120, 0.2),
    ("l20_r64_b17", 20, 64, 256, tuple(synth.dilation_cycle(20)), 17, 100, 0.0),
]


STREAM_CASES = [c for c in CASES if c[0] in ("r32_s128", "l9_r64_s128_b3", "l20_r128_b3")]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_int8_parity(case, monkeypatch):
    _int8_case(case, monkeypatch, force_stream=False)


@pytest.mark.parametrize("case", STREAM_CASES, ids=[c[0] for c in STREAM_CASES])
def test_int8_parity_per_stream_kernel(case, monkeypatch):
    """The per-stream kernel's int8 rows (16 codes per lane and load) for r = 32, 64, 128 and
    s = 128, 256, which the multi-CU kernel serves by default."""
    _int8_case(case, monkeypatch, force_stream=True)


def _int8_case(case, monkeypatch, force_stream):
    import paper_1702_07825_amd as wn
    name, L, r, s, dil, B, T, bias = case
    if force_stream:
        monkeypatch.setenv("WN_KERNEL", "stream")
    seed = zlib.crc32(name.encode()) % 1000
    print("int8 case %s%s: L=%d r=%d s=%d B=%d T=%d" % (name, " (per-stream kernel)" if force_stream else "", L, r,
                                                      s, B, T), flush=True)
    w = synth.make_weights(L, r, s, seed=seed, bias_scale=bias)
    w["w_res"][0, 3] = 0.0  # a row of zeros: scale 0
    net = wn.WaveNet(w, dil, weight_dtype="i8")
    assert net.kernel_variant(B) == ("stream_l2" if force_stream else I8_KERNEL[r])
    cond = synth.make_cond(L, r, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    y = net.generate(cond, u)
    y2 = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    ws = net.new_workspace(B)
    parts, a = [], 0
    for b_ in (1, 2, 61, 62, T):
        parts.append(net.generate(cond[:, a:b_].contiguous(), u[:, a:b_].contiguous(), workspace=ws, reset=(a == 0)))
        a = b_
    torch.cuda.synchronize()
    assert net.status(ws) == 0
    assert torch.equal(y, y2)
    assert torch.equal(torch.cat(parts, 1), y)
    y_np, lg_np = y.cpu().numpy(), lg.cpu().numpy()
    assert y_np.min() >= 0 and y_np.max() <= 255
    cond_np, u_np = cond.cpu().numpy(), u.cpu().numpy()
    ys, lo, mg = oracle.run_streams(oracle.Model(w, dil, int8_weights=True), cond_np, u=u_np, y_in=y_np, threads=8)
    err = float(np.abs(lg_np - lo).max())
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[ok]))
    _, lo32, _ = oracle.run_streams(oracle.Model(w, dil), cond_np, y_in=y_np, threads=8)
    err32 = float(np.abs(lg_np - lo32).max())
    print("  max|dlogit| vs the int8 oracle %.3g (vs the unquantized fp32 model %.3g); confident %d/%d, "
          "mismatches %d" % (err, err32, int(ok.sum()), ok.size, mism), flush=True)
    assert err <= 1e-3
    assert mism == 0
    assert err32 < 0.5  # the quantized model stays close to the one it was made from
    net.close()
