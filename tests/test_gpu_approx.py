"""GPU parity of the approximate nonlinearities (the paper's Appendix C: tanh and sigmoid through
e~(x) = 1 + |x| + 0.5658 x^2 + 0.143 x^4, the softmax's e^x through the 2^x bit pattern) in every
kernel family, through the C ABI, against the oracle run with the same approximations.

Bars as for exact nonlinearities: teacher-forced logits within max-abs 1e-3 (bf16 weights against
the oracle's bf16 mode), sample indices bit-exact wherever the oracle's CDF margin exceeds 1e-4.
The GPU evaluates the same formulas in fp32 (reciprocals instead of divisions); the logits also
differ from the exact-nonlinearity run, so the option is in effect.
"""
import zlib

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

LOGIT_TOL = 1e-3
MARGIN = 1e-4
I8_KERNEL = "multi_cu_chain"  # the kernel int8 models with r = 64 run on

CASES = [
    # name, kernel forced, expected variant, L, r, s, dil, B, T, dtype, bias, taps
    ("stream_tiny", "stream", "stream_l2", 4, 16, 32, (1, 2, 4, 8), 2, 300, "f32", 0.4, 1),
    ("chain_l20_r64", "", "multi_cu_chain", 20, 64, 256, tuple(synth.dilation_cycle(20)), 1, 300, "f32", 0.2, 1),
    ("chain_l20_r128_b3_2tap", "", "multi_cu_chain", 20, 128, 256, tuple(synth.dilation_cycle(20)), 3, 100, "f32",
     0.1, 2),
    ("group_l20_b5", "mfma_group", "mfma_group", 20, 64, 256, tuple(synth.dilation_cycle(20)), 5, 140, "bf16", 0.2, 1),
    ("mfma_chain_l20_b9", "multi_cu_mfma", "multi_cu_mfma", 20, 64, 256, tuple(synth.dilation_cycle(20)), 9, 140,
     "bf16", 0.2, 1),
    ("mfma_chain_i8_l20_b17", "multi_cu_mfma", "multi_cu_mfma", 20, 64, 256, tuple(synth.dilation_cycle(20)), 17,
     100, "i8", 0.2, 1),
    ("i8_l20_r64_b2", "", I8_KERNEL, 20, 64, 256, tuple(synth.dilation_cycle(20)), 2, 150, "i8", 0.2, 1),
]


def _net(wn, w, dil, dtype, kernel, monkeypatch, approx):
    if kernel:
        monkeypatch.setenv("WN_KERNEL", kernel)
    else:
        monkeypatch.delenv("WN_KERNEL", raising=False)
    return wn.WaveNet(w, dil, weight_dtype=dtype, approx_nonlin=approx)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_approximate_nonlinearities_parity(case, monkeypatch):
    import paper_1702_07825_amd as wn
    name, kernel, variant, L, r, s, dil, B, T, dtype, bias, taps = case
    print("approx case %s: L=%d r=%d s=%d B=%d T=%d %s taps=%d" % (name, L, r, s, B, T, dtype, taps), flush=True)
    seed = zlib.crc32(name.encode()) % 1000
    w = synth.make_weights(L, r, s, seed=seed, bias_scale=bias, embed_taps=taps)
    net = _net(wn, w, dil, dtype, kernel, monkeypatch, True)
    assert net.kernel_variant(B) == variant
    cond = synth.make_cond(L, r, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    y = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    exact = _net(wn, w, dil, dtype, kernel, monkeypatch, False)
    lg_exact = exact.teacher_force(cond, y)
    torch.cuda.synchronize()
    y_np, lg_np = y.cpu().numpy(), lg.cpu().numpy()
    model = oracle.Model(w, dil, bf16_weights=(dtype == "bf16"), int8_weights=(dtype == "i8"), approx_nonlin=True)
    ys, lo, mg = oracle.run_streams(model, cond.cpu().numpy(), u=u.cpu().numpy(), y_in=y_np, threads=8)
    err = float(np.abs(lg_np - lo).max())
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[ok]))
    diff = float(np.abs(lg_np - lg_exact.cpu().numpy()).max())
    print("  max|dlogit|=%.3g low-margin steps=%d/%d mismatches=%d; vs exact nonlinearities %.3g" %
          (err, int((~ok).sum()), ok.size, mism, diff), flush=True)
    assert err <= LOGIT_TOL
    assert mism == 0
    assert diff > 1e-5

    # the other sampling rules draw through the same approximate exp
    for sampler in [(wn.SAMPLE_TEMPERATURE, 0.8, 256), (wn.SAMPLE_TOPK, 1.0, 16), (wn.SAMPLE_MEAN, 1.0, 256)]:
        ys2 = net.generate(cond, u, sampler=sampler)
        lg2 = net.teacher_force(cond, ys2)
        torch.cuda.synchronize()
        ys2_np = ys2.cpu().numpy()
        _, lo2, _ = oracle.run_streams(model, cond.cpu().numpy(), y_in=ys2_np, threads=8)
        assert float(np.abs(lg2.cpu().numpy() - lo2).max()) <= LOGIT_TOL
        bad = 0
        for b in range(B):
            for t in range(T):
                yo, m = oracle.sample(lo2[b, t], float(u[b, t]), sampler, approx_nonlin=True)
                if m > (1e-3 if sampler[0] == wn.SAMPLE_MEAN else MARGIN) and yo != ys2_np[b, t]:
                    bad += 1
        print("  sampler %s: mismatches at confident steps %d" % (sampler, bad), flush=True)
        assert bad == 0
    net.close()
    exact.close()
