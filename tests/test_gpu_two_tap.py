"""GPU parity of the two-tap input embedding (Section 5.1: x0 = E_prev[y_{t-2}] + E_cur[y_{t-1}] +
B_embed, y_{t-2} before the first step contributing nothing) in every kernel family, through the
C ABI, against the CPU oracle.

Bars as for the one-tap model: teacher-forced logits within max-abs 1e-3 of the oracle (fp32
weights; bf16 weights against the oracle's bf16 mode), sample indices bit-exact wherever the
oracle's CDF margin exceeds 1e-4.  Also: a call split in two (the state carries y_{t-2}) equals
one call bit for bit, and E_prev = 0 reproduces the one-table model bit for bit.
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
    # name, kernel forced ("" = the library's choice), expected variant, L, r, s, dil, B, T, dtype, bias
    ("stream_tiny", "stream", "stream_l2", 4, 16, 32, (1, 2, 4, 8), 3, 300, "f32", 0.4),
    ("stream_r16_bf16", "", "stream_l2", 3, 16, 32, (1, 2, 4), 2, 200, "bf16", 0.3),
    ("chain_l20_r64", "", "multi_cu_chain", 20, 64, 256, tuple(synth.dilation_cycle(20)), 1, 300, "f32", 0.1),
    ("chain_l20_r128_b3", "", "multi_cu_chain", 20, 128, 256, tuple(synth.dilation_cycle(20)), 3, 120, "f32", 0.0),
    ("chain_r32_b2", "", "multi_cu_chain", 6, 32, 128, (1, 2, 4, 8, 16, 32), 2, 200, "f32", 0.2),
    ("group_l20_b5", "mfma_group", "mfma_group", 20, 64, 256, tuple(synth.dilation_cycle(20)), 5, 140, "bf16", 0.1),
    ("group_l40_b17", "mfma_group", "mfma_group", 40, 64, 256, tuple(synth.dilation_cycle(40)), 17, 60, "bf16", 0.0),
    ("i8_l20_r64", "", I8_KERNEL, 20, 64, 256, tuple(synth.dilation_cycle(20)), 1, 200, "i8", 0.1),
    ("i8_stream_r16", "stream", "stream_l2", 3, 16, 32, (1, 2, 4), 2, 200, "i8", 0.3),
]


def _wn():
    import paper_1702_07825_amd as wn
    return wn


def _net(w, dil, dtype, kernel, monkeypatch):
    if kernel:
        monkeypatch.setenv("WN_KERNEL", kernel)
    else:
        monkeypatch.delenv("WN_KERNEL", raising=False)
    return _wn().WaveNet(w, dil, weight_dtype=dtype)


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_two_tap_parity(case, monkeypatch):
    name, kernel, variant, L, r, s, dil, B, T, dtype, bias = case
    print("two-tap case %s: L=%d r=%d s=%d B=%d T=%d %s" % (name, L, r, s, B, T, dtype), flush=True)
    seed = zlib.crc32(name.encode()) % 1000
    w = synth.make_weights(L, r, s, seed=seed, bias_scale=bias, embed_taps=2)
    net = _net(w, dil, dtype, kernel, monkeypatch)
    assert net.embed_taps == 2 and net.kernel_variant(B) == variant
    cond = synth.make_cond(L, r, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    y = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    y_np, lg_np = y.cpu().numpy(), lg.cpu().numpy()
    model = oracle.Model(w, dil, bf16_weights=(dtype == "bf16"), int8_weights=(dtype == "i8"))
    assert model.receptive_field == 2 + sum(dil)
    ys, lo, mg = oracle.run_streams(model, cond.cpu().numpy(), u=u.cpu().numpy(), y_in=y_np, threads=8)
    err = float(np.abs(lg_np - lo).max())
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[ok]))
    print("  max|dlogit|=%.3g low-margin steps=%d/%d mismatches=%d" % (err, int((~ok).sum()), ok.size, mism),
          flush=True)
    assert err <= LOGIT_TOL
    assert mism == 0

    # one call == two calls (the second starts from the state: y_{t-1} and y_{t-2})
    for split in (1, T // 3):
        ws = net.new_workspace(B)
        y1 = net.generate(cond[:, :split].contiguous(), u[:, :split].contiguous(), workspace=ws, reset=True)
        y2 = net.generate(cond[:, split:].contiguous(), u[:, split:].contiguous(), workspace=ws, reset=False)
        torch.cuda.synchronize()
        assert torch.equal(torch.cat([y1, y2], 1), y), "split at %d" % split
        ws = net.new_workspace(B)
        l1 = net.teacher_force(cond[:, :split].contiguous(), y[:, :split].contiguous(), workspace=ws, reset=True)
        l2 = net.teacher_force(cond[:, split:].contiguous(), y[:, split:].contiguous(), workspace=ws, reset=False)
        torch.cuda.synchronize()
        assert torch.equal(torch.cat([l1, l2], 1), lg), "teacher-forced split at %d" % split

    # E_prev = 0: the one-table model with E = E_cur, bit for bit
    w0 = dict(w)
    w0["embed"] = w["embed"].copy()
    w0["embed"][0] = 0.0
    w1 = dict(w)
    w1["embed"] = w["embed"][1].copy()
    n0, n1 = _net(w0, dil, dtype, kernel, monkeypatch), _net(w1, dil, dtype, kernel, monkeypatch)
    assert n0.kernel_variant(B) == n1.kernel_variant(B) == variant
    a_, b_ = n0.teacher_force(cond, y), n1.teacher_force(cond, y)
    torch.cuda.synchronize()
    assert torch.equal(a_, b_)
    for n in (net, n0, n1):
        n.close()
