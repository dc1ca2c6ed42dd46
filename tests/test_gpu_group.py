"""GPU parity of the batched MFMA kernel (bf16 weights, r = 64, any number of streams).

Each case runs through the C ABI and is compared with the CPU oracle in its bf16-weight mode
(teacher-forced logits within 1e-3, sample indices bit-exact wherever the oracle's CDF margin
exceeds 1e-4), with the fp32 oracle (2e-2) and with the per-stream kernel on the same inputs.
Cases cover one stream, full and partial groups, the fewest layers the kernel takes
(2, dilation 1), s = 128 and 256, dilations longer than the call, and calls split at odd steps.
A workgroup serves 8 streams (16 beyond 2048 streams); the two group sizes agree to rounding.
"""
import zlib

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

MARGIN = 1e-4


@pytest.fixture(autouse=True)
def _group_kernel(monkeypatch):
    # the batched kernel serves a bf16 model when selected by name (the default choice prefers the
    # multi-CU kernels where their replicas carry the batch)
    monkeypatch.setenv("WN_KERNEL", "mfma_group")


def _log(msg):
    print(msg, flush=True)


CASES = [
    # name, L, s, dilations, B, T, bias
    ("l2_d1_b1", 2, 128, (1, 1), 1, 300, 0.3),
    ("l3_b16", 3, 256, (1, 2, 4), 16, 200, 0.0),
    ("l3_d1_b5", 3, 256, (1, 1, 1), 5, 200, 0.2),
    ("l5_s128_b17", 5, 128, (1, 3, 9, 2, 4), 17, 150, 0.4),
    ("l20_b33", 20, 256, tuple(synth.dilation_cycle(20)), 33, 120, 0.1),
    ("l40_b20", 40, 256, tuple(synth.dilation_cycle(40)), 20, 60, 0.0),
    ("long_dilations_b18", 4, 256, (700, 1, 300, 2), 18, 400, 0.2),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_group_kernel_parity(case, monkeypatch):
    import paper_1702_07825_amd as wn
    name, L, s, dil, B, T, bias = case
    seed = zlib.crc32(name.encode()) % 1000
    _log("group case %s: L=%d s=%d B=%d T=%d" % (name, L, s, B, T))
    w = synth.make_weights(L, 64, s, seed=seed, bias_scale=bias)
    net = wn.WaveNet(w, dil, weight_dtype="bf16")
    assert net.kernel_variant(B) == "mfma_group"
    cond = synth.make_cond(L, 64, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    y = net.generate(cond, u)
    y2 = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    y_np, lg_np = y.cpu().numpy(), lg.cpu().numpy()
    cond_np, u_np = cond.cpu().numpy(), u.cpu().numpy()
    assert y_np.min() >= 0 and y_np.max() <= 255

    model = oracle.Model(w, dil, bf16_weights=True)
    ys, lo, mg = oracle.run_streams(model, cond_np, u=u_np, y_in=y_np, threads=8)
    err = float(np.abs(lg_np - lo).max())
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[ok]))
    _, lo32, _ = oracle.run_streams(oracle.Model(w, dil), cond_np, y_in=y_np, threads=8)
    err32 = float(np.abs(lg_np - lo32).max())
    _log("  max|dlogit| bf16 oracle %.3g, fp32 oracle %.3g; confident %d/%d, mismatches %d" %
         (err, err32, int(ok.sum()), ok.size, mism))
    assert err <= 1e-3
    assert err32 <= 2e-2
    assert mism == 0

    # a call split at odd steps continues exactly where the previous one stopped
    ws = net.new_workspace(B)
    parts, a = [], 0
    for b_ in (1, 2, 37, 38, T):
        parts.append(net.generate(cond[:, a:b_].contiguous(), u[:, a:b_].contiguous(), workspace=ws, reset=(a == 0)))
        a = b_
    ws2 = net.new_workspace(B)
    lgp = [net.teacher_force(cond[:, :29].contiguous(), y[:, :29].contiguous(), workspace=ws2, reset=True),
           net.teacher_force(cond[:, 29:].contiguous(), y[:, 29:].contiguous(), workspace=ws2, reset=False)]
    torch.cuda.synchronize()
    assert net.status(ws) == 0 and net.status(ws2) == 0
    assert torch.equal(torch.cat(parts, 1), y)
    assert torch.equal(torch.cat(lgp, 1), lg)

    # the per-stream kernel, which keeps the activations in fp32, agrees on the same inputs
    monkeypatch.setenv("WN_KERNEL", "stream")
    ref = wn.WaveNet(w, dil, weight_dtype="bf16")
    assert ref.kernel_variant(B) == "stream_l2"
    lg_ref = ref.teacher_force(cond, y)
    torch.cuda.synchronize()
    d_ref = float((lg_ref - lg).abs().max())
    _log("  max|dlogit| vs per-stream kernel %.3g" % d_ref)
    assert d_ref <= 1e-3
    ref.close()
    net.close()


@pytest.mark.parametrize("B", [5, 13, 16, 17])
def test_group_sizes_agree(B, monkeypatch):
    """8 and 16 streams per workgroup.  With 8, each MFMA pairs a stream's hi and lo parts in two
    columns (the sums meet in another order), so the two agree to rounding: logits within 1e-4 of
    each other, and each meets the oracle bars, also across a call split at an odd step."""
    import paper_1702_07825_amd as wn
    L, dil, T = 6, (1, 2, 4, 8, 1, 3), 90
    _log("group sizes, B=%d" % B)
    w = synth.make_weights(L, 64, 256, seed=B, bias_scale=0.2)
    cond = synth.make_cond(L, 64, B, T, seed=B, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=B), device="cuda")
    model = oracle.Model(w, dil, bf16_weights=True)
    cond_np, u_np = cond.cpu().numpy(), u.cpu().numpy()
    out = {}
    for gs in (8, 16):
        monkeypatch.setenv("WN_GROUP_STREAMS", str(gs))
        net = wn.WaveNet(w, dil, weight_dtype="bf16")
        assert net.kernel_variant(B) == "mfma_group"
        assert net.launch_info(B) == (-(-B // gs), -(-B // gs))
        y = net.generate(cond, u)
        lg = net.teacher_force(cond, y)
        ws = net.new_workspace(B)
        ya = net.generate(cond[:, :41].contiguous(), u[:, :41].contiguous(), workspace=ws, reset=True)
        yb = net.generate(cond[:, 41:].contiguous(), u[:, 41:].contiguous(), workspace=ws, reset=False)
        torch.cuda.synchronize()
        assert net.status(ws) == 0
        assert torch.equal(torch.cat([ya, yb], 1), y)
        y_np, lg_np = y.cpu().numpy(), lg.cpu().numpy()
        ys, lo, mg = oracle.run_streams(model, cond_np, u=u_np, y_in=y_np, threads=8)
        ok = mg > MARGIN
        assert float(np.abs(lg_np - lo).max()) <= 1e-3
        assert int(np.sum(ys[ok] != y_np[ok])) == 0
        out[gs] = (y_np, lg_np)
        net.close()
    # the same teacher-forced inputs through both group sizes
    monkeypatch.setenv("WN_GROUP_STREAMS", "16")
    net16 = wn.WaveNet(w, dil, weight_dtype="bf16")
    lg16 = net16.teacher_force(cond, torch.tensor(out[8][0], device="cuda"))
    torch.cuda.synchronize()
    d = float(np.abs(lg16.cpu().numpy() - out[8][1]).max())
    _log("  max|dlogit| between 8 and 16 streams per workgroup: %.3g" % d)
    assert d <= 1e-4
    net16.close()


def test_group_kernel_variant_selection(monkeypatch):
    import paper_1702_07825_amd as wn
    w = synth.make_weights(20, 64, 256, seed=2)
    monkeypatch.delenv("WN_KERNEL")
    dflt = wn.WaveNet(w, synth.dilation_cycle(20), weight_dtype="bf16")
    # the default: the fp32 multi-CU kernel (exact fp32 copy) up to 2 streams per replica, the MFMA
    # multi-CU kernel while its replicas carry the batch, then this one
    assert [dflt.kernel_variant(b) for b in (1, 16, 30)] == ["multi_cu_chain"] * 3
    assert [dflt.kernel_variant(b) for b in (31, 45, 256, 512)] == ["multi_cu_mfma"] * 4
    assert [dflt.kernel_variant(b) for b in (513, 2048)] == ["mfma_group"] * 2
    dflt.close()
    monkeypatch.setenv("WN_KERNEL", "mfma_group")
    net = wn.WaveNet(w, synth.dilation_cycle(20), weight_dtype="bf16")
    assert [net.kernel_variant(b) for b in (1, 16, 256)] == ["mfma_group"] * 3
    # 8 streams per workgroup up to 2048 streams (one workgroup per CU), then 16
    assert [net.launch_info(b) for b in (1, 9, 256, 2048, 2049)] == [(1, 1), (2, 2), (32, 32), (256, 256), (129, 129)]
    net.close()
    # one layer, or r other than 64, stays on the per-stream kernel when this one is asked for
    w1 = synth.make_weights(1, 64, 256, seed=2)
    net1 = wn.WaveNet(w1, (1,), weight_dtype="bf16")
    assert net1.kernel_variant(16) == "stream_l2"
    net1.close()
    w2 = synth.make_weights(4, 32, 128, seed=2)
    net2 = wn.WaveNet(w2, (1, 2, 4, 8), weight_dtype="bf16")
    assert net2.kernel_variant(16) == "stream_l2"
    net2.close()


def test_more_streams_than_eight_per_cu():
    """2049 streams: the default choice moves to 16 streams per workgroup (129 workgroups, the last
    holding one stream); sampled streams across the batch meet the oracle bars."""
    import paper_1702_07825_amd as wn
    L, dil, T, B = 2, (1, 2), 6, 2049
    _log("group: B=%d T=%d" % (B, T))
    w = synth.make_weights(L, 64, 128, seed=7, bias_scale=0.3)
    net = wn.WaveNet(w, dil, weight_dtype="bf16")
    assert net.kernel_variant(B) == "mfma_group"
    assert net.launch_info(B) == (129, 129)
    cond = synth.make_cond(L, 64, B, T, seed=7, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=7), device="cuda")
    ws = net.new_workspace(B)
    y = net.generate(cond, u, workspace=ws)
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    assert net.status(ws) == 0
    pick = np.array([0, 1, 15, 16, 17, 1000, 2031, 2032, 2047, 2048])
    y_np, lg_np = y.cpu().numpy()[pick], lg.cpu().numpy()[pick]
    model = oracle.Model(w, dil, bf16_weights=True)
    ys, lo, mg = oracle.run_streams(model, cond.cpu().numpy()[pick], u=u.cpu().numpy()[pick], y_in=y_np, threads=8)
    ok = mg > MARGIN
    assert float(np.abs(lg_np - lo).max()) <= 1e-3
    assert int(np.sum(ys[ok] != y_np[ok])) == 0
    net.close()
