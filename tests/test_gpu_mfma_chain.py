"""GPU parity of the multi-CU MFMA kernel (bf16 and int8 weights, r = 64): the streams of a replica
carried together through chain CUs with resident weights, 8 per replica in paired columns (the
default) or 16, one per column (WN_MFMA_COLUMNS=16, the layout of the largest batches), with
front-loaded aux layer runs (the default) or uniform ones (WN_AUX_LAYERS=5).

Each case runs through the C ABI and is compared with the CPU oracle in the matching weight mode
(bf16, or int8 with its quantization rule): teacher-forced logits within 1e-3, sample indices
bit-exact wherever the oracle's CDF margin exceeds 1e-4; with the fp32 oracle within 2e-2 for bf16
models.  Cases cover one stream, a full replica of 16, several replicas with a partial one, the
fewest layers, every dilation 1 (histories read in the step they are written), dilations longer
than the call, 40 layers (four chain CUs), int8 weights with a zero row, two taps, and calls split
at odd steps (one-shot and chunked runs agree bit for bit), in both column layouts.  The batched
MFMA kernel (one CU per group of streams) agrees with it to rounding on the same inputs.
"""
import zlib

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

MARGIN = 1e-4
KERNEL = "multi_cu_mfma"


def _log(msg):
    print(msg, flush=True)


CASES = [
    # name, L, dilations, B, T, dtype, bias, taps, columns (8: paired, 16: one stream per column)
    ("l20_b1", 20, tuple(synth.dilation_cycle(20)), 1, 300, "bf16", 0.1, 1, 8),
    ("l20_b16", 20, tuple(synth.dilation_cycle(20)), 16, 200, "bf16", 0.2, 1, 8),
    ("l20_b37", 20, tuple(synth.dilation_cycle(20)), 37, 120, "bf16", 0.0, 1, 8),
    ("l2_d1_b1", 2, (1, 1), 1, 300, "bf16", 0.3, 1, 8),
    ("l3_d1_b3", 3, (1, 1, 1), 3, 200, "bf16", 0.2, 1, 8),
    ("l5_b5", 5, (1, 3, 9, 2, 4), 5, 150, "bf16", 0.4, 1, 8),
    ("long_dilations_b2", 4, (700, 1, 300, 2), 2, 800, "bf16", 0.2, 1, 8),
    ("l40_b20", 40, tuple(synth.dilation_cycle(40)), 20, 60, "bf16", 0.0, 1, 8),
    ("l20_2tap_b3", 20, tuple(synth.dilation_cycle(20)), 3, 150, "bf16", 0.1, 2, 8),
    ("i8_l20_b3", 20, tuple(synth.dilation_cycle(20)), 3, 200, "i8", 0.2, 1, 8),
    ("i8_l9_b17", 9, (1, 1, 2, 1, 8, 1, 3, 1, 2), 17, 120, "i8", 0.3, 1, 8),
    ("c16_l20_b16", 20, tuple(synth.dilation_cycle(20)), 16, 200, "bf16", 0.2, 1, 16),
    ("c16_l20_b37", 20, tuple(synth.dilation_cycle(20)), 37, 120, "bf16", 0.0, 1, 16),
    ("c16_l3_d1_b3", 3, (1, 1, 1), 3, 200, "bf16", 0.2, 1, 16),
    ("c16_l40_b20", 40, tuple(synth.dilation_cycle(40)), 20, 60, "bf16", 0.0, 1, 16),
    ("c16_l20_2tap_b3", 20, tuple(synth.dilation_cycle(20)), 3, 150, "bf16", 0.1, 2, 16),
    ("c16_i8_l9_b17", 9, (1, 1, 2, 1, 8, 1, 3, 1, 2), 17, 120, "i8", 0.3, 1, 16),
    # uniform aux runs of 5 layers (the layout of batches whose front-loaded replicas do not fit)
    ("u5_l20_b16", 20, tuple(synth.dilation_cycle(20)), 16, 200, "bf16", 0.2, 1, 8),
    ("u5_i8_l20_b37", 20, tuple(synth.dilation_cycle(20)), 37, 120, "i8", 0.1, 1, 8),
    ("u5_c16_l20_b17", 20, tuple(synth.dilation_cycle(20)), 17, 120, "bf16", 0.1, 1, 16),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_mfma_chain_parity(case, monkeypatch):
    import paper_1702_07825_amd as wn
    name, L, dil, B, T, dtype, bias, taps, cols = case
    seed = zlib.crc32(name.encode()) % 1000
    _log("multi-CU MFMA case %s: L=%d B=%d T=%d %s taps=%d columns=%d" % (name, L, B, T, dtype, taps, cols))
    monkeypatch.setenv("WN_KERNEL", KERNEL)
    if cols == 16:
        monkeypatch.setenv("WN_MFMA_COLUMNS", "16")
    else:
        monkeypatch.delenv("WN_MFMA_COLUMNS", raising=False)
    if name.startswith("u5_"):
        monkeypatch.setenv("WN_AUX_LAYERS", "5")
    else:
        monkeypatch.delenv("WN_AUX_LAYERS", raising=False)
    w = synth.make_weights(L, 64, 256, seed=seed, bias_scale=bias, embed_taps=taps)
    if dtype == "i8":
        w["w_res"][0, 3] = 0.0  # a row of zeros: scale 0
    net = wn.WaveNet(w, dil, weight_dtype=dtype)
    assert net.kernel_variant(B) == KERNEL
    cond = synth.make_cond(L, 64, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    y = net.generate(cond, u)
    y2 = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    assert net.status(net.new_workspace(B)) == 0
    assert torch.equal(y, y2)
    y_np, lg_np = y.cpu().numpy(), lg.cpu().numpy()
    cond_np, u_np = cond.cpu().numpy(), u.cpu().numpy()
    assert y_np.min() >= 0 and y_np.max() <= 255

    mode = {"bf16_weights": True} if dtype == "bf16" else {"int8_weights": True}
    model = oracle.Model(w, dil, **mode)
    ys, lo, mg = oracle.run_streams(model, cond_np, u=u_np, y_in=y_np, threads=8)
    err = float(np.abs(lg_np - lo).max())
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[ok]))
    _log("  max|dlogit| oracle (%s) %.3g; confident %d/%d, mismatches %d" % (dtype, err, int(ok.sum()), ok.size, mism))
    assert err <= 1e-3
    assert mism == 0
    if dtype == "bf16":
        _, lo32, _ = oracle.run_streams(oracle.Model(w, dil), cond_np, y_in=y_np, threads=8)
        err32 = float(np.abs(lg_np - lo32).max())
        _log("  max|dlogit| fp32 oracle %.3g" % err32)
        assert err32 <= 2e-2

    # calls split at odd steps continue exactly where the previous one stopped
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
    net.close()

    if dtype == "bf16" and taps == 1:
        # the batched MFMA kernel (every layer of a group on one CU) agrees on the same inputs
        monkeypatch.setenv("WN_KERNEL", "mfma_group")
        ref = wn.WaveNet(w, dil, weight_dtype=dtype)
        assert ref.kernel_variant(B) == "mfma_group"
        lg_ref = ref.teacher_force(cond, y)
        torch.cuda.synchronize()
        d_ref = float((lg_ref - lg).abs().max())
        _log("  max|dlogit| vs the batched kernel %.3g" % d_ref)
        assert d_ref <= 1e-3
        ref.close()


def test_mfma_chain_launch_layout(monkeypatch):
    """l = 20: replicas of up to 8 streams in paired columns take 2 chain CUs, 1 head CU and 5 aux CUs
    (front-loaded layer runs 5, 5, 5, 3, 2) while 8 CUs per replica fit the chip (32 replicas), else
    4 aux CUs of 5 layers (up to 36 replicas); larger batches take replicas of up to 16 streams with
    2 chain, 2 head and 5 or 4 aux CUs (up to 32 replicas)."""
    import paper_1702_07825_amd as wn
    monkeypatch.setenv("WN_KERNEL", KERNEL)
    monkeypatch.delenv("WN_MFMA_COLUMNS", raising=False)
    monkeypatch.delenv("WN_AUX_LAYERS", raising=False)
    L = 20
    w = synth.make_weights(L, 64, 256, seed=3)
    net = wn.WaveNet(w, synth.dilation_cycle(L), weight_dtype="bf16")
    for B, cus in ((1, 8), (8, 8), (9, 16), (16, 16), (17, 24), (256, 256), (257, 231), (288, 252), (289, 171),
                   (512, 256)):
        assert net.kernel_variant(B) == KERNEL
        assert net.launch_info(B)[0] == cus, B
    assert net.kernel_variant(513) != KERNEL
    monkeypatch.setenv("WN_MFMA_COLUMNS", "16")
    for B, cus in ((1, 9), (17, 18), (256, 144)):
        assert net.launch_info(B)[0] == cus, B
    monkeypatch.delenv("WN_MFMA_COLUMNS")
    monkeypatch.setenv("WN_AUX_LAYERS", "5")
    for B, cus in ((1, 7), (256, 224)):
        assert net.launch_info(B)[0] == cus, B
    net.close()


def test_mfma_chain_timeout_then_reset(monkeypatch):
    """A wait that gives up (forced from the host with a spin limit of 1) ends the call with
    WN_ETIMEOUT and every block leaves; a run from zero on the same workspace is then correct."""
    import paper_1702_07825_amd as wn
    monkeypatch.setenv("WN_KERNEL", KERNEL)
    L, B, T = 20, 3, 64
    w = synth.make_weights(L, 64, 256, seed=5, bias_scale=0.1)
    dil = synth.dilation_cycle(L)
    cond = synth.make_cond(L, 64, B, T, seed=5, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=5), device="cuda")
    good = wn.WaveNet(w, dil, weight_dtype="bf16")
    y_ref = good.generate(cond, u)
    torch.cuda.synchronize()
    monkeypatch.setenv("WN_SPIN_LIMIT", "1")
    bad = wn.WaveNet(w, dil, weight_dtype="bf16")
    ws = bad.new_workspace(B)
    bad.generate(cond, u, workspace=ws, reset=True)
    torch.cuda.synchronize()
    assert bad.status(ws) == wn.WN_ETIMEOUT
    monkeypatch.delenv("WN_SPIN_LIMIT")
    y = good.generate(cond, u, workspace=ws, reset=True)
    torch.cuda.synchronize()
    assert good.status(ws) == 0
    assert torch.equal(y, y_ref)
    bad.close()
    good.close()


@pytest.mark.parametrize("dtype", ["bf16", "i8"])
def test_default_choice(dtype, monkeypatch):
    """bf16 and int8 models: the fp32 multi-CU kernel (on the exact fp32 copy) while its replicas
    carry at most 2 streams each (l = 20: B <= 30), this kernel beyond that while its replicas carry
    the batch (B <= 512), then the batched kernel (bf16) or the per-stream one (int8)."""
    import paper_1702_07825_amd as wn
    monkeypatch.delenv("WN_KERNEL", raising=False)
    monkeypatch.delenv("WN_MFMA_COLUMNS", raising=False)
    L = 20
    w = synth.make_weights(L, 64, 256, seed=4)
    net = wn.WaveNet(w, synth.dilation_cycle(L), weight_dtype=dtype)
    assert [net.kernel_variant(b) for b in (1, 16, 30)] == ["multi_cu_chain"] * 3
    assert [net.kernel_variant(b) for b in (31, 45, 256, 512)] == [KERNEL] * 4
    assert net.kernel_variant(513) == ("mfma_group" if dtype == "bf16" else "stream_l2")
    net.close()


@pytest.mark.parametrize("B,cols", [(9, 8), (256, 8), (40, 16)])
def test_same_xcd_posts_change_nothing(B, cols, monkeypatch):
    """Posts to a reader on the same XCD stop at its L2; written through instead (WN_LOCAL_POSTS=0)
    every sample and logit is the same, also when every CU of the chip is in the launch (B = 256: 32
    replicas, 4 per XCD) and when the same workspace runs again from zero (every tag repeats, and a
    word a previous call left in an L2 must not be taken for this call's)."""
    import paper_1702_07825_amd as wn
    _log("multi-CU MFMA same-XCD posts: B=%d columns=%d" % (B, cols))
    monkeypatch.setenv("WN_KERNEL", KERNEL)
    monkeypatch.delenv("WN_AUX_LAYERS", raising=False)
    if cols == 16:
        monkeypatch.setenv("WN_MFMA_COLUMNS", "16")
    else:
        monkeypatch.delenv("WN_MFMA_COLUMNS", raising=False)
    L, T = 20, 120
    w = synth.make_weights(L, 64, 256, seed=B + cols, bias_scale=0.1)
    cond = synth.make_cond(L, 64, B, T, seed=B + cols, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=B + cols), device="cuda")
    out = {}
    for lp in ("0", "1"):
        monkeypatch.setenv("WN_LOCAL_POSTS", lp)
        net = wn.WaveNet(w, synth.dilation_cycle(L), weight_dtype="bf16")
        assert net.kernel_variant(B) == KERNEL
        ws = net.new_workspace(B)
        y = net.generate(cond, u, workspace=ws)
        y_again = net.generate(cond, u, workspace=ws, reset=True)
        lg = net.teacher_force(cond, y)
        torch.cuda.synchronize()
        assert net.status(ws) == 0
        assert torch.equal(y, y_again)
        out[lp] = (y.cpu(), lg.cpu())
        net.close()
    assert torch.equal(out["0"][0], out["1"][0])
    assert torch.equal(out["0"][1], out["1"][1])
