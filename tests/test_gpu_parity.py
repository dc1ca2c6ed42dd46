"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Bars: teacher-forced logits within max-abs 1e-3 (fp32 weights; bf16 weights are
compared with the oracle's bf16 mode at 1e-3 and with the fp32 oracle at 2e-2);
sample indices bit-exact at every step whose oracle CDF margin exceeds 1e-4,
judged on the GPU's own sample sequence (the oracle replays it teacher-forced).
"""
import os
import zlib
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

LOGIT_TOL = {"f32": 1e-3, "bf16": 1e-3, "i8": 1e-3}
BF16_VS_F32_TOL = 2e-2
MARGIN = 1e-4


def _wn():
    import paper_1702_07825_amd as wn
    return wn


def _setup(L, r, s, dil, B, T, seed, dtype="f32", bias=0.0, init=128):
    wn = _wn()
    w = synth.make_weights(L, r, s, seed=seed, bias_scale=bias)
    net = wn.WaveNet(w, dil, initial_sample=init, weight_dtype=dtype)
    cond = synth.make_cond(L, r, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    model = oracle.Model(w, dil, initial_sample=init, bf16_weights=(dtype == "bf16"), int8_weights=(dtype == "i8"))
    return w, net, cond, u, model


def _log(msg):
    print(msg, flush=True)


SMALL = [
    # name, L, r, s, dil, B, T, dtype, bias
    ("tiny", 4, 16, 32, (1, 2, 4, 8), 1, 1600, "f32", 0.0),
    ("tiny_bias", 4, 16, 32, (1, 2, 4, 8), 3, 333, "f32", 0.4),
    ("odd_dilations", 3, 16, 32, (3, 1, 7), 2, 257, "f32", 0.3),
    ("l20_r64", 20, 64, 256, tuple(synth.dilation_cycle(20)), 1, 300, "f32", 0.0),
    ("l40_r64", 40, 64, 256, tuple(synth.dilation_cycle(40)), 1, 150, "f32", 0.1),
    ("l20_r128_b3", 20, 128, 256, tuple(synth.dilation_cycle(20)), 3, 120, "f32", 0.0),
    ("l20_r64_bf16_b5", 20, 64, 256, tuple(synth.dilation_cycle(20)), 5, 140, "bf16", 0.0),
    ("r32_s128", 6, 32, 128, (1, 2, 4, 8, 16, 32), 2, 200, "f32", 0.2),
    ("r64_s128", 5, 64, 128, (1, 3, 9, 2, 4), 2, 200, "f32", 0.2),
    ("one_layer", 1, 16, 32, (1,), 1, 50, "f32", 0.5),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[0] for c in SMALL])
def test_logits_and_indices(case):
    name, L, r, s, dil, B, T, dtype, bias = case
    _log("case %s: L=%d r=%d s=%d B=%d T=%d %s" % (name, L, r, s, B, T, dtype))
    w, net, cond, u, model = _setup(L, r, s, dil, B, T, seed=zlib.crc32(name.encode()) % 1000, dtype=dtype, bias=bias)
    y = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    y_np, lg_np = y.cpu().numpy(), lg.cpu().numpy()
    cond_np, u_np = cond.cpu().numpy(), u.cpu().numpy()
    assert y_np.min() >= 0 and y_np.max() <= 255
    ys, lo, mg = oracle.run_streams(model, cond_np, u=u_np, y_in=y_np, threads=8)
    err = np.abs(lg_np - lo).max()
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[ok]))
    _log("  max|dlogit|=%.3g low-margin steps=%d/%d mismatches=%d (low-margin disagreements %d)" %
         (err, int((~ok).sum()), ok.size, mism, int(np.sum(ys[~ok] != y_np[~ok]))))
    assert err <= LOGIT_TOL[dtype]
    assert mism == 0
    if dtype == "bf16":
        m32 = oracle.Model(w, dil)
        _, lo32, _ = oracle.run_streams(m32, cond_np, y_in=y_np, threads=8)
        assert np.abs(lg_np - lo32).max() <= BF16_VS_F32_TOL
    # free-running agreement up to the first low-margin step of the oracle's own run
    for b in range(B):
        yo, _, mo = oracle.run(model, cond_np[b], u=u_np[b], want_logits=False)
        first_low = int(np.argmax(mo <= MARGIN)) if np.any(mo <= MARGIN) else T
        np.testing.assert_array_equal(y_np[b, :first_low], yo[:first_low])
    net.close()


def test_chunked_equals_one_shot_and_determinism():
    L, r, s, dil, B, T = 4, 16, 32, (1, 2, 4, 8), 3, 500
    w, net, cond, u, model = _setup(L, r, s, dil, B, T, seed=11, bias=0.3)
    y1 = net.generate(cond, u)
    y2 = net.generate(cond, u)
    ws = net.new_workspace(B)
    parts, a = [], 0
    for b_ in (1, 2, 64, 65, 300, 500):
        parts.append(net.generate(cond[:, a:b_].contiguous(), u[:, a:b_].contiguous(), workspace=ws, reset=(a == 0)))
        a = b_
    lg1 = net.teacher_force(cond, y1)
    ws2 = net.new_workspace(B)
    lg_parts = [net.teacher_force(cond[:, :137].contiguous(), y1[:, :137].contiguous(), workspace=ws2, reset=True),
                net.teacher_force(cond[:, 137:].contiguous(), y1[:, 137:].contiguous(), workspace=ws2, reset=False)]
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    assert torch.equal(torch.cat(parts, dim=1), y1)
    assert torch.equal(torch.cat(lg_parts, dim=1), lg1)
    assert net.status(ws) == 0
    net.close()


def test_stream_permutation():
    L, r, s, dil, B, T = 20, 64, 256, tuple(synth.dilation_cycle(20)), 4, 100
    w, net, cond, u, model = _setup(L, r, s, dil, B, T, seed=12)
    y = net.generate(cond, u)
    perm = torch.tensor([2, 0, 3, 1], device="cuda")
    yp = net.generate(cond[perm].contiguous(), u[perm].contiguous())
    torch.cuda.synchronize()
    assert torch.equal(yp, y[perm])
    net.close()


def test_edge_cases():
    wn = _wn()
    L, r, s, dil = 4, 16, 32, (1, 2, 4, 8)
    w, net, cond, u, model = _setup(L, r, s, dil, 2, 1, seed=13, bias=0.2)
    # T = 1
    y = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    ys, lo, mg = oracle.run_streams(model, cond.cpu().numpy(), u=u.cpu().numpy(), y_in=y.cpu().numpy())
    assert np.abs(lg.cpu().numpy() - lo).max() <= 1e-3
    # T = 0 is a no-op that still validates the handle
    empty = torch.empty((2, 0, L, 2 * r), device="cuda")
    out = net.generate(empty, torch.empty((2, 0), device="cuda"))
    assert out.shape == (2, 0)
    # short workspace and bad shapes are rejected before any launch
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(wn.WnError) as e:
        net.generate(cond, u, workspace=small)
    assert e.value.code == wn.WN_EINVAL
    with pytest.raises(ValueError):
        net.generate(cond, u[:, :0])
    net.close()


def test_initial_sample_and_bias_paths():
    """Non-default y_{-1} and nonzero biases everywhere."""
    L, r, s, dil, B, T = 3, 64, 256, (1, 2, 4), 2, 64
    w, net, cond, u, model = _setup(L, r, s, dil, B, T, seed=14, bias=0.8, init=3)
    y = torch.tensor(synth.make_samples(B, T, seed=14), device="cuda")
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    _, lo, _ = oracle.run_streams(model, cond.cpu().numpy(), y_in=y.cpu().numpy())
    assert np.abs(lg.cpu().numpy() - lo).max() <= 1e-3
    net.close()


# ---------------------------------------------------------------------------------------------
# Full-size workloads, in the launch configuration the benchmark times.  The oracle checks
# sampled steps: the logits of step t depend only on the last R = 1 + sum(d) inputs, so a
# teacher-forced oracle run over the window [t - sum(d), t] reproduces them exactly.
# ---------------------------------------------------------------------------------------------

def _window(w, dil, dtype, cond_b, u_b, y_b, t):
    """Oracle logits, draw and margin of step t from a teacher-forced run over
    [t - (taps - 1) - sum(d), t], the window step t depends on (taps = embedding taps)."""
    taps = 1 if np.asarray(w["embed"]).ndim == 2 else 2
    t0 = max(0, t - (taps - 1) - int(sum(dil)))
    init = 128 if t0 == 0 else int(y_b[t0 - 1])
    m = oracle.Model(w, dil, initial_sample=init, bf16_weights=(dtype == "bf16"), int8_weights=(dtype == "i8"))
    ys, lo, mg = oracle.run(m, cond_b[t0:t + 1], u=u_b[t0:t + 1], y_in=y_b[t0:t + 1])
    return lo[-1], int(ys[-1]), float(mg[-1])


FULL = ["l20_r64_b1", "l40_r64_b1", "tiny", "l20_r128_b32", "l20_r64_b256_bf16", "l20_r64_b1_2tap_48k",
        "l20_r64_b1_i8", "l20_r64_b256_i8"]


def _whole_stream(w, dil, dtype, cb, ub, yb):
    """The oracle teacher-forced over a whole stream: logits, draws and margins of every step."""
    m = oracle.Model(w, dil, bf16_weights=(dtype == "bf16"), int8_weights=(dtype == "i8"))
    return oracle.run(m, cb, u=ub, y_in=yb)


@pytest.mark.parametrize("name", FULL)
def test_full_size_sampled(name):
    """At the benchmark's full sizes, in the launch the benchmark times: every step of stream 0
    (the oracle replays the GPU's whole sample sequence, teacher-forced, past every wrap of the
    d = 512 histories), plus sampled steps of the last and the middle stream of a batch (each
    checked on a window of sum(d) + 1 steps, the receptive field)."""
    wl = synth.WORKLOADS[name]
    _log("full-size %s: %s" % (name, wl.description))
    w = synth.make_weights(wl.n_layers, wl.r, wl.s, seed=0, embed_taps=wl.embed_taps)
    wn = _wn()
    net = wn.WaveNet(w, wl.dilations, weight_dtype=wl.weight_dtype)
    cond = synth.make_cond(wl.n_layers, wl.r, wl.B, wl.T, seed=0, device="cuda")
    u = torch.tensor(synth.make_uniforms(wl.B, wl.T, seed=0), device="cuda")
    y = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    y_np = y.cpu().numpy()
    assert y_np.min() >= 0 and y_np.max() <= 255
    rng = np.random.default_rng(0)
    jobs = []
    for b in sorted(set([wl.B - 1, wl.B // 2]) - {0}):
        steps = sorted(set([wl.T - 1] + [int(x) for x in rng.integers(0, wl.T, 1)]))
        cb, ub = cond[b].cpu().numpy(), u[b].cpu().numpy()
        for t in steps:
            jobs.append((b, t, cb, ub, lg[b, t].cpu().numpy()))
    c0, u0, lg0 = cond[0].cpu().numpy(), u[0].cpu().numpy(), lg[0].cpu().numpy()
    with ThreadPoolExecutor(max_workers=8) as ex:
        whole = ex.submit(_whole_stream, w, wl.dilations, wl.weight_dtype, c0, u0, y_np[0])
        res = list(ex.map(lambda j: _window(w, wl.dilations, wl.weight_dtype, j[2], j[3], y_np[j[0]], j[1]), jobs))
        ys0, lo0, mg0 = whole.result()
    worst0 = float(np.abs(lo0 - lg0).max())
    ok0 = mg0 > MARGIN
    mism0 = int(np.sum(ys0[ok0] != y_np[0][ok0]))
    _log("  stream 0, all %d steps: max|dlogit|=%.3g confident=%d mismatches=%d" %
         (wl.T, worst0, int(ok0.sum()), mism0))
    worst, checked, mism = 0.0, 0, 0
    for (b, t, _, _, lg_bt), (lo, yo, mg) in zip(jobs, res):
        worst = max(worst, float(np.abs(lo - lg_bt).max()))
        if mg > MARGIN:
            checked += 1
            mism += int(yo != y_np[b, t])
    _log("  %d sampled (stream, step) pairs of other streams: max|dlogit|=%.3g confident=%d mismatches=%d" %
         (len(jobs), worst, checked, mism))
    assert worst0 <= LOGIT_TOL[wl.weight_dtype] and mism0 == 0
    assert worst <= LOGIT_TOL[wl.weight_dtype]
    assert mism == 0
    net.close()


WRAP = [
    # name, r, s, B, dtype, expected kernel
    ("chain_b1", 64, 256, 1, "f32", "multi_cu_chain"),
    ("chain_b3", 64, 256, 3, "f32", "multi_cu_chain"),
    ("chain_r128_b2", 128, 256, 2, "f32", "multi_cu_chain"),
    ("group_b9", 64, 256, 9, "bf16", "mfma_group"),
    ("mfma_chain_b9", 64, 256, 9, "bf16", "multi_cu_mfma"),
    ("mfma_chain_i8_b64", 64, 256, 64, "i8", "multi_cu_mfma"),
]


@pytest.mark.parametrize("case", WRAP, ids=[c[0] for c in WRAP])
def test_chunks_across_history_wraps(case, monkeypatch):
    """l = 20 with dilations up to 512 over 1100 steps, in chunks whose boundaries straddle steps
    512 and 1024 (where the d = 512 histories wrap): chunked generation and teacher forcing equal
    the one-shot call bit for bit, and the one-shot call matches the oracle on every step."""
    name, r, s, B, dtype, kern = case
    monkeypatch.setenv("WN_KERNEL", kern)
    L, T = 20, 1100
    dil = tuple(synth.dilation_cycle(L))
    _log("wrap case %s: L=%d r=%d B=%d T=%d" % (name, L, r, B, T))
    w, net, cond, u, model = _setup(L, r, s, dil, B, T, seed=zlib.crc32(name.encode()) % 1000, dtype=dtype, bias=0.2)
    assert net.kernel_variant(B) == kern
    y = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    ws = net.new_workspace(B)
    ws2 = net.new_workspace(B)
    parts, lparts, a = [], [], 0
    for b_ in (1, 511, 513, 1023, 1025, T):
        parts.append(net.generate(cond[:, a:b_].contiguous(), u[:, a:b_].contiguous(), workspace=ws, reset=(a == 0)))
        lparts.append(net.teacher_force(cond[:, a:b_].contiguous(), y[:, a:b_].contiguous(), workspace=ws2,
                                        reset=(a == 0)))
        a = b_
    torch.cuda.synchronize()
    assert net.status(ws) == 0 and net.status(ws2) == 0
    assert torch.equal(torch.cat(parts, 1), y)
    assert torch.equal(torch.cat(lparts, 1), lg)
    y_np = y.cpu().numpy()
    ys, lo, mg = oracle.run_streams(model, cond.cpu().numpy(), u=u.cpu().numpy(), y_in=y_np, threads=8)
    err = float(np.abs(lg.cpu().numpy() - lo).max())
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[ok]))
    _log("  max|dlogit|=%.3g confident=%d/%d mismatches=%d" % (err, int(ok.sum()), ok.size, mism))
    assert err <= LOGIT_TOL[dtype] and mism == 0
    net.close()


# ---------------------------------------------------------------------------------------------
# The multi-CU kernel that serves single-stream fp32 models (l=20/40, r=64, s=256).
# ---------------------------------------------------------------------------------------------

def _force_stream(monkeypatch):
    monkeypatch.setenv("WN_KERNEL", "stream")


def test_multi_cu_kernel_is_used_for_one_stream():
    wn = _wn()
    w = synth.make_weights(20, 64, 256, seed=1)
    net = wn.WaveNet(w, synth.dilation_cycle(20))
    # up to 15 replicas of 17 CUs (two layers per aux CU); by default at most 13 streams each (the
    # per-stream kernel is faster beyond), up to 16 when forced
    assert [net.kernel_variant(b) for b in (1, 2, 195)] == ["multi_cu_chain"] * 3
    assert [net.kernel_variant(b) for b in (196, 240, 241)] == ["stream_l2"] * 3
    net.close()
    os.environ["WN_KERNEL"] = "multi_cu_chain"
    try:
        forced = wn.WaveNet(w, synth.dilation_cycle(20))
        assert forced.kernel_variant(240) == "multi_cu_chain" and forced.kernel_variant(241) == "stream_l2"
        forced.close()
    finally:
        del os.environ["WN_KERNEL"]


@pytest.mark.parametrize("L,S", [(20, 256), (9, 128), (40, 256), (3, 256), (7, 128)])
def test_multi_cu_kernel_parity_and_state(L, S, monkeypatch):
    """Chain kernel vs oracle (logits, confident indices), chunked == one-shot, run twice == once."""
    r, T = 64, 400
    dil = tuple(synth.dilation_cycle(L))
    _log("multi-CU L=%d r=%d s=%d T=%d" % (L, r, S, T))
    w, net, cond, u, model = _setup(L, r, S, dil, 1, T, seed=L + S, bias=0.3)
    assert net.kernel_variant(1) == "multi_cu_chain"
    y = net.generate(cond, u)
    y2 = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    ws = net.new_workspace(1)
    parts, a = [], 0
    for b_ in (1, 2, 150, 151, T):
        parts.append(net.generate(cond[:, a:b_].contiguous(), u[:, a:b_].contiguous(), workspace=ws, reset=(a == 0)))
        a = b_
    ws2 = net.new_workspace(1)
    lgp = [net.teacher_force(cond[:, :77].contiguous(), y[:, :77].contiguous(), workspace=ws2, reset=True),
           net.teacher_force(cond[:, 77:].contiguous(), y[:, 77:].contiguous(), workspace=ws2, reset=False)]
    torch.cuda.synchronize()
    assert net.status(ws) == 0 and net.status(ws2) == 0
    assert torch.equal(y, y2)
    assert torch.equal(torch.cat(parts, 1), y)
    assert torch.equal(torch.cat(lgp, 1), lg)
    y_np = y.cpu().numpy()
    ys, lo, mg = oracle.run(model, cond.cpu().numpy()[0], u=u.cpu().numpy()[0], y_in=y_np[0])
    err = np.abs(lg.cpu().numpy()[0] - lo).max()
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[0][ok]))
    _log("  max|dlogit|=%.3g confident=%d mismatches=%d" % (err, int(ok.sum()), mism))
    assert err <= 1e-3 and mism == 0
    # the generic kernel agrees on the same inputs
    _force_stream(monkeypatch)
    wn = _wn()
    ref = wn.WaveNet(w, dil, weight_dtype="f32")
    assert ref.kernel_variant(1) == "stream_l2"
    lg_ref = ref.teacher_force(cond, y)
    torch.cuda.synchronize()
    assert float((lg_ref - lg).abs().max()) <= 1e-4
    ref.close()
    net.close()
