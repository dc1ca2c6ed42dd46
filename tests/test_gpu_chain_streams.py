"""GPU parity of the multi-CU kernel serving several streams (fp32 weights).

Replicas of the chain / head / aux roles run side by side and each interleaves
its streams step by step; these cases cover several streams per replica, an
uneven last replica, more steps than the kernel stages per stream, r = 128 with
one layer per chain CU, and a single chain CU whose last-layer skip projection
goes through the aux CU.  Bars as in test_gpu_parity: teacher-forced logits
within 1e-3 of the oracle, indices bit-exact at every step whose oracle CDF
margin exceeds 1e-4 (the oracle replays the GPU's own samples).
"""
import zlib

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

MARGIN = 1e-4


def _setup(L, r, s, dil, B, T, seed, bias=0.0):
    import paper_1702_07825_amd as wn
    w = synth.make_weights(L, r, s, seed=seed, bias_scale=bias)
    net = wn.WaveNet(w, dil)
    cond = synth.make_cond(L, r, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    return w, net, cond, u, oracle.Model(w, dil)


CASES = [
    # name, L, r, s, dilations, B, T, bias
    # (replicas x streams per replica; a replica is nch chain + 4 head + ceil(L / 2) aux CUs: two
    # layers per aux CU, at r = 128 with the first layer's W_skip in LDS)
    ("l20_r128_b11", 20, 128, 256, tuple(synth.dilation_cycle(20)), 11, 300, 0.2),  # 6 x 2 (last 1), 25 CUs each
    ("l20_r64_b12", 20, 64, 256, tuple(synth.dilation_cycle(20)), 12, 300, 0.0),    # 12 x 1, 17 CUs each
    # more streams per replica than two-layer aux CUs can stage at r = 128: one layer per aux CU
    ("l20_r128_b80", 20, 128, 256, tuple(synth.dilation_cycle(20)), 80, 60, 0.1),   # 7 x 12 (last 8), 35 CUs each
    ("l3_r128_b5", 3, 128, 256, (1, 3, 2), 5, 200, 0.3),                             # 5 x 1, 9 CUs each
    ("l1_r128_b2", 1, 128, 256, (1,), 2, 150, 0.4),                                  # one chain CU, skip on aux
    ("l5_r128_b3", 5, 128, 256, (2, 1, 4, 1, 3), 3, 200, 0.3),                      # chain CUs of 1, 2, 1, 1 layers
    ("l9_r32_b40", 9, 32, 128, (1, 2, 4, 8, 16, 32, 64, 128, 256), 40, 200, 0.2),    # 20 x 2, 10 CUs each
    # the largest batch one launch serves at l = 20, r = 64: 15 replicas of 17 CUs, 16 streams each
    ("l20_r64_b240", 20, 64, 256, tuple(synth.dilation_cycle(20)), 240, 40, 0.1),
    # the most layers the library takes: 10 chain CUs of up to 7 layers, 32 aux CUs
    ("l64_r64_b1", 64, 64, 256, tuple(synth.dilation_cycle(64)), 1, 120, 0.1),
    # one stream with chain CUs of 5 and 4 layers: the one-stream build whose layer counts are read at
    # run time (7- and 6-layer chain CUs get builds with the count fixed)
    ("l9_r64_b1", 9, 64, 256, (1, 2, 4, 8, 16, 32, 64, 128, 256), 1, 300, 0.2),       # 1 x 1, 11 CUs
    # two d = 1 layers on one aux CU (both history reads wait for the chain CU's step), an odd layer
    # count whose last aux CU holds only the last layer (its skip projection is on the chain)
    ("l7_r64_d1s_b2", 7, 64, 256, (1, 1, 2, 1, 1, 4, 1), 2, 200, 0.3),               # 2 x 1, 10 CUs each
]


# (workgroups, replicas) wn_launch_info reports for the layouts stated above
LAUNCH = {"l20_r128_b11": (150, 6), "l20_r128_b80": (245, 7), "l20_r64_b12": (204, 12), "l3_r128_b5": (45, 5), "l1_r128_b2": (12, 2),
          "l5_r128_b3": (33, 3), "l9_r32_b40": (200, 20), "l20_r64_b240": (255, 15), "l64_r64_b1": (46, 1), "l9_r64_b1": (11, 1),
          "l7_r64_d1s_b2": (18, 2)}


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_multi_stream_chain_parity(case, monkeypatch):
    name, L, r, s, dil, B, T, bias = case
    # the multi-CU kernel by name: by default fp32 batches of more than 13 streams per replica at
    # r <= 64 go to the per-stream kernel
    monkeypatch.setenv("WN_KERNEL", "multi_cu_chain")
    print("case %s: L=%d r=%d s=%d B=%d T=%d" % (name, L, r, s, B, T), flush=True)
    w, net, cond, u, model = _setup(L, r, s, dil, B, T, seed=zlib.crc32(name.encode()) % 1000, bias=bias)
    assert net.kernel_variant(B) == "multi_cu_chain"
    wgs, reps = net.launch_info(B)
    assert 1 <= reps <= wgs <= 256 and -(-B // reps) <= 16
    assert (wgs, reps) == LAUNCH[name]
    ws = net.new_workspace(B)
    y = net.generate(cond, u, workspace=ws)
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    assert net.status(ws) == 0
    y_np, lg_np = y.cpu().numpy(), lg.cpu().numpy()
    assert y_np.min() >= 0 and y_np.max() <= 255
    ys, lo, mg = oracle.run_streams(model, cond.cpu().numpy(), u=u.cpu().numpy(), y_in=y_np, threads=8)
    err = float(np.abs(lg_np - lo).max())
    ok = mg > MARGIN
    mism = int(np.sum(ys[ok] != y_np[ok]))
    print("  max|dlogit|=%.3g confident=%d/%d mismatches=%d" % (err, int(ok.sum()), ok.size, mism), flush=True)
    assert err <= 1e-3
    assert mism == 0
    net.close()


def test_multi_stream_chain_state_and_placement():
    """Chunked calls continue exactly; results do not depend on which replica or slot serves a stream."""
    L, r, s, B, T = 20, 128, 256, 11, 260
    dil = tuple(synth.dilation_cycle(L))
    w, net, cond, u, _ = _setup(L, r, s, dil, B, T, seed=21, bias=0.1)
    y = net.generate(cond, u)
    y2 = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    ws = net.new_workspace(B)
    parts, a = [], 0
    for b_ in (1, 2, 129, 130, T):
        parts.append(net.generate(cond[:, a:b_].contiguous(), u[:, a:b_].contiguous(), workspace=ws, reset=(a == 0)))
        a = b_
    ws2 = net.new_workspace(B)
    lgp = [net.teacher_force(cond[:, :77].contiguous(), y[:, :77].contiguous(), workspace=ws2, reset=True),
           net.teacher_force(cond[:, 77:].contiguous(), y[:, 77:].contiguous(), workspace=ws2, reset=False)]
    perm = torch.tensor([10, 3, 7, 0, 9, 1, 5, 8, 2, 6, 4], device="cuda")
    yp = net.generate(cond[perm].contiguous(), u[perm].contiguous())
    # fewer streams: a different plan (one stream per replica) for the same first streams
    y5 = net.generate(cond[:5].contiguous(), u[:5].contiguous())
    torch.cuda.synchronize()
    assert net.status(ws) == 0 and net.status(ws2) == 0
    assert torch.equal(y, y2)
    assert torch.equal(torch.cat(parts, 1), y)
    assert torch.equal(torch.cat(lgp, 1), lg)
    assert torch.equal(yp, y[perm])
    assert torch.equal(y5, y[:5])
    net.close()


def test_multi_stream_chain_matches_per_stream_kernel(monkeypatch):
    L, r, s, B, T = 20, 128, 256, 7, 120
    dil = tuple(synth.dilation_cycle(L))
    w, net, cond, u, _ = _setup(L, r, s, dil, B, T, seed=22, bias=0.2)
    y = net.generate(cond, u)
    lg = net.teacher_force(cond, y)
    monkeypatch.setenv("WN_KERNEL", "stream")
    import paper_1702_07825_amd as wn
    ref = wn.WaveNet(w, dil)
    assert ref.kernel_variant(B) == "stream_l2"
    lg_ref = ref.teacher_force(cond, y)
    torch.cuda.synchronize()
    d = float((lg_ref - lg).abs().max())
    print("  max|dlogit| chain vs per-stream kernel %.3g" % d, flush=True)
    assert d <= 1e-4
    ref.close()
    net.close()


@pytest.mark.parametrize("B", [1, 2])
def test_timeout_path_drains_and_recovers(B, monkeypatch):
    """Every wait of the multi-CU kernel is bounded.  With the host's spin limit forced to one
    poll, a launch must end with WN_ETIMEOUT in the status word (every block leaves, so the call
    returns), and the next call that starts from zero on the same workspace must run cleanly.
    B = 1 runs the one-stream build (fixed layer counts), B = 2 the multi-stream one."""
    import paper_1702_07825_amd as wn
    L, r, s, dil, T = 20, 64, 256, tuple(synth.dilation_cycle(20)), 50
    w, net, cond, u, model = _setup(L, r, s, dil, B, T, seed=77, bias=0.1)
    assert net.kernel_variant(B) == "multi_cu_chain"
    ws = net.new_workspace(B)
    monkeypatch.setenv("WN_SPIN_LIMIT", "1")
    print("forced timeout run, B=%d" % B, flush=True)
    net.generate(cond, u, workspace=ws)
    assert net.status(ws) == wn.WN_ETIMEOUT
    monkeypatch.delenv("WN_SPIN_LIMIT")
    y = net.generate(cond, u, workspace=ws, reset=True)
    assert net.status(ws) == 0
    lg = net.teacher_force(cond, y)
    torch.cuda.synchronize()
    ys, lo, mg = oracle.run_streams(model, cond.cpu().numpy(), u=u.cpu().numpy(), y_in=y.cpu().numpy(), threads=8)
    assert float(np.abs(lg.cpu().numpy() - lo).max()) <= 1e-3
    ok = mg > MARGIN
    assert np.array_equal(ys[ok], y.cpu().numpy()[ok])
    net.close()


@pytest.mark.parametrize("L,r,B", [(20, 64, 1), (20, 128, 11), (40, 64, 2), (64, 64, 1)])
def test_same_xcd_posts_change_nothing(L, r, B, monkeypatch):
    """Posts to a reader on the same XCD stop at its L2; written through instead (WN_LOCAL_POSTS=0)
    every sample and logit is the same.  l = 20 and l = 40 at r = 64 place a replica on one XCD
    (17 and 30 CUs: all posts local); r = 128 and l = 64 spill aux CUs to other XCDs (local and
    written-through posts mix)."""
    import paper_1702_07825_amd as wn
    print("same-XCD posts: L=%d r=%d B=%d" % (L, r, B), flush=True)
    dil = tuple(synth.dilation_cycle(L))
    w = synth.make_weights(L, r, 256, seed=L + r + B, bias_scale=0.1)
    T = 200
    cond = synth.make_cond(L, r, B, T, seed=L + r + B, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=L + r + B), device="cuda")
    out = {}
    for lp in ("0", "1"):
        monkeypatch.setenv("WN_LOCAL_POSTS", lp)
        net = wn.WaveNet(w, dil)
        assert net.kernel_variant(B) == "multi_cu_chain"
        ws = net.new_workspace(B)
        y = net.generate(cond, u, workspace=ws)
        # the same workspace from zero again: every tag repeats, and words left in an XCD's L2 by
        # the previous call must not be taken for this call's
        y_again = net.generate(cond, u, workspace=ws, reset=True)
        lg = net.teacher_force(cond, y)
        torch.cuda.synchronize()
        assert net.status(ws) == 0
        assert torch.equal(y, y_again)
        out[lp] = (y.cpu(), lg.cpu())
        net.close()
    assert torch.equal(out["0"][0], out["1"][0])
    assert torch.equal(out["0"][1], out["1"][1])


@pytest.mark.parametrize("L,r,B,dil", [(20, 64, 1, None), (40, 64, 2, None), (9, 64, 3, (1, 1, 2, 1, 8, 1, 3, 1, 2)),
                                        (20, 128, 3, None), (5, 128, 2, (1, 2, 1, 4, 1))])
def test_one_and_two_layers_per_aux_cu_agree(L, r, B, dil, monkeypatch):
    """Aux CUs holding two layers each (the default) or one (WN_AUX_LAYERS=1; at r = 128 every aux
    CU then reads its layer's W_skip from LDS): the same model gives the same logits up to the order
    of the skip sums, and each layout's samples match the oracle at every confident step."""
    s, T = 256, 300
    dil = tuple(synth.dilation_cycle(L)) if dil is None else dil
    print("aux layouts L=%d r=%d B=%d" % (L, r, B), flush=True)
    w, net, cond, u, model = _setup(L, r, s, dil, B, T, seed=31 + L, bias=0.2)
    ys, lgs = [], []
    for nla in ("2", "1"):
        monkeypatch.setenv("WN_AUX_LAYERS", nla)
        y = net.generate(cond, u)
        ys.append(y)
        lgs.append(net.teacher_force(cond, ys[0]))
    torch.cuda.synchronize()
    d = float((lgs[0] - lgs[1]).abs().max())
    print("  max|dlogit| between the layouts %.3g" % d, flush=True)
    assert d <= 1e-4
    for y in ys:
        y_np = y.cpu().numpy()
        yo, lo, mg = oracle.run_streams(model, cond.cpu().numpy(), u=u.cpu().numpy(), y_in=y_np, threads=8)
        ok = mg > MARGIN
        assert np.array_equal(yo[ok], y_np[ok])
    net.close()
