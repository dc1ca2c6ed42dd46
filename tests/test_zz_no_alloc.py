"""The conditioning network's entry point that allocates nothing (wn_condition_static,
include/wn_cond.h) against the one that takes a workspace (wn_condition), through the C ABI.

Both run the same kernels on the same inputs, so their outputs must be identical, element for
element.  Two calls in a row on one handle (the second with fewer streams and frames, so it
reuses a scratch array that still holds the first call's larger contents), a call at the paper's
sizes, and a size beyond the static array's maximum, which is refused before anything runs.
"""
import numpy as np
import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _run_pair(net, x, T):
    B, L, r = x.shape[0], net.n_layers, net.r
    ref = net(x, T)
    out = torch.full((B, T, L, 2 * r), float("nan"), dtype=torch.float32, device="cuda")
    net.condition_static(x, T, out)
    torch.cuda.synchronize()
    return ref, out


def test_static_scratch_matches_workspace_twice():
    import paper_1702_07825_amd as wn
    print("no-alloc: F=227 h1=48 l=3 r=12, two calls (B=3, 77 frames; then B=1, 31 frames)", flush=True)
    w = synth.make_cond_weights(227, 48, 3 * 12, seed=11, bias_scale=0.2)
    net = wn.Conditioner(w, 3, 12, 256, 16000)
    x1 = torch.tensor(synth.make_features(3, 77, seed=5), device="cuda")
    ref1, out1 = _run_pair(net, x1, 4801)
    assert torch.equal(ref1, out1)
    x2 = torch.tensor(synth.make_features(1, 31, seed=6), device="cuda")
    ref2, out2 = _run_pair(net, x2, 31 * 16000 // 256)
    assert torch.equal(ref2, out2)
    # the first call's result is not disturbed by the second call's use of the scratch
    assert torch.equal(ref1, out1)
    net.close()


def test_static_scratch_paper_sizes():
    import paper_1702_07825_amd as wn
    print("no-alloc: paper sizes, F=227 h1=256 l=20 r=64, one 1 s utterance (256 frames)", flush=True)
    w = synth.make_cond_weights(synth.N_FEATURES, 256, 20 * 64, seed=12, bias_scale=0.1)
    net = wn.Conditioner(w, 20, 64, 256, 16000)
    assert net.workspace_bytes(1, 256) <= wn.COND_SCRATCH_BYTES
    x = torch.tensor(synth.make_features(1, 256, seed=7), device="cuda")
    ref, out = _run_pair(net, x, 16000)
    assert torch.equal(ref, out)
    net.close()


def test_static_scratch_rejects_beyond_its_size():
    import paper_1702_07825_amd as wn
    print("no-alloc: a call needing more than the static scratch is refused", flush=True)
    w = synth.make_cond_weights(227, 256, 20 * 64, seed=13, bias_scale=0.1)
    net = wn.Conditioner(w, 20, 64, 256, 16000)
    B, Tf = 8, 256
    assert net.workspace_bytes(B, Tf) > wn.COND_SCRATCH_BYTES
    x = torch.zeros((B, Tf, 227), dtype=torch.float32, device="cuda")
    out = torch.zeros((B, 16, 20, 128), dtype=torch.float32, device="cuda")
    with pytest.raises(wn.WnError) as ei:
        net.condition_static(x, 16, out)
    assert ei.value.code == wn.WN_EINVAL
    torch.cuda.synchronize()
    assert not bool(out.abs().sum().item())  # nothing ran
    net.close()
