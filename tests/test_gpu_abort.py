"""Host-requested abort (wn_abort) on every kernel family, through the C ABI.

A request that stands when a call starts stops it at its first step; a request made while a call
runs stops it within 64 steps.  Either way every workgroup leaves normally (the call returns and
the stream synchronises), wn_status reports WN_EABORTED, the outputs of the steps not taken are
not written, and after the request is withdrawn a call from zero on the same workspace gives the
same samples as an undisturbed run.  The chain kernel stops through its status word, which every
waiting role reads; the per-stream and batched kernels decide per workgroup.
"""
import time

import pytest

import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = [
    # name, L, r, s, B, weight dtype, expected kernel, T (short), T (long, for the mid-run abort)
    ("stream_tiny", 4, 16, 32, 2, "f32", "stream_l2", 200, 200000),
    ("chain_l20_r64_b1", 20, 64, 256, 1, "f32", "multi_cu_chain", 200, 16000),
    ("chain_l20_r64_b3", 20, 64, 256, 3, "f32", "multi_cu_chain", 200, 16000),
    ("group_l20_bf16_b24", 20, 64, 256, 24, "bf16", "mfma_group", 200, 16000),
    ("mfma_chain_l20_bf16_b9", 20, 64, 256, 9, "bf16", "multi_cu_mfma", 200, 16000),
]


def _setup(L, r, s, B, T, dtype, seed):
    import paper_1702_07825_amd as wn
    dil = synth.dilation_cycle(L) if L > 4 else [1, 2, 4, 8][:L]
    w = synth.make_weights(L, r, s, seed=seed, bias_scale=0.1)
    net = wn.WaveNet(w, dil, weight_dtype=dtype)
    cond = synth.make_cond(L, r, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    return net, cond, u


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_standing_request_stops_at_first_step(case, monkeypatch):
    import paper_1702_07825_amd as wn
    name, L, r, s, B, dt, kern, T, _ = case
    monkeypatch.setenv("WN_KERNEL", kern)
    print("abort case %s (standing request): L=%d r=%d B=%d T=%d" % (name, L, r, B, T), flush=True)
    net, cond, u = _setup(L, r, s, B, T, dt, seed=5)
    assert net.kernel_variant(B) == kern
    ws = net.new_workspace(B)
    ref = net.generate(cond, u, workspace=ws)
    assert net.status(ws) == wn.WN_OK
    net.abort(True)
    y = torch.full((B, T), -1, dtype=torch.int32, device="cuda")
    net.generate(cond, u, samples=y, workspace=ws)
    assert net.status(ws) == wn.WN_EABORTED
    assert bool((y == -1).all())  # no step was taken
    net.teacher_force(cond, ref, workspace=ws)
    assert net.status(ws) == wn.WN_EABORTED
    net.abort(False)
    y2 = net.generate(cond, u, workspace=ws, reset=True)
    assert net.status(ws) == wn.WN_OK
    assert torch.equal(y2, ref)
    net.close()


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_request_during_a_call_stops_it(case, monkeypatch):
    import paper_1702_07825_amd as wn
    name, L, r, s, B, dt, kern, T, TL = case
    monkeypatch.setenv("WN_KERNEL", kern)
    print("abort case %s (request while running): L=%d r=%d B=%d T=%d" % (name, L, r, B, TL), flush=True)
    net, cond, u = _setup(L, r, s, B, TL, dt, seed=6)
    ws = net.new_workspace(B)
    # an undisturbed run of the first T steps, and the duration of a whole call
    ref = net.generate(cond[:, :T].contiguous(), u[:, :T].contiguous(), workspace=ws)
    t0 = time.perf_counter()
    net.generate(cond, u, workspace=ws)
    assert net.status(ws) == wn.WN_OK
    full = time.perf_counter() - t0
    print("  a whole call takes %.1f ms" % (1e3 * full), flush=True)
    assert full > 0.1
    y = torch.full((B, TL), -1, dtype=torch.int32, device="cuda")
    t0 = time.perf_counter()
    net.generate(cond, u, samples=y, workspace=ws, reset=True)
    time.sleep(0.2 * full)
    net.abort(True)
    st = net.status(ws)
    took = time.perf_counter() - t0
    net.abort(False)
    print("  aborted call returned %d after %.1f ms" % (st, 1e3 * took), flush=True)
    assert st == wn.WN_EABORTED
    assert bool((y[:, -1] == -1).all())  # the last steps were not taken
    assert took < 0.8 * full
    y2 = net.generate(cond[:, :T].contiguous(), u[:, :T].contiguous(), workspace=ws, reset=True)
    assert net.status(ws) == wn.WN_OK
    assert torch.equal(y2, ref)
    net.close()
