"""GPU parity of the sampling rules of the paper's Appendix A.4 ("Sampling from Output
Distribution"): temperature, top k, mode and mean beside direct sampling, through
wn_generate_sampled on each kernel family.

The oracle replays the GPU's own samples (teacher forcing) and takes its own decision at every
step under the same rule; the two must agree wherever the oracle's margin for that rule (distance
of u from the CDF, gap between the k-th and (k+1)-th logits, gap between the two largest logits,
distance of the mean from a half-integer) exceeds MARGIN.  W_out is scaled up so that the
distributions are sharp enough for the rules to differ visibly.
"""
import zlib

import numpy as np
import pytest

import oracle
import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

MARGIN = {0: 1e-4, 1: 1e-4, 2: 1e-4, 3: 1e-4, 4: 1e-3}
SAMPLERS = [(1, 0.7, 256), (1, 1.6, 256), (2, 1.0, 1), (2, 1.0, 5), (2, 1.0, 40), (3, 1.0, 256), (4, 1.0, 256)]
MODELS = [
    # name, L, r, s, dilations, B, T, dtype, expected kernel
    ("tiny_stream", 4, 16, 32, (1, 2, 4, 8), 2, 300, "f32", "stream_l2"),
    ("l20_r64_chain_b1", 20, 64, 256, tuple(synth.dilation_cycle(20)), 1, 200, "f32", "multi_cu_chain"),
    ("l20_r128_chain_b11", 20, 128, 256, tuple(synth.dilation_cycle(20)), 11, 120, "f32", "multi_cu_chain"),
    ("l5_bf16_group_b17", 5, 64, 256, (1, 3, 9, 2, 4), 17, 150, "bf16", "mfma_group"),
    ("l20_bf16_mfma_chain_b9", 20, 64, 256, tuple(synth.dilation_cycle(20)), 9, 150, "bf16", "multi_cu_mfma"),
]


def _setup(name, L, r, s, dil, B, T, dtype):
    import paper_1702_07825_amd as wn
    seed = zlib.crc32(name.encode()) % 1000
    w = synth.make_weights(L, r, s, seed=seed, bias_scale=0.2)
    w["w_out"] *= 4.0
    net = wn.WaveNet(w, dil, weight_dtype=dtype)
    cond = synth.make_cond(L, r, B, T, seed=seed, device="cuda")
    u = torch.tensor(synth.make_uniforms(B, T, seed=seed), device="cuda")
    return w, net, cond, u, oracle.Model(w, dil, bf16_weights=(dtype == "bf16"), int8_weights=(dtype == "i8"))


@pytest.mark.parametrize("model", MODELS, ids=[m[0] for m in MODELS])
def test_sampling_rules_match_the_oracle(model, monkeypatch):
    name, L, r, s, dil, B, T, dtype, kernel = model
    monkeypatch.setenv("WN_KERNEL", kernel)
    w, net, cond, u, om = _setup(name, L, r, s, dil, B, T, dtype)
    assert net.kernel_variant(B) == kernel
    cond_np, u_np = cond.cpu().numpy(), u.cpu().numpy()
    y_direct = net.generate(cond, u)
    for smp in SAMPLERS:
        print("%s sampler %s" % (name, smp), flush=True)
        y = net.generate(cond, u, sampler=smp)
        torch.cuda.synchronize()
        y_np = y.cpu().numpy()
        assert y_np.min() >= 0 and y_np.max() <= 255
        ys, _, mg = oracle.run_streams(om, cond_np, u=u_np, y_in=y_np, want_logits=False, threads=8, sampler=smp)
        ok = mg > MARGIN[smp[0]]
        mism = int(np.sum(ys[ok] != y_np[ok]))
        print("  confident %d/%d, mismatches %d, differs from direct at %d steps" %
              (int(ok.sum()), ok.size, mism, int((y_np != y_direct.cpu().numpy()).sum())), flush=True)
        assert ok.mean() > 0.5
        assert mism == 0
    net.close()


def test_sampling_rule_identities_on_the_gpu():
    """t = 1 and k = a are direct sampling and k = 1 is the mode, bit for bit, on one kernel."""
    w, net, cond, u, om = _setup("identities", 20, 64, 256, tuple(synth.dilation_cycle(20)), 3, 200, "f32")
    y0 = net.generate(cond, u)
    yt = net.generate(cond, u, sampler=(1, 1.0, 256))
    yk = net.generate(cond, u, sampler=(2, 1.0, 256))
    ym = net.generate(cond, u, sampler=(3, 1.0, 256))
    y1 = net.generate(cond, u, sampler=(2, 1.0, 1))
    torch.cuda.synchronize()
    assert torch.equal(yt, y0) and torch.equal(yk, y0)
    assert torch.equal(y1, ym)
    assert not torch.equal(ym, y0)
    net.close()


def test_sampler_arguments_are_checked():
    import paper_1702_07825_amd as wn
    w, net, cond, u, om = _setup("args", 4, 16, 32, (1, 2, 4, 8), 1, 10, "f32")
    for bad in [(5, 1.0, 256), (1, 0.0, 256), (1, float("nan"), 256), (1, float("inf"), 256), (2, 1.0, 0),
                (2, 1.0, 257)]:
        with pytest.raises(wn.WnError) as e:
            net.generate(cond, u, sampler=bad)
        assert e.value.code == wn.WN_EINVAL
    net.close()
