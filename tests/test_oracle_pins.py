"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every test here runs on the CPU.  Each one checks the oracle against an
independent computation or an exact property, so that a plausible mistake in it
(a dropped bias, a wrong sign, a history slot off by one, swapped gate halves,
a transposed matrix) fails at least one of them.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import synth
from tests import brute_force

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _model(L, r, s, dil, a=256, seed=0, bias=0.5, wscale=1.0, init=128, bf16=False, taps=1):
    w = synth.make_weights(L, r, s, a, seed=seed, bias_scale=bias, weight_scale=wscale, embed_taps=taps)
    return w, oracle.Model(w, dil, initial_sample=init, bf16_weights=bf16)


def _cond(L, r, T, seed):
    return synth.make_cond(L, r, 1, T, seed=seed)[0].numpy()


CASES = [
    # (L, r, s, a, dilations, T)
    (4, 16, 32, 256, (1, 2, 4, 8), 70),
    (3, 8, 12, 7, (3, 1, 2), 40),
    (5, 4, 6, 256, (2, 2, 1, 5, 3), 50),
    (1, 2, 3, 5, (1,), 12),
]


@pytest.mark.parametrize("taps", [1, 2])
@pytest.mark.parametrize("L,r,s,a,dil,T", CASES)
def test_incremental_equals_whole_sequence_conv(L, r, s, a, dil, T, taps):
    """History-buffer generation == the full causal dilated convolution (appendix A.1 equations),
    with the one-table embedding and with the width-2 input convolution (Section 5.1)."""
    w, m = _model(L, r, s, dil, a=a, seed=L * 7 + r, bias=0.5, init=a // 2, taps=taps)
    cond = _cond(L, r, T, seed=11)
    y = synth.make_samples(1, T, a=a, seed=5)[0]
    _, lg, _ = oracle.run(m, cond, y_in=y)
    ref = brute_force.logits(w, dil, cond, y, initial_sample=a // 2)
    np.testing.assert_allclose(lg, ref, rtol=0, atol=1e-10)
    assert np.abs(lg).max() > 1e-2  # not a degenerate all-zero case


def test_no_recurrence_special_case_is_a_dense_mlp():
    """With W_prev = W_cur = 0 each step's logits are a pure function of that step's conditioning."""
    L, r, s, a, dil, T = 3, 8, 16, 256, (1, 2, 4), 30
    w = synth.make_weights(L, r, s, a, seed=3, bias_scale=0.7)
    w["w_prev"][:] = 0
    w["w_cur"][:] = 0
    m = oracle.Model(w, dil)
    cond = _cond(L, r, T, seed=4).astype(np.float64)
    y = synth.make_samples(1, T, seed=9)[0]
    _, lg, _ = oracle.run(m, cond.astype(np.float32), y_in=y)
    pre = cond + w["b_gate"][None].astype(np.float64)               # [T, L, 2r]
    hid = np.tanh(pre[:, :, :r]) / (1.0 + np.exp(-pre[:, :, r:]))     # [T, L, r]
    q = hid.reshape(T, L * r) @ np.concatenate(list(w["w_skip"]), axis=1).T.astype(np.float64) + w["b_skip"]
    za = np.maximum(np.maximum(q, 0) @ w["w_relu"].T.astype(np.float64) + w["b_relu"], 0)
    ref = za @ w["w_out"].T.astype(np.float64) + w["b_out"]
    np.testing.assert_allclose(lg, ref, rtol=0, atol=1e-11)


def test_head_and_sampler_special_case():
    """W_out = 0, B_out = log(q): p equals q and the draw is the textbook inverse CDF (searchsorted)."""
    rng = np.random.default_rng(0)
    L, r, s, a, dil, T = 2, 4, 8, 256, (1, 2), 400
    w = synth.make_weights(L, r, s, a, seed=1, bias_scale=0.3)
    qv = rng.dirichlet(np.full(a, 0.7))
    qv = np.maximum(qv, 1e-12)
    qv /= qv.sum()
    w["w_out"][:] = 0
    w["b_out"] = np.log(qv).astype(np.float32)
    m = oracle.Model(w, dil)
    cond = _cond(L, r, T, seed=2)
    u = synth.make_uniforms(1, T, seed=3)[0]
    ys, lg, mg = oracle.run(m, cond, u=u)
    np.testing.assert_array_equal(lg, np.repeat(w["b_out"][None].astype(np.float64), T, 0))
    pf = np.exp(w["b_out"].astype(np.float64))
    pf /= pf.sum()
    _, p, _ = oracle.draw(lg[0], 0.5)
    np.testing.assert_allclose(p, pf, rtol=1e-12, atol=0)
    cdf = np.cumsum(pf)
    ref = np.minimum(np.searchsorted(cdf.astype(np.float32), u, side="right"), a - 1)
    np.testing.assert_array_equal(ys, ref)
    ref_margin = np.abs(u[:, None].astype(np.float64) - cdf[None, : a - 1]).min(axis=1)
    np.testing.assert_allclose(mg, ref_margin, rtol=0, atol=1e-15)


def test_draw_edge_cases():
    a = 256
    lg = np.zeros(a)
    assert oracle.draw(lg, 0.0)[0] == 0
    assert oracle.draw(lg, np.nextafter(np.float32(1), np.float32(0)))[0] == a - 1
    # uniform p: C_k = (k+1)/256 exactly; u = C_k goes up (strict <): y = k + 1
    assert oracle.draw(lg, 10 / 256)[0] == 10
    assert oracle.draw(lg, np.nextafter(np.float32(10 / 256), np.float32(0)))[0] == 9
    # all mass on one class
    spike = np.full(a, -1e4)
    spike[77] = 0
    for u in (0.0, 0.3, 0.999):
        assert oracle.draw(spike, u)[0] == 77
    # monotone in u
    rng = np.random.default_rng(1)
    lg = rng.standard_normal(a)
    ys = [oracle.draw(lg, u)[0] for u in np.linspace(0, 0.9999, 500)]
    assert all(b >= a_ for a_, b in zip(ys, ys[1:]))


def _changed_steps(ref, lg):
    return set(np.nonzero(np.any(ref != lg, axis=1))[0].tolist())


def _subset_sums(ds):
    sums = {0}
    for d in ds:
        sums |= {x + d for x in sums}
    return sums


@pytest.mark.parametrize("dil", [(1, 2, 4, 8), (3, 1, 2), (2, 5)])
def test_receptive_field_and_causality(dil):
    """Step t sees exactly y_{t-1-o}, o in the subset sums of the dilations (so R = 1 + sum d for 1,2,4,...)."""
    L, r, s = len(dil), 6, 8
    T = 3 * (1 + sum(dil)) + 10
    w, m = _model(L, r, s, dil, seed=21, bias=0.4)
    cond = _cond(L, r, T, seed=22)
    y = synth.make_samples(1, T, seed=23)[0]
    _, ref, _ = oracle.run(m, cond, y_in=y)
    k = T // 3
    y2 = y.copy()
    y2[k] = (y2[k] + 101) % 256
    _, lg, _ = oracle.run(m, cond, y_in=y2)
    expect = {k + 1 + o for o in _subset_sums(dil)} & set(range(T))
    assert _changed_steps(ref, lg) == expect
    if dil == (1, 2, 4, 8):
        assert max(expect) - k == oracle.receptive_field(dil) == 16
        assert expect == set(range(k + 1, k + 17))
    # conditioning of layer j at step k reaches steps k + (subset sums of the later dilations)
    for j in range(L):
        c2 = cond.copy()
        c2[k, j, :] += 0.5
        _, lg, _ = oracle.run(m, c2, y_in=y)
        assert _changed_steps(ref, lg) == {k + o for o in _subset_sums(dil[j + 1:])}


@pytest.mark.parametrize("dil", [(1, 2, 4, 8), (3, 1, 2)])
def test_two_tap_receptive_field_and_causality(dil):
    """With two embedding taps y_k reaches steps k + 1 + e + o, e in {0, 1}, o in the subset sums
    of the dilations: R = 2 + sum d (17 for 1,2,4,8)."""
    L, r, s = len(dil), 6, 8
    T = 3 * (2 + sum(dil)) + 10
    w, m = _model(L, r, s, dil, seed=24, bias=0.4, taps=2)
    cond = _cond(L, r, T, seed=25)
    y = synth.make_samples(1, T, seed=26)[0]
    _, ref, _ = oracle.run(m, cond, y_in=y)
    k = T // 3
    y2 = y.copy()
    y2[k] = (y2[k] + 101) % 256
    _, lg, _ = oracle.run(m, cond, y_in=y2)
    expect = {k + 1 + e + o for e in (0, 1) for o in _subset_sums(dil)} & set(range(T))
    assert _changed_steps(ref, lg) == expect
    assert max(expect) - k == m.receptive_field == 2 + sum(dil)
    if dil == (1, 2, 4, 8):
        assert expect == set(range(k + 1, k + 18))


def test_two_tap_embedding_special_cases():
    """E_prev = 0 reproduces the one-table model with E = E_cur exactly; E_cur = 0 makes step t's
    input depend on y_{t-2} alone, and step 0's on nothing but B_embed (zero left padding)."""
    L, r, s, dil, T = 3, 8, 16, (1, 2, 4), 60
    w = synth.make_weights(L, r, s, seed=41, bias_scale=0.4, embed_taps=2)
    cond = _cond(L, r, T, seed=42)
    y = synth.make_samples(1, T, seed=43)[0]
    w0 = dict(w)
    w0["embed"] = w["embed"].copy()
    w0["embed"][0] = 0.0
    w1 = dict(w)
    w1["embed"] = w["embed"][1].copy()
    _, lg0, _ = oracle.run(oracle.Model(w0, dil), cond, y_in=y)
    _, lg1, _ = oracle.run(oracle.Model(w1, dil), cond, y_in=y)
    np.testing.assert_array_equal(lg0, lg1)
    wp = dict(w)
    wp["embed"] = w["embed"].copy()
    wp["embed"][1] = 0.0
    mp = oracle.Model(wp, dil)
    _, ref, _ = oracle.run(mp, cond, y_in=y)
    # changing only the initial sample (step 0's y_{t-1}, step 1's y_{t-2}) changes nothing at step 0
    _, lg, _ = oracle.run(oracle.Model(wp, dil, initial_sample=3), cond, y_in=y)
    assert np.array_equal(lg[0], ref[0]) and not np.array_equal(lg[1], ref[1])
    # with E_prev the only table and no recurrence (W_prev = 0, W_cur = 0 past layer 1), y_k
    # reaches step k + 2 only
    wz = dict(wp)
    wz["w_prev"] = np.zeros_like(w["w_prev"])
    wz["w_cur"] = w["w_cur"].copy()
    wz["w_cur"][1:] = 0.0
    y2 = y.copy()
    y2[20] = (y2[20] + 77) % 256
    mz = oracle.Model(wz, dil)
    _, a_, _ = oracle.run(mz, cond, y_in=y)
    _, b_, _ = oracle.run(mz, cond, y_in=y2)
    assert _changed_steps(a_, b_) == {22}


def test_receptive_field_paper_figures():
    g = json.load(open(os.path.join(GOLDEN, "paper_figures.json")))
    r40 = oracle.receptive_field(synth.dilation_cycle(40))
    r20 = oracle.receptive_field(synth.dilation_cycle(20))
    assert (r40, r20) == (4093, 2047)
    assert abs(r20 / r40 - g["receptive_field_ratio_20_vs_40_layers"]["value"]) < 1e-3
    # 40 layers at 48 kHz: the paper says 83 ms; the 2^(i mod 10) schedule gives 85.3 ms
    assert abs(r40 / 48000 - g["receptive_field_40_layers_at_48khz_s"]["value"]) / 0.083 < 0.03


def test_chunked_equals_one_shot():
    L, r, s, dil, T = 4, 16, 32, (1, 2, 4, 8), 200
    w, m = _model(L, r, s, dil, seed=31, bias=0.2)
    cond = _cond(L, r, T, seed=32)
    u = synth.make_uniforms(1, T, seed=33)[0]
    y1, lg1, _ = oracle.run(m, cond, u=u)
    st = oracle.State(m)
    parts = []
    for a_, b_ in [(0, 1), (1, 17), (17, 17), (17, 100), (100, 200)]:
        ys, lg, _ = oracle.run(m, cond[a_:b_], u=u[a_:b_], state=st)
        parts.append((ys, lg))
    assert st.t == T and st.last_sample == y1[-1]
    np.testing.assert_array_equal(np.concatenate([p[0] for p in parts]), y1)


def test_two_tap_chunked_equals_one_shot():
    """The state carries y_{t-2} across calls: chunk boundaries change nothing with two taps."""
    L, r, s, dil, T = 4, 16, 32, (1, 2, 4, 8), 120
    w, m = _model(L, r, s, dil, seed=34, bias=0.2, taps=2)
    cond = _cond(L, r, T, seed=35)
    u = synth.make_uniforms(1, T, seed=36)[0]
    y1, lg1, _ = oracle.run(m, cond, u=u)
    st = oracle.State(m)
    assert st.prev_sample == -1
    parts = []
    for a_, b_ in [(0, 1), (1, 2), (2, 50), (50, 120)]:
        parts.append(oracle.run(m, cond[a_:b_], u=u[a_:b_], state=st)[:2])
    assert st.t == T and st.last_sample == y1[-1] and st.prev_sample == y1[-2]
    np.testing.assert_array_equal(np.concatenate([p[0] for p in parts]), y1)
    np.testing.assert_array_equal(np.concatenate([p[1] for p in parts]), lg1)
    np.testing.assert_array_equal(np.concatenate([p[1] for p in parts]), lg1)


def test_generate_equals_teacher_forcing_on_its_own_samples():
    L, r, s, dil, T = 4, 16, 32, (1, 2, 4, 8), 150
    w, m = _model(L, r, s, dil, seed=41)
    cond = _cond(L, r, T, seed=42)
    u = synth.make_uniforms(1, T, seed=43)[0]
    y, lg, mg = oracle.run(m, cond, u=u)
    y2, lg2, mg2 = oracle.run(m, cond, u=u, y_in=y)
    np.testing.assert_array_equal(lg, lg2)
    np.testing.assert_array_equal(y, y2)
    np.testing.assert_array_equal(mg, mg2)


def test_bf16_weights_round_to_nearest_even():
    """The oracle's bf16 storage mode == the fp32 oracle on weights rounded by torch's bfloat16 cast."""
    L, r, s, dil, T = 3, 16, 32, (1, 2, 4), 40
    w = synth.make_weights(L, r, s, seed=51, bias_scale=0.3)
    mats = ("embed", "w_prev", "w_cur", "w_res", "w_skip", "w_relu", "w_out")
    wr = {k: (torch.tensor(v).to(torch.bfloat16).to(torch.float32).numpy() if k in mats else v)
          for k, v in w.items()}
    for k in mats:
        np.testing.assert_array_equal(oracle.round_bf16(w[k]), wr[k])
    edge = np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 3.0e38, np.inf, -0.0], np.float32)
    np.testing.assert_array_equal(oracle.round_bf16(edge),
                                  torch.tensor(edge).to(torch.bfloat16).to(torch.float32).numpy())
    cond = _cond(L, r, T, seed=52)
    y = synth.make_samples(1, T, seed=53)[0]
    _, lg_b, _ = oracle.run(oracle.Model(w, dil, bf16_weights=True), cond, y_in=y)
    _, lg_r, _ = oracle.run(oracle.Model(wr, dil), cond, y_in=y)
    np.testing.assert_array_equal(lg_b, lg_r)
    _, lg_f, _ = oracle.run(oracle.Model(w, dil), cond, y_in=y)
    assert 1e-5 < np.abs(lg_b - lg_f).max() < 5e-2


def _numpy_quantize_rows_i8(w):
    """int8 per-row quantizer written with numpy: scale = max|w| / 127 in fp32, codes = nearest
    integer of w / scale (ties to even) clipped to +-127, zero rows all zero."""
    w = np.asarray(w, np.float32).reshape(-1, np.asarray(w).shape[-1])
    scale = (np.abs(w).max(axis=1).astype(np.float64) / 127.0).astype(np.float32)
    safe = np.where(scale > 0, scale, 1).astype(np.float64)
    codes = np.clip(np.rint(w.astype(np.float64) / safe[:, None]), -127, 127)
    codes[scale == 0] = 0
    return codes.astype(np.int8), scale


def test_int8_quantizer_matches_numpy():
    """The oracle's int8 storage rule == a numpy quantizer, on random rows, a zero row, a row with one
    non-zero entry and rows whose quotients are exact halves (ties go to the even code)."""
    rng = np.random.default_rng(61)
    w = rng.normal(0, 0.2, (40, 64)).astype(np.float32)
    w[3] = 0.0
    w[5] = 0.0
    w[5, 17] = -0.37
    step = np.float32(2.0 ** -7)  # rows with max 127 * 2^-7 have scale 2^-7 exactly
    for i, row in enumerate((8, 9, 10)):
        w[row] = (np.arange(64) % 9 - 4 + 0.5).astype(np.float32) * step
        w[row, 0] = 127 * step * (-1) ** i
    codes, scale = oracle.quantize_rows_i8(w)
    codes_np, scale_np = _numpy_quantize_rows_i8(w)
    np.testing.assert_array_equal(scale, scale_np)
    np.testing.assert_array_equal(codes, codes_np)
    assert scale[3] == 0 and not codes[3].any()
    assert codes[5, 17] == -127 and np.count_nonzero(codes[5]) == 1
    assert scale[8] == step
    # ties: k + 1/2 goes to the even one of k, k + 1
    half = (np.arange(64) % 9 - 4 + 0.5)[1:]
    np.testing.assert_array_equal(codes[8, 1:], (2 * np.round(half / 2)).astype(np.int8))
    assert np.abs(codes).max() <= 127
    # every weight is within half a step of its stored value
    err = np.abs(codes.astype(np.float64) * scale[:, None] - w)
    assert np.all(err <= 0.5 * scale[:, None].astype(np.float64) * (1 + 1e-6))


def test_int8_weights_model():
    """The int8 storage mode uses code * scale exactly: with weights already on an int8 grid whose rows
    reach +-127 steps (scale a power of two) it equals the fp32 oracle bit for bit; in general it
    matches the fp32 oracle run on the dequantized weights (rounded to fp32) within rounding, and it
    differs from the unquantized model."""
    L, r, s, dil, T = 3, 16, 32, (1, 2, 4), 40
    mats = ("embed", "w_prev", "w_cur", "w_res", "w_skip", "w_relu", "w_out")
    w = synth.make_weights(L, r, s, seed=62, bias_scale=0.3)
    cond = _cond(L, r, T, seed=63)
    y = synth.make_samples(1, T, seed=64)[0]
    rng = np.random.default_rng(65)
    grid = dict(w)
    for k in mats:
        cols = w[k].shape[-1]
        c = rng.integers(-126, 127, w[k].shape).reshape(-1, cols)
        c[:, 0] = 127
        e = rng.integers(-9, -4, c.shape[0])
        grid[k] = (c * np.ldexp(1.0, e)[:, None]).reshape(w[k].shape).astype(np.float32)
    _, lg_q, _ = oracle.run(oracle.Model(grid, dil, int8_weights=True), cond, y_in=y)
    _, lg_g, _ = oracle.run(oracle.Model(grid, dil), cond, y_in=y)
    np.testing.assert_array_equal(lg_q, lg_g)
    deq = dict(w)
    for k in mats:
        codes, scale = _numpy_quantize_rows_i8(w[k])
        deq[k] = (codes.astype(np.float64) * scale[:, None].astype(np.float64)).astype(np.float32).reshape(w[k].shape)
    _, lg_8, _ = oracle.run(oracle.Model(w, dil, int8_weights=True), cond, y_in=y)
    _, lg_d, _ = oracle.run(oracle.Model(deq, dil), cond, y_in=y)
    assert np.abs(lg_8 - lg_d).max() < 1e-5
    _, lg_f, _ = oracle.run(oracle.Model(w, dil), cond, y_in=y)
    assert 1e-4 < np.abs(lg_8 - lg_f).max() < 5e-2


def test_model_size_and_flops_match_the_paper():
    g = json.load(open(os.path.join(GOLDEN, "paper_figures.json")))
    n = oracle.param_count(40, 64, 256)
    shapes = synth.weight_shapes(40, 64, 256, 256)
    assert n == sum(int(np.prod(s)) for s in shapes.values()) == 1630528
    assert abs(n - g["parameters"]["value"]) / g["parameters"]["value"] < 0.05
    assert abs(4 * n - g["parameters"]["bytes_fp32"]) / g["parameters"]["bytes_fp32"] < 0.05
    bw = 4 * n * g["weight_bandwidth_per_second"]["rate_hz"]
    assert abs(bw - g["weight_bandwidth_per_second"]["value"]) / g["weight_bandwidth_per_second"]["value"] < 0.10
    f = oracle.flops_per_sample(40, 64, 256, 256, 10, 10) * 16384
    assert abs(f - g["flops_per_audio_second"]["value"]) / g["flops_per_audio_second"]["value"] < 0.01
    # per layer: 10 r^2 + 11 r (the r-only terms of the layer cost)
    per_layer = oracle.flops_per_sample(2, 64, 0, 0, 0, 0) - oracle.flops_per_sample(1, 64, 0, 0, 0, 0)
    assert per_layer == 10 * 64 ** 2 + 11 * 64
    assert abs(per_layer - g["flops_per_layer"]["value"]) / g["flops_per_layer"]["value"] < 0.02
    # 60 us per sample at 16 kHz and 1.5 us per layer for 40 layers
    assert abs(1e6 / 16384 - g["per_sample_budget_us_16khz"]["value"]) < 2
    assert abs(1e6 / 16384 / 40 - g["per_layer_budget_us_40_layers"]["value"]) < 0.1


def test_mulaw_round_trip_and_closed_form():
    mu = oracle.mulaw
    codes = np.arange(256)
    np.testing.assert_array_equal(mu.encode(mu.decode(codes)), codes)
    assert mu.encode(0.0) == 128 and mu.encode(1.0) == 255 and mu.encode(-1.0) == 0
    np.testing.assert_allclose(mu.decode(255 - codes), -mu.decode(codes), atol=1e-15)
    x = np.linspace(-1, 1, 20001)
    np.testing.assert_allclose(mu.expand(mu.compress(x)), x, atol=1e-12)
    e = mu.encode(x)
    assert np.all(np.diff(e) >= 0)
    # companding: steps near 0 are about (1 + mu) / ln(1 + mu) * ... finer than near full scale
    dec = mu.decode(codes)
    step0, step1 = dec[129] - dec[128], dec[255] - dec[254]
    assert step1 / step0 > 100
    # the transform's endpoints and odd symmetry
    assert mu.compress(1.0) == pytest.approx(1.0, abs=1e-15)
    np.testing.assert_allclose(mu.compress(-x), -mu.compress(x), atol=1e-15)


def test_history_is_zero_padded_before_the_first_step():
    """At t = 0 every layer's past input is zero: the W_prev halves contribute nothing."""
    L, r, s, dil = 3, 8, 16, (1, 2, 4)
    w, m = _model(L, r, s, dil, seed=61, bias=0.3)
    cond = _cond(L, r, 1, seed=62)
    _, lg, _ = oracle.run(m, cond, y_in=np.array([5], np.int32))
    w2 = {k: v.copy() for k, v in w.items()}
    w2["w_prev"][:] = 123.0
    _, lg2, _ = oracle.run(oracle.Model(w2, dil), cond, y_in=np.array([5], np.int32))
    np.testing.assert_array_equal(lg, lg2)


def test_window_of_receptive_field_reproduces_full_run():
    """Step t's logits depend only on steps [t - sum(d), t]: a teacher-forced run over that window,
    started from zero histories with y_{t0-1} as its initial sample, gives them bit for bit."""
    L, r, s, dil = 4, 16, 32, (1, 2, 4, 8)
    T = 120
    w, m = _model(L, r, s, dil, seed=71, bias=0.3)
    cond = _cond(L, r, T, seed=72)
    u = synth.make_uniforms(1, T, seed=73)[0]
    y, lg, mg = oracle.run(m, cond, u=u)
    sd = sum(dil)
    for t in (sd, sd + 1, 57, T - 1):
        t0 = t - sd
        mw = oracle.Model(w, dil, initial_sample=int(y[t0 - 1]) if t0 > 0 else 128)
        yw, lw, mw_ = oracle.run(mw, cond[t0:t + 1], u=u[t0:t + 1], y_in=y[t0:t + 1])
        np.testing.assert_array_equal(lw[-1], lg[t])
        assert yw[-1] == y[t] and mw_[-1] == mg[t]
    # one step shorter is not enough (the oldest input is reached through every layer)
    t = T - 1
    t0 = t - sd + 1
    mw = oracle.Model(w, dil, initial_sample=int(y[t0 - 1]))
    _, lw, _ = oracle.run(mw, cond[t0:t + 1], y_in=y[t0:t + 1])
    assert np.any(lw[-1] != lg[t])


def _known_distribution_run(seed, T=400):
    """A model whose every step has the same known distribution: W_out = 0, B_out = log q."""
    rng = np.random.default_rng(seed)
    L, r, s, a, dil = 2, 4, 8, 256, (1, 2)
    w = synth.make_weights(L, r, s, a, seed=seed, bias_scale=0.3)
    qv = np.maximum(rng.dirichlet(np.full(a, 0.5)), 1e-12)
    w["w_out"][:] = 0
    w["b_out"] = np.log(qv / qv.sum()).astype(np.float32)
    m = oracle.Model(w, dil)
    cond = _cond(L, r, T, seed=seed + 1)
    u = synth.make_uniforms(1, T, seed=seed + 2)[0]
    pf = np.exp(w["b_out"].astype(np.float64))
    return m, cond, u, pf / pf.sum(), a


@pytest.mark.parametrize("sampler", [(1, 0.5, 256), (1, 2.0, 256), (2, 1.0, 1), (2, 1.0, 3), (2, 1.0, 17),
                                     (2, 1.0, 256), (3, 1.0, 256), (4, 1.0, 256)])
def test_sampling_variants_on_a_known_distribution(sampler):
    """Each rule of the paper's sampling appendix against its textbook form on a known P:
    temperature draws from P^(1/t)/Z, top k from P kept at or above its k-th largest value and
    renormalised, mode is argmax P, mean is E_P[y] to the nearest index; draws are inverse CDFs
    (numpy searchsorted on the float32-rounded CDF)."""
    mode, t, k = sampler
    m, cond, u, p, a = _known_distribution_run(seed=40 + mode * 7 + k % 5)
    ys, lg, mg = oracle.run(m, cond, u=u, sampler=sampler)
    if mode == 3:
        ref = np.full(len(u), int(np.argmax(p)))
    elif mode == 4:
        ref = np.full(len(u), int(np.floor((np.arange(a) * p).sum() + 0.5)))
    else:
        q = p ** (1.0 / t) if mode == 1 else p.copy()
        last = a - 1
        if mode == 2:
            kth = np.sort(p)[::-1][k - 1]
            q[p < kth] = 0.0
            last = int(np.nonzero(q)[0].max())
        q /= q.sum()
        cdf = np.cumsum(q)
        ref = np.minimum(np.searchsorted(cdf.astype(np.float32)[:a - 1], u, side="right"), last)
    ok = mg > 1e-9
    assert ok.sum() > 0.9 * len(u)
    np.testing.assert_array_equal(ys[ok], ref[ok])
    if mode == 2:
        assert set(np.unique(ys)) <= set(np.nonzero(p >= np.sort(p)[::-1][k - 1])[0])


def test_sampling_variant_identities_on_a_model():
    """On a random model's own generation: t = 1 and k = a are direct sampling, k = 1 is the
    mode, and a temperature near 0 draws the mode wherever the top two logits are apart."""
    L, r, s, dil, T = 4, 16, 32, (1, 2, 4, 8), 300
    w = synth.make_weights(L, r, s, seed=5, bias_scale=0.5)
    w["w_out"] *= 4.0  # sharper distributions, so that the mode and the draws differ visibly
    m = oracle.Model(w, dil)
    cond = _cond(L, r, T, seed=6)
    u = synth.make_uniforms(1, T, seed=7)[0]
    y0, _, _ = oracle.run(m, cond, u=u)
    for smp in [(1, 1.0, 256), (2, 1.0, 256)]:
        np.testing.assert_array_equal(oracle.run(m, cond, u=u, sampler=smp)[0], y0)
    ym, lg, _ = oracle.run(m, cond, u=u, sampler=(3, 1.0, 256))
    np.testing.assert_array_equal(oracle.run(m, cond, u=u, sampler=(2, 1.0, 1))[0], ym)
    np.testing.assert_array_equal(ym, np.argmax(lg, axis=1))
    assert not np.array_equal(ym, y0)
    yc, lgc, _ = oracle.run(m, cond, u=u, sampler=(1, 1e-4, 256))
    top2 = np.sort(lgc, axis=1)[:, -2:]
    apart = (top2[:, 1] - top2[:, 0]) > 1e-2
    np.testing.assert_array_equal(yc[apart], np.argmax(lgc, axis=1)[apart])
    # teacher forcing on the mode's own samples reproduces its logits
    _, lgt, _ = oracle.run(m, cond, y_in=ym)
    np.testing.assert_array_equal(lgt, lg)


def test_sampler_rejects_invalid_rules():
    lg = np.zeros(256)
    for bad in [(1, 0.0, 256), (1, -1.0, 256), (2, 1.0, 0), (2, 1.0, 257), (5, 1.0, 256)]:
        with pytest.raises(ValueError):
            oracle.sample(lg, 0.5, bad)


@pytest.mark.parametrize("lo,hi,w_hi", [(100, 101, 0.7), (100, 101, 0.3), (0, 255, 0.5004), (3, 9, 0.3)])
def test_sampling_mean_rounds_to_the_nearest_index(lo, hi, w_hi):
    """E_P[y] of a distribution on two classes (plus a negligible floor elsewhere) is
    lo + w_hi (hi - lo) up to that floor; the mean rule takes the nearest index."""
    a = 256
    p = np.full(a, 1e-30)
    p[lo], p[hi] = 1.0 - w_hi, w_hi
    lg = np.log(p)
    y, mg = oracle.sample(lg, 0.5, (4, 1.0, a))
    mean = lo + w_hi * (hi - lo)
    assert mg > 1e-6
    assert y == int(np.floor(mean + 0.5))


# ---------------------------------------------------------------------------------------------
# Conditioning network (Appendix A.2)
# ---------------------------------------------------------------------------------------------

def _small_cond(seed, F=7, h1=5, h2=6, Tf=11, bias=0.3):
    w = synth.make_cond_weights(F, h1, h2, seed=seed, bias_scale=bias)
    x = np.random.default_rng(seed).normal(size=(Tf, F)).astype(np.float32)
    return w, x


@pytest.mark.parametrize("frame_rate,audio_rate", [(4, 16), (3, 8), (1, 1), (256, 16000)])
def test_conditioning_equals_whole_sequence_form(frame_rate, audio_rate):
    """Oracle (per-frame recurrences) == torch conv1d gates + closed-form fo-pool + flipped
    backward direction + gather upsampling, including non-integer rate ratios."""
    w, x = _small_cond(seed=frame_rate + audio_rate)
    Tf = x.shape[0]
    Ta = (Tf * audio_rate + frame_rate - 1) // frame_rate
    c = oracle.condition(w, x, Ta, frame_rate, audio_rate)
    ref = brute_force.condition(w, x, Ta, frame_rate, audio_rate)
    np.testing.assert_allclose(c, ref, rtol=0, atol=1e-12)
    assert np.abs(c).max() > 1e-2


def test_conditioning_with_forget_gate_zero_is_feedforward():
    """f = 0 and o = 1 in both layers: h = h~, so the network is tanh(conv(tanh(conv(x)))), written
    here with numpy matmuls frame by frame."""
    w, x = _small_cond(seed=3)
    for k in ("1", "2"):
        h = w["b" + k].shape[1] // 3
        w["w" + k][:, h:] = 0.0                    # o and f rows see no input
        w["b" + k][:, h:2 * h] = 1e4               # o = 1
        w["b" + k][:, 2 * h:] = -1e4               # f = 0
    Tf = x.shape[0]
    z = x.astype(np.float64)
    for k in ("1", "2"):
        wk, bk = w["w" + k].astype(np.float64), w["b" + k].astype(np.float64)
        h = bk.shape[1] // 3
        prev_f = np.vstack([np.zeros((1, z.shape[1])), z[:-1]])   # forward direction: frame t - 1
        prev_b = np.vstack([z[1:], np.zeros((1, z.shape[1]))])    # backward direction: frame t + 1
        fwd = np.tanh(prev_f @ wk[0, :h, 0].T + z @ wk[0, :h, 1].T + bk[0, :h])
        bwd = np.tanh(prev_b @ wk[1, :h, 0].T + z @ wk[1, :h, 1].T + bk[1, :h])
        z = np.hstack([fwd, bwd])
    h2 = z.shape[1] // 2
    ref = np.stack([z[:, :h2], z[:, h2:]], 2).reshape(Tf, 2 * h2)
    np.testing.assert_allclose(oracle.condition(w, x, Tf, 1, 1), ref, rtol=0, atol=1e-12)


def test_conditioning_forget_gate_one_holds_zero_and_interleave():
    """f = 1 holds h at its initial 0 (all outputs 0); o = 0 in the backward direction of the
    second layer zeroes exactly the odd (backward) channels of the interleaved output."""
    w, x = _small_cond(seed=4)
    h2 = w["b2"].shape[1] // 3
    w1 = {k: v.copy() for k, v in w.items()}
    w1["w2"][:, 2 * h2:] = 0.0
    w1["b2"][:, 2 * h2:] = 1e4
    assert np.all(oracle.condition(w1, x, 11, 1, 1) == 0.0)
    wb = {k: v.copy() for k, v in w.items()}
    wb["w2"][1, h2:2 * h2] = 0.0
    wb["b2"][1, h2:2 * h2] = -1e4
    c = oracle.condition(wb, x, 11, 1, 1)
    assert np.all(c[:, 1::2] == 0.0) and np.abs(c[:, 0::2]).min() > 0.0
    np.testing.assert_array_equal(c[:, 0::2], oracle.condition(w, x, 11, 1, 1)[:, 0::2])


def test_conditioning_time_reversal():
    """Reversing the frames and swapping the two directions' weights (and, in layer 2, the halves
    of its input, since layer 1's output then comes backward half first) reverses the output in
    time and swaps each interleaved channel pair."""
    w, x = _small_cond(seed=5)
    sw = {k: v[::-1].copy() for k, v in w.items()}
    h1 = w["b1"].shape[1] // 3
    sw["w2"] = np.concatenate([sw["w2"][..., h1:], sw["w2"][..., :h1]], axis=-1).copy()
    c = oracle.condition(w, x, x.shape[0], 1, 1)
    cr = oracle.condition(sw, x[::-1].copy(), x.shape[0], 1, 1)
    swapped = cr.reshape(cr.shape[0], -1, 2)[:, :, ::-1].reshape(cr.shape)
    np.testing.assert_allclose(swapped[::-1], c, rtol=0, atol=1e-12)


def test_conditioning_upsampling_by_repetition():
    """256 Hz frames at 16384 Hz repeat 64 times each; at 16000 Hz the runs are 62 or 63 long."""
    w, x = _small_cond(seed=6, Tf=20)
    for audio_rate, runs in ((16384, {64}), (16000, {62, 63})):
        Ta = 19 * audio_rate // 256
        c = oracle.condition(w, x, Ta, 256, audio_rate)
        change = np.nonzero(np.any(c[1:] != c[:-1], axis=1))[0] + 1
        lengths = np.diff(np.concatenate([[0], change]))
        assert set(lengths.tolist()) <= runs and len(lengths) == 18
    with pytest.raises(ValueError):
        oracle.condition(w, x, 20 * 64 + 1, 256, 16384)  # past the last frame


# ---------------------------------------------------------------------------------------------
# Approximate nonlinearities (Appendix C; error figures in Section 5.1)
# ---------------------------------------------------------------------------------------------

def test_approximate_nonlinearities_meet_the_papers_error_figures():
    """Against numpy's tanh, logistic and exp on dense grids: the largest errors are the paper's
    figures to the digits it prints (tanh 1.5e-3; sigmoid 2.5e-3 printed, 2.59e-3 measured; exp
    2.4e-5 printed: the fit's relative error at the top of its interval), and close to them, so
    that a changed coefficient moves them out of the window."""
    x = np.linspace(-30.0, 30.0, 1200001)
    et = np.abs(oracle.approx_nonlin("tanh", x) - np.tanh(x)).max()
    es = np.abs(oracle.approx_nonlin("sigmoid", x) - 1.0 / (1.0 + np.exp(-x))).max()
    assert 1.50e-3 <= et <= 1.52e-3, et
    assert 2.55e-3 <= es <= 2.60e-3, es
    v = np.linspace(-85.0, 0.0, 4000001)
    ev = oracle.approx_nonlin("exp", v)
    rel = np.abs(ev - np.exp(v)) / np.exp(v)
    # the fit's own relative error (2^z at z = 0 is 1 + 2.62e-5) everywhere but in narrow windows
    # just below each power of two, where the fit's excess carries the fraction into the exponent
    # and the error doubles to the fit's error at z = 1 (4.79e-5)
    carry = ev >= 2.0 ** np.ceil(v / np.log(2.0))
    assert 0 < carry.mean() < 1e-4
    assert 2.55e-5 <= rel[~carry].max() <= 2.65e-5, rel[~carry].max()
    assert 4.7e-5 <= rel.max() <= 4.8e-5, rel.max()
    assert np.abs(ev - np.exp(v)).max() <= 4.8e-5


def test_approximate_nonlinearities_identities():
    x = np.linspace(-12.0, 12.0, 24001)
    t, sg = oracle.approx_nonlin("tanh", x), oracle.approx_nonlin("sigmoid", x)
    np.testing.assert_array_equal(t, -oracle.approx_nonlin("tanh", -x))          # odd
    np.testing.assert_allclose(sg + oracle.approx_nonlin("sigmoid", -x), 1.0, rtol=0, atol=4.5e-16)
    assert oracle.approx_nonlin("tanh", np.array([0.0]))[0] == 0.0
    assert oracle.approx_nonlin("sigmoid", np.array([0.0]))[0] == 0.5
    assert np.all(np.diff(t) >= 0) and np.all(np.diff(sg) >= 0)                   # monotone
    assert np.all(np.abs(t) < 1) and np.all((sg > 0) & (sg < 1))
    v = np.linspace(-100.0, 0.0, 200001)
    ev = oracle.approx_nonlin("exp", v)
    assert np.all(np.diff(ev) >= 0)
    # powers of two: y = k ln 2 / ln 2 is k or a rounding below it, so the value is 2^k times
    # g(0) = 1 + 2.62e-5, or the carried fit at z = 1 (1 + 4.79e-5)
    k = np.arange(-120, 1)
    np.testing.assert_allclose(oracle.approx_nonlin("exp", k * np.log(2.0)), 2.0 ** k, rtol=4.8e-5, atol=0)
    assert np.all(oracle.approx_nonlin("exp", k * np.log(2.0)) > 2.0 ** k)
    # no exponent left below 2^-126: zero
    assert np.all(oracle.approx_nonlin("exp", np.array([-88.0, -100.0, -1e4])) == 0.0)


def test_approximate_nonlinearities_in_the_model():
    """With approx_nonlin the gate uses the approximate tanh and sigmoid (whole-sequence form with
    those two functions: 1e-10) and the draw the approximate exp (known-distribution special case:
    numpy searchsorted on the normalised approximate exps)."""
    L, r, s, a, dil, T = 4, 16, 32, 256, (1, 2, 4, 8), 60
    w = synth.make_weights(L, r, s, a, seed=51, bias_scale=0.5)
    m = oracle.Model(w, dil, approx_nonlin=True)
    cond = _cond(L, r, T, seed=52)
    y = synth.make_samples(1, T, seed=53)[0]
    _, lg, _ = oracle.run(m, cond, y_in=y)

    def ta(t):
        return torch.tensor(oracle.approx_nonlin("tanh", t.numpy()), dtype=torch.float64)

    def sa(t):
        return torch.tensor(oracle.approx_nonlin("sigmoid", t.numpy()), dtype=torch.float64)

    ref = brute_force.logits(w, dil, cond, y, tanh=ta, sigmoid=sa)
    np.testing.assert_allclose(lg, ref, rtol=0, atol=1e-10)
    _, lg_exact, _ = oracle.run(oracle.Model(w, dil), cond, y_in=y)
    assert 1e-4 < np.abs(lg - lg_exact).max() < 5e-2

    rng = np.random.default_rng(5)
    qv = rng.dirichlet(np.full(a, 0.7))
    w2 = synth.make_weights(2, 4, 8, a, seed=1, bias_scale=0.3)
    w2["w_out"][:] = 0
    w2["b_out"] = np.log(np.maximum(qv, 1e-12)).astype(np.float32)
    m2 = oracle.Model(w2, (1, 2), approx_nonlin=True)
    u = synth.make_uniforms(1, 400, seed=6)[0]
    ys, _, mg = oracle.run(m2, _cond(2, 4, 400, seed=7), u=u)
    b = w2["b_out"].astype(np.float64)
    pa = oracle.approx_nonlin("exp", b - b.max())
    cdf = np.cumsum(pa / pa.sum())
    ref = np.minimum(np.searchsorted(cdf.astype(np.float32), u, side="right"), a - 1)
    np.testing.assert_array_equal(ys, ref)
    np.testing.assert_allclose(mg, np.abs(u[:, None].astype(np.float64) - cdf[None, : a - 1]).min(axis=1),
                               rtol=0, atol=1e-14)
    _, p_ax, _ = oracle.draw(b, 0.5, approx_nonlin=True)
    _, p_ex, _ = oracle.draw(b, 0.5)
    np.testing.assert_allclose(p_ax, pa / pa.sum(), rtol=1e-13, atol=0)
    assert np.abs(p_ax / p_ex - 1).max() > 1e-5
    for sm in [(1, 0.7, a), (2, 1.0, 12), (4, 1.0, a)]:   # temperature, top k, mean take it too
        y_ax = oracle.sample(b, 0.37, sm, approx_nonlin=True)[0]
        y_ex = oracle.sample(b, 0.37, sm)[0]
        assert abs(y_ax - y_ex) <= 1
