"""Whole-sequence (non-incremental) WaveNet forward pass, used only to pin the oracle.

It evaluates the appendix's equations (Appendix A.1) over the entire teacher-forced
sequence at once, with torch's dilated conv1d (kernel width 2, zero left padding)
instead of per-step matrix-vector products and history buffers, and with the skip
projection applied to the concatenation of all layers' hidden states.  Float64, CPU.
"""
import numpy as np
import torch
import torch.nn.functional as F


def logits(w, dilations, cond, y_in, initial_sample=128, tanh=torch.tanh, sigmoid=torch.sigmoid):
    """w: dict of fp32 arrays; cond [T, l, 2r]; y_in [T] (step t consumes y_in[t-1]). Returns [T, a] float64.
    ``tanh`` and ``sigmoid`` are the gate's nonlinearities (float64 tensor -> tensor)."""
    t64 = {k: torch.tensor(np.asarray(v), dtype=torch.float64) for k, v in w.items()}
    L, two_r, r = t64["w_prev"].shape
    a = t64["w_out"].shape[0]
    cond = torch.tensor(np.asarray(cond), dtype=torch.float64)
    T = cond.shape[0]
    y_prev = torch.tensor(np.concatenate([[initial_sample], np.asarray(y_in)[:-1]]).astype(np.int64))
    onehot = F.one_hot(y_prev, a).to(torch.float64)               # [T, a]: step t's input y_{t-1}
    E = t64["embed"]
    if E.dim() == 2:
        # the input convolution over a one-hot signal: one row of the embedding per step
        X = (onehot @ E + t64["b_embed"]).T                        # [r, T]
    else:
        # width-2 causal convolution over the one-hot inputs, zero before the first: tap 0 sees
        # step t's previous input y_{t-2}, tap 1 its input y_{t-1}
        kernel = torch.stack([E[0].T, E[1].T], dim=-1)             # [r, a, 2]
        X = F.conv1d(F.pad(onehot.T[None], (1, 0)), kernel, bias=t64["b_embed"])[0]
    hidden = []
    for j, d in enumerate(dilations):
        kernel = torch.stack([t64["w_prev"][j], t64["w_cur"][j]], dim=-1)   # [2r, r, 2]: tap 0 sees t-d
        Xp = F.pad(X[None], (int(d), 0))
        A = F.conv1d(Xp, kernel, bias=t64["b_gate"][j], dilation=int(d))[0] + cond[:, j, :].T
        H = tanh(A[:r]) * sigmoid(A[r:])
        hidden.append(H)
        X = X + F.conv1d(H[None], t64["w_res"][j][:, :, None], bias=t64["b_res"][j])[0]
    Hcat = torch.cat(hidden, dim=0)                                       # [l r, T]
    Wskip = torch.cat([t64["w_skip"][j] for j in range(L)], dim=1)        # [s, l r]
    Zs = torch.relu(Wskip @ Hcat + t64["b_skip"][:, None])
    Za = torch.relu(t64["w_relu"] @ Zs + t64["b_relu"][:, None])
    return (t64["w_out"] @ Za + t64["b_out"][:, None]).T.numpy()


def _fo_pool_closed_form(ht, f):
    """h_t = sum_{s<=t} (1 - f_s) h~_s prod_{s<u<=t} f_u for every t at once (fp64), [T, h]."""
    T = ht.shape[0]
    logf = torch.log(f)
    cl = torch.cumsum(logf, 0)                                   # [T, h]
    # prod_{s<u<=t} f_u = exp(cl_t - cl_s) for s <= t
    diff = cl[:, None, :] - cl[None, :, :]                       # [t, s, h]
    mask = torch.tril(torch.ones(T, T, dtype=torch.bool))[:, :, None]
    prod = torch.where(mask, torch.exp(torch.where(mask, diff, torch.zeros_like(diff))), torch.zeros_like(diff))
    return (prod * ((1.0 - f) * ht)[None]).sum(1)


def _qrnn_direction(x, w, b):
    """One direction over x [T, in] in its own order: z [T, h].  w [3h, 2, in], b [3h]."""
    T, cin = x.shape
    h = w.shape[0] // 3
    # width-2 causal convolution: tap 0 on the previous frame, tap 1 on the current one
    kern = torch.as_tensor(w, dtype=torch.float64).permute(0, 2, 1)       # [3h, in, 2]
    a = F.conv1d(F.pad(x.T[None], (1, 0)), kern, torch.as_tensor(b, dtype=torch.float64))[0].T  # [T, 3h]
    ht, o, f = torch.tanh(a[:, :h]), torch.sigmoid(a[:, h:2 * h]), torch.sigmoid(a[:, 2 * h:])
    return o * _fo_pool_closed_form(ht, f)


def condition(weights, features, n_audio, frame_rate, audio_rate):
    """The conditioning network written whole-sequence: torch conv1d gates, the fo-pool in closed
    form, the backward direction as the forward one on flipped frames, channels interleaved by
    stacking, upsampling by gathering frame floor(tau * frame_rate / audio_rate)."""
    x = torch.as_tensor(features, dtype=torch.float64)
    for wk, bk in (("w1", "b1"), ("w2", "b2")):
        w, b = weights[wk], weights[bk]
        fwd = _qrnn_direction(x, w[0], b[0])
        bwd = torch.flip(_qrnn_direction(torch.flip(x, [0]), w[1], b[1]), [0])
        x = torch.cat([fwd, bwd], 1)
    h2 = x.shape[1] // 2
    c = torch.stack([x[:, :h2], x[:, h2:]], 2).reshape(x.shape[0], 2 * h2)   # channel 2k + d
    idx = torch.arange(n_audio, dtype=torch.int64) * frame_rate // audio_rate
    return c[idx].numpy()
