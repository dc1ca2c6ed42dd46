"""Whole-sequence (non-incremental) WaveNet forward pass, used only to pin the oracle.

It evaluates the appendix's equations (Appendix A.1) over the entire teacher-forced
sequence at once, with torch's dilated conv1d (kernel width 2, zero left padding)
instead of per-step matrix-vector products and history buffers, and with the skip
projection applied to the concatenation of all layers' hidden states.  Float64, CPU.
"""
import numpy as np
import torch
import torch.nn.functional as F


def logits(w, dilations, cond, y_in, initial_sample=128):
    """w: dict of fp32 arrays; cond [T, l, 2r]; y_in [T] (step t consumes y_in[t-1]). Returns [T, a] float64."""
    t64 = {k: torch.tensor(np.asarray(v), dtype=torch.float64) for k, v in w.items()}
    L, two_r, r = t64["w_prev"].shape
    a = t64["w_out"].shape[0]
    cond = torch.tensor(np.asarray(cond), dtype=torch.float64)
    T = cond.shape[0]
    y_prev = torch.tensor(np.concatenate([[initial_sample], np.asarray(y_in)[:-1]]).astype(np.int64))
    onehot = F.one_hot(y_prev, a).to(torch.float64)               # [T, a]
    # the input convolution over a one-hot signal: one row of the embedding per step
    X = (onehot @ t64["embed"] + t64["b_embed"]).T                 # [r, T]
    hidden = []
    for j, d in enumerate(dilations):
        kernel = torch.stack([t64["w_prev"][j], t64["w_cur"][j]], dim=-1)   # [2r, r, 2]: tap 0 sees t-d
        Xp = F.pad(X[None], (int(d), 0))
        A = F.conv1d(Xp, kernel, bias=t64["b_gate"][j], dilation=int(d))[0] + cond[:, j, :].T
        H = torch.tanh(A[:r]) * torch.sigmoid(A[r:])
        hidden.append(H)
        X = X + F.conv1d(H[None], t64["w_res"][j][:, :, None], bias=t64["b_res"][j])[0]
    Hcat = torch.cat(hidden, dim=0)                                       # [l r, T]
    Wskip = torch.cat([t64["w_skip"][j] for j in range(L)], dim=1)        # [s, l r]
    Zs = torch.relu(Wskip @ Hcat + t64["b_skip"][:, None])
    Za = torch.relu(t64["w_relu"] @ Zs + t64["b_relu"][:, None])
    return (t64["w_out"] @ Za + t64["b_out"][:, None]).T.numpy()
