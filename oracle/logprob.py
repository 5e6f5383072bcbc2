"""Per-token log-prob, importance ratio and clip (test infrastructure only).

For each scored token t with hidden state h_t and target id y_t:

    z_t      = W h_t                       (logits over the vocabulary)
    lse_t    = log sum_v exp(z_tv)
    logp_t   = z_{t, y_t} - lse_t          (log-softmax at the target)
    ratio_t  = exp(logp_t - logp_old_t)    (importance ratio of the GRPO loss)
    clipped_t = min(max(ratio_t, 1 - eps_low), 1 + eps_high)

The ratio must be formed under the live view the token was decoded from
(Appendix C, "Pitfall A, RL view"; Proposition "rl_4d"); the asymmetric clip
pair comes from the training hyper-parameters of Appendix F.  A target of -1
marks a token that carries no loss (Section 4.1, per-branch loss mask): logp 0,
ratio 1, clipped 1, zero gradient.

Gradient into the hidden state for upstream g_t = dL/dlogp_t:

    dH_t = g_t * (W[y_t] - sum_v softmax(z_t)_v W[v])

which is the textbook derivative of log-softmax at one index; into the
weights, dW = G^T H with G_tv = g_t (1[v = y_t] - softmax(z_t)_v).
"""
from __future__ import annotations

from typing import Optional

import torch


def token_logprob(hidden, weight, target, logp_old: Optional[torch.Tensor] = None,
                  eps_low: float = 0.2, eps_high: float = 0.2,
                  dtype=torch.float64, chunk: int = 256):
    """Returns (logp, ratio, clipped, lse); ratio/clipped are None without logp_old."""
    T = hidden.shape[0]
    W = weight.to(dtype)
    logp = torch.zeros(T, dtype=dtype)
    lse = torch.zeros(T, dtype=dtype)
    tgt = target.to(torch.long)
    for c0 in range(0, T, chunk):
        c1 = min(T, c0 + chunk)
        z = hidden[c0:c1].to(dtype) @ W.T
        l = torch.logsumexp(z, dim=1)
        lse[c0:c1] = l
        y = tgt[c0:c1]
        ok = y >= 0
        zy = torch.where(ok, z.gather(1, y.clamp(min=0)[:, None])[:, 0], l)
        logp[c0:c1] = torch.where(ok, zy - l, torch.zeros_like(l))
    if logp_old is None:
        return logp, None, None, lse
    ratio = torch.exp(logp - logp_old.to(dtype))
    ratio = torch.where(tgt >= 0, ratio, torch.ones_like(ratio))
    clipped = torch.clamp(ratio, 1.0 - eps_low, 1.0 + eps_high)
    return logp, ratio, clipped, lse


def token_logprob_bwd(hidden, weight, target, dlogp, dtype=torch.float64, chunk: int = 256):
    """dH = g * (W[y] - softmax(z) W), zero for target -1 rows."""
    T, H = hidden.shape
    W = weight.to(dtype)
    out = torch.zeros(T, H, dtype=dtype)
    tgt = target.to(torch.long)
    for c0 in range(0, T, chunk):
        c1 = min(T, c0 + chunk)
        z = hidden[c0:c1].to(dtype) @ W.T
        p = torch.softmax(z, dim=1)
        y = tgt[c0:c1]
        ok = (y >= 0).to(dtype)
        g = dlogp[c0:c1].to(dtype) * ok
        out[c0:c1] = g[:, None] * (W[y.clamp(min=0)] - p @ W)
    return out


def token_logprob_dweight(hidden, weight, target, dlogp, dtype=torch.float64, chunk: int = 256):
    """Gradient into the LM-head weights: dW = G^T H with G = g (onehot - softmax(z)),
    i.e. dW[v] = sum_t g_t (1[v = y_t] - p_tv) h_t (zero contribution from target -1)."""
    T, H = hidden.shape
    W = weight.to(dtype)
    out = torch.zeros(W.shape, dtype=dtype)
    tgt = target.to(torch.long)
    for c0 in range(0, T, chunk):
        c1 = min(T, c0 + chunk)
        h = hidden[c0:c1].to(dtype)
        p = torch.softmax(h @ W.T, dim=1)
        y = tgt[c0:c1]
        ok = (y >= 0).to(dtype)
        g = dlogp[c0:c1].to(dtype) * ok
        G = -g[:, None] * p
        G[torch.arange(c1 - c0), y.clamp(min=0)] += g
        out += G.T @ h
    return out


def ppo_clip_dlogp(ratio, adv, eps_low: float, eps_high: float, scale: float = 1.0):
    """d/dlogp of  -scale * min(ratio * A, clip(ratio) * A)  per token.

    The min picks the unclipped term unless clipping makes the objective
    smaller; where the clipped term is active its derivative is zero.
    """
    r = ratio.to(torch.float64)
    a = adv.to(torch.float64)
    unclipped = r * a
    clipped = torch.clamp(r, 1.0 - eps_low, 1.0 + eps_high) * a
    active = unclipped <= clipped
    return torch.where(active, -scale * r * a, torch.zeros_like(r))
