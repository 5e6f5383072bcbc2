"""GRPO token loss and the drift diagnostics on the scored tokens (test
infrastructure only).

The training recipe (Appendix F) is GRPO with the asymmetric clip pair
(0.2 low, 0.28 high), a KL penalty of weight beta against a reference policy
taken with the low-variance estimator, and advantages normalised within each
group of samples of one prompt.  The conditioning proofs (Propositions
"rl_tree" and "rl_4d") need the ratio, the advantage weight and the KL term
of token y_t all to be computed from logits under its live view: here they
are functions of the per-token log-probs that the view-masked forward and the
fused LM head produce.

Readings where the paper names a method without its formula:
  * advantage A_i = (r_i - mean_g r) / (std_g r + adv_eps), std the sample
    (n-1) standard deviation of the group, 0 for groups of one;
  * surrogate per loss token: min(rho A, clip(rho, 1-eps_low, 1+eps_high) A),
    rho = exp(logp - logp_old), logp_old the rollout log-prob;
  * KL estimator k3 = exp(ref - logp) - (ref - logp) - 1;
  * loss = mean over the loss tokens of (-surrogate + beta k3) (token mean
    over the whole batch).
Diagnostics: logdiff (Eq. "logdiff", the mean |logp - logp_old| over the loss
tokens), the fractions of loss tokens whose clipped term is the active one
(gradient zero) on the low and the high side, the mean k3, the mean ratio.

All arithmetic in fp64 unless the caller passes another dtype.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import torch


def group_advantages(reward, group_size: int, adv_eps: float = 1e-6, dtype=torch.float64):
    r = reward.to(dtype).reshape(-1, group_size)
    mean = r.mean(dim=1, keepdim=True)
    if group_size > 1:
        std = r.std(dim=1, unbiased=True, keepdim=True)
    else:
        std = torch.zeros_like(mean)
    return ((r - mean) / (std + adv_eps)).reshape(-1)


def token_trajectory(traj_ptr: Sequence[int], n_tokens: int) -> torch.Tensor:
    """Index of the trajectory each packed token belongs to."""
    out = torch.empty(n_tokens, dtype=torch.long)
    ptr = [int(x) for x in traj_ptr]
    for i in range(len(ptr) - 1):
        out[ptr[i]:ptr[i + 1]] = i
    return out


def grpo_loss(traj_ptr, reward, logp, logp_old, logp_ref: Optional[torch.Tensor],
              loss_mask: Optional[torch.Tensor], group_size: int, eps_low: float,
              eps_high: float, beta: float, adv_eps: float = 1e-6,
              dtype=torch.float64) -> Dict[str, torch.Tensor]:
    """Returns advantage, dlogp (d loss / d logp per token), and the statistics."""
    T = logp.numel()
    adv = group_advantages(reward, group_size, adv_eps, dtype)
    A = adv[token_trajectory(traj_ptr, T)]
    lp = logp.to(dtype)
    old = logp_old.to(dtype)
    m = torch.ones(T, dtype=torch.bool) if loss_mask is None else loss_mask.bool()
    n = int(m.sum())
    rho = torch.exp(lp - old)
    lo, hi = 1.0 - eps_low, 1.0 + eps_high
    clipped = torch.clamp(rho, lo, hi)
    unclip_term, clip_term = rho * A, clipped * A
    surrogate = torch.minimum(unclip_term, clip_term)
    # the clipped term is the active one where it is strictly smaller
    clip_active = clip_term < unclip_term
    d_surr = torch.where(clip_active, torch.zeros_like(rho), A * rho)
    if logp_ref is not None and beta != 0.0:
        x = logp_ref.to(dtype) - lp
        k3 = torch.exp(x) - x - 1.0
        d_k3 = 1.0 - torch.exp(x)
    else:
        k3 = torch.zeros_like(lp)
        d_k3 = torch.zeros_like(lp)
    per_tok = -surrogate + beta * k3
    inv = 1.0 / n if n else 0.0
    dlogp = torch.where(m, (-d_surr + beta * d_k3) * inv, torch.zeros_like(lp))
    mf = m.to(dtype)
    stats = {
        "loss": (per_tok * mf).sum() * inv,
        "logdiff": ((lp - old).abs() * mf).sum() * inv,
        "clip_frac_low": ((clip_active & (rho < lo)) & m).to(dtype).sum() * inv,
        "clip_frac_high": ((clip_active & (rho > hi)) & m).to(dtype).sum() * inv,
        "kl_ref": (k3 * mf).sum() * inv,
        "ratio_mean": (rho * mf).sum() * inv,
        "n_loss_tokens": torch.tensor(float(n), dtype=dtype),
        "adv_abs_mean": adv.abs().mean(),
    }
    return {"advantage": adv, "dlogp": dlogp, "stats": stats, "ratio": rho,
            "clip_active": clip_active}


def logdiff(logp_train, logp_rollout, loss_mask=None):
    """Eq. "logdiff" alone (the drift of the recomputed log-probs)."""
    d = (logp_train.to(torch.float64) - logp_rollout.to(torch.float64)).abs()
    if loss_mask is not None:
        d = d[loss_mask.bool()]
    return d.mean()
