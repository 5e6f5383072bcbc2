"""Pins of the GRPO loss / drift-diagnostics oracle (CPU only): closed-form
group advantages, the four clip quadrants by hand, the k3 estimator's value
and zero set, token-mean weighting, the loss mask, and the gradient against
finite differences away from the clip edges."""
import math

import pytest
import torch

from oracle import grpo as OG

F64 = torch.float64


def test_group_advantage_closed_form():
    r = torch.tensor([1.0, 0.0, 0.0, 0.0, 2.0, 2.0, 2.0, 2.0], dtype=F64)
    a = OG.group_advantages(r, 4, adv_eps=0.0 + 1e-12)
    # mean 0.25, unbiased std 0.5 -> (0.75, -0.25) / 0.5
    assert torch.allclose(a[:4], torch.tensor([1.5, -0.5, -0.5, -0.5], dtype=F64), atol=1e-9)
    assert torch.all(a[4:] == 0)     # equal rewards: no signal
    assert OG.group_advantages(torch.tensor([3.0, 5.0]), 1).abs().max() == 0


def _single(rho, A, eps_low=0.2, eps_high=0.28, beta=0.0, ref_minus_lp=None):
    lp = torch.tensor([-1.0], dtype=F64)
    old = lp - math.log(rho)
    ref = None if ref_minus_lp is None else lp + ref_minus_lp
    # one scored token in trajectory 0; trajectory 1 (empty) completes a group of two,
    # so the token's advantage is sign(A) / sqrt(2)
    out = OG.grpo_loss([0, 1, 1], torch.tensor([A, -A], dtype=F64), lp, old, ref, None, 2,
                       eps_low, eps_high, beta, adv_eps=0.0)
    return out


@pytest.mark.parametrize("rho,A_sign,active", [
    (1.5, +1, True),    # A > 0, ratio above 1+eps_high: clipped term smaller -> no gradient
    (0.5, +1, False),   # A > 0, ratio below 1-eps_low: unclipped is the min
    (0.5, -1, True),    # A < 0, ratio below 1-eps_low: clipped term smaller
    (1.5, -1, False),   # A < 0, ratio above 1+eps_high: unclipped is the min
    (1.1, +1, False),   # inside the range: both equal, gradient flows
])
def test_clip_quadrants(rho, A_sign, active):
    out = _single(rho, float(A_sign))
    A = float(out["advantage"][0])
    assert (A > 0) == (A_sign > 0)
    assert bool(out["clip_active"][0]) == active
    want = 0.0 if active else -A * rho
    assert abs(float(out["dlogp"][0]) - want) < 1e-12
    clipped = min(max(rho, 0.8), 1.28)
    assert abs(float(out["stats"]["loss"]) + min(rho * A, clipped * A)) < 1e-12


def test_k3_value_and_zero():
    out = _single(1.0, 1.0, beta=0.5, ref_minus_lp=0.5)
    k3 = math.exp(0.5) - 0.5 - 1.0
    assert abs(float(out["stats"]["kl_ref"]) - k3) < 1e-12
    A = float(out["advantage"][0])
    assert abs(float(out["stats"]["loss"]) - (-A + 0.5 * k3)) < 1e-12
    zero = _single(1.0, 1.0, beta=0.5, ref_minus_lp=0.0)
    assert float(zero["stats"]["kl_ref"]) == 0.0


def test_token_mean_and_mask():
    # two trajectories of lengths 3 and 1 in one group; ratio 1 everywhere
    ptr = [0, 3, 4]
    r = torch.tensor([1.0, 0.0], dtype=F64)
    lp = torch.tensor([-1.0, -2.0, -0.5, -3.0], dtype=F64)
    out = OG.grpo_loss(ptr, r, lp, lp, None, None, 2, 0.2, 0.28, 0.0, adv_eps=0.0)
    A = out["advantage"]
    assert torch.allclose(A, torch.tensor([1 / math.sqrt(0.5) * 0.5, -1 / math.sqrt(0.5) * 0.5],
                                          dtype=F64))
    # token mean: (3 A0 + A1) / 4 with a minus sign
    assert abs(float(out["stats"]["loss"]) + (3 * A[0] + A[1]) / 4) < 1e-12
    assert torch.allclose(out["dlogp"], -A[[0, 0, 0, 1]] / 4)
    assert float(out["stats"]["logdiff"]) == 0.0
    mask = torch.tensor([1, 0, 1, 0], dtype=torch.uint8)
    om = OG.grpo_loss(ptr, r, lp, lp, None, mask, 2, 0.2, 0.28, 0.0, adv_eps=0.0)
    assert float(om["stats"]["n_loss_tokens"]) == 2
    assert om["dlogp"][1] == 0 and om["dlogp"][3] == 0
    assert abs(float(om["dlogp"][0]) + float(A[0]) / 2) < 1e-12


def test_logdiff_known_values():
    a = torch.tensor([-1.0, -2.0, -0.5])
    b = torch.tensor([-2.0, 0.0, -0.5])
    assert abs(float(OG.logdiff(a, b)) - 1.0) < 1e-12
    assert abs(float(OG.logdiff(a, b, torch.tensor([1, 1, 0]))) - 1.5) < 1e-12


def test_gradient_finite_differences():
    gen = torch.Generator().manual_seed(4)
    T, G = 40, 4
    ptr = [0, 7, 15, 21, 30, 33, 40, 40, 40]     # includes empty trajectories
    r = torch.randn(8, generator=gen, dtype=F64)
    lp = -2.0 + torch.randn(T, generator=gen, dtype=F64)
    old = lp + 0.3 * torch.randn(T, generator=gen, dtype=F64)
    ref = lp + 0.2 * torch.randn(T, generator=gen, dtype=F64)
    mask = (torch.rand(T, generator=gen) < 0.8).to(torch.uint8)
    args = dict(group_size=G, eps_low=0.2, eps_high=0.28, beta=0.05)
    out = OG.grpo_loss(ptr, r, lp, old, ref, mask, **args)
    rho = out["ratio"]
    h = 1e-7
    for t in range(T):
        if min(abs(rho[t] - 0.8), abs(rho[t] - 1.28)) < 1e-4:
            continue
        p, m = lp.clone(), lp.clone()
        p[t] += h
        m[t] -= h
        fd = (OG.grpo_loss(ptr, r, p, old, ref, mask, **args)["stats"]["loss"] -
              OG.grpo_loss(ptr, r, m, old, ref, mask, **args)["stats"]["loss"]) / (2 * h)
        assert abs(float(fd) - float(out["dlogp"][t])) < 1e-7
