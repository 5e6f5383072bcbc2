"""Pins for the log-prob oracle: closed forms, special cases, finite
differences and the clip edges."""
import math

import pytest
import torch

from oracle import logprob as LP

F64 = torch.float64


def _rand(T, H, Vv, seed):
    g = torch.Generator().manual_seed(seed)
    h = torch.randn(T, H, generator=g, dtype=F64)
    w = 0.3 * torch.randn(Vv, H, generator=g, dtype=F64)
    y = torch.randint(0, Vv, (T,), generator=g, dtype=torch.int32)
    return h, w, y


def test_equal_rows_give_uniform():
    h, w, y = _rand(5, 6, 11, 0)
    w[:] = w[0]
    logp, _, _, lse = LP.token_logprob(h, w, y)
    assert torch.allclose(logp, torch.full_like(logp, -math.log(11)), atol=1e-13)
    dh = LP.token_logprob_bwd(h, w, y, torch.ones(5, dtype=F64))
    assert dh.abs().max() < 1e-13


def test_zero_hidden_gives_uniform():
    h, w, y = _rand(4, 6, 9, 1)
    logp, _, _, lse = LP.token_logprob(torch.zeros_like(h), w, y)
    assert torch.allclose(logp, torch.full_like(logp, -math.log(9)), atol=1e-13)
    assert torch.allclose(lse, torch.full_like(lse, math.log(9)), atol=1e-13)


def test_two_word_vocab_is_log_sigmoid():
    h, w, y = _rand(7, 5, 2, 2)
    logp, _, _, _ = LP.token_logprob(h, w, y)
    z = h @ w.T
    other = 1 - y.long()
    margin = z.gather(1, y.long()[:, None])[:, 0] - z.gather(1, other[:, None])[:, 0]
    expect = torch.tensor([-math.log1p(math.exp(-float(m))) for m in margin], dtype=F64)
    assert torch.allclose(logp, expect, atol=1e-13)


def test_probabilities_sum_to_one():
    h, w, y = _rand(6, 8, 13, 3)
    _, _, _, lse = LP.token_logprob(h, w, y)
    tot = torch.zeros(6, dtype=F64)
    for v in range(13):
        yy = torch.full((6,), v, dtype=torch.int32)
        lp, _, _, _ = LP.token_logprob(h, w, yy)
        tot += lp.exp()
    assert torch.allclose(tot, torch.ones(6, dtype=F64), atol=1e-13)


def test_ratio_and_clip_edges():
    h, w, y = _rand(6, 8, 13, 4)
    logp, _, _, _ = LP.token_logprob(h, w, y)
    shifts = torch.tensor([0.0, math.log(1.2), math.log(0.8), math.log(1.5), math.log(0.5), 0.1],
                          dtype=F64)
    old = logp - shifts
    _, ratio, clipped, _ = LP.token_logprob(h, w, y, old, 0.2, 0.28)
    assert torch.allclose(ratio, shifts.exp(), atol=1e-13)
    expect = torch.tensor([1.0, 1.2, 0.8, 1.28, 0.8, math.exp(0.1)], dtype=F64)
    assert torch.allclose(clipped, expect, atol=1e-13)


def test_skipped_tokens():
    h, w, y = _rand(5, 4, 7, 5)
    y[2] = -1
    old = torch.full((5,), -1.0, dtype=F64)
    logp, ratio, clipped, lse = LP.token_logprob(h, w, y, old)
    assert logp[2] == 0 and ratio[2] == 1 and clipped[2] == 1
    dh = LP.token_logprob_bwd(h, w, y, torch.ones(5, dtype=F64))
    assert torch.all(dh[2] == 0) and dh[1].abs().max() > 0


def test_finite_differences():
    h, w, y = _rand(3, 5, 7, 6)
    g = torch.tensor([0.7, -1.3, 2.0], dtype=F64)
    dh = LP.token_logprob_bwd(h, w, y, g)
    eps = 1e-6
    for t in range(3):
        for i in range(5):
            hp, hm = h.clone(), h.clone()
            hp[t, i] += eps
            hm[t, i] -= eps
            fp = float((LP.token_logprob(hp, w, y)[0] * g).sum())
            fm = float((LP.token_logprob(hm, w, y)[0] * g).sum())
            assert abs((fp - fm) / (2 * eps) - float(dh[t, i])) < 1e-8


def test_chunking_is_invisible():
    h, w, y = _rand(11, 6, 9, 7)
    a = LP.token_logprob(h, w, y, chunk=256)
    b = LP.token_logprob(h, w, y, chunk=3)
    assert torch.allclose(a[0], b[0], atol=1e-14) and torch.allclose(a[3], b[3], atol=1e-14)


@pytest.mark.parametrize("adv", [1.5, -0.7])
def test_ppo_clip_gradient_matches_finite_difference(adv):
    eps_lo, eps_hi = 0.2, 0.28
    logr = torch.tensor([-0.5, -0.1, 0.0, 0.1, 0.4], dtype=F64)
    a = torch.full((5,), adv, dtype=F64)
    g = LP.ppo_clip_dlogp(logr.exp(), a, eps_lo, eps_hi)

    def obj(lr):
        r = lr.exp()
        return -torch.minimum(r * a, r.clamp(1 - eps_lo, 1 + eps_hi) * a)
    d = 1e-7
    fd = (obj(logr + d) - obj(logr - d)) / (2 * d)
    assert torch.allclose(g, fd, atol=1e-6)


def test_weight_gradient_finite_differences_and_autograd():
    """dW = G^T H against central differences of sum_t g_t logp_t in W, against
    autograd, and its invariant: the vocabulary rows of G sum to zero, so the
    rows of dW do too."""
    gen = torch.Generator().manual_seed(21)
    T, H, V = 7, 5, 11
    h = torch.randn(T, H, generator=gen, dtype=F64)
    w = torch.randn(V, H, generator=gen, dtype=F64)
    y = torch.randint(0, V, (T,), generator=gen)
    y[3] = -1
    g = torch.randn(T, generator=gen, dtype=F64)
    dW = LP.token_logprob_dweight(h, w, y, g)
    assert torch.allclose(dW.sum(dim=0), torch.zeros(H, dtype=F64), atol=1e-12)
    def f(wm):
        lp, _, _, _ = LP.token_logprob(h, wm, y)
        return float((lp * g).sum())
    eps = 1e-6
    for v in range(V):
        for k in range(H):
            wp, wm = w.clone(), w.clone()
            wp[v, k] += eps
            wm[v, k] -= eps
            assert abs((f(wp) - f(wm)) / (2 * eps) - float(dW[v, k])) < 1e-7
    wa = w.clone().requires_grad_(True)
    lp = torch.log_softmax(h @ wa.T, dim=1).gather(1, y.clamp(min=0)[:, None])[:, 0]
    ((lp * (y >= 0)) * g).sum().backward()
    assert torch.allclose(wa.grad, dW, atol=1e-12)
