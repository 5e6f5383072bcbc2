"""Pins of the SDCC oracle (Section 5.1) to facts outside itself, and the
library's host-side leaf list and final-walk mask against it (CPU only).

Pins: the diverging leaves and both prefixes of the running example (Table
"running-prefixes"); the leaf rule against the paper's other construction of
the teacher context (Eq. "teacher-reconstruction" with every active span
re-inserted); the Bernoulli closed form of the KL and its asymmetry (a
reversed direction fails it); the uniform-teacher form; zero at equal or
shifted logits; Pinsker's bound (Proposition "pinsker-bound"); the gradient
against finite differences and autograd; and the lambda schedule of
Appendix F.
"""
import math

import numpy as np
import pytest
import torch

from oracle import sdcc as OS
from oracle import views as V
from paper_2609_00865_amd import mv, synth
from tests.fixtures import load, trajectory_from

F64 = torch.float64


# ---------------------------------------------------------------------------
# diverging leaves
# ---------------------------------------------------------------------------
def test_running_example_leaves_and_prefixes():
    fix = load("running_example.json")
    traj, pos = trajectory_from(fix)
    names = {i: n for n, i in pos.items()}
    leaves = OS.diverging_leaves(traj)
    want = [pos[e["leaf"]] for e in fix["leaves"] if e["diverges_by"]]
    assert [t for t, _, _ in leaves] == want
    live = V.views(traj)
    survivors = sorted(V.final_walk(traj))
    for e in fix["leaves"]:
        t = pos[e["leaf"]]
        # the table leaves out the prompt s
        lv = [names[j] for j in sorted(live[t - 1]) if j != pos["s"]]
        fw = [names[j] for j in survivors if j < t and j != pos["s"]]
        assert lv == e["live"] and fw == e["final"]
        assert sorted(set(lv) - set(fw)) == sorted(e["diverges_by"])
    assert leaves == [(6, 5, 4), (7, 6, 6), (9, 8, 7), (10, 9, 9), (12, 11, 10)]


@pytest.mark.parametrize("seed", range(30))
def test_leaves_match_teacher_reconstruction(seed):
    """View(t-1) equals the final-walk prefix with every span still active at t
    re-inserted at its slot, for every surviving token; the leaves are exactly
    the tokens where that re-insertion is non-empty."""
    rng = np.random.default_rng(500 + seed)
    lens = [int(x) for x in rng.integers(2, 120, size=int(rng.integers(1, 4)))]
    trajs = synth.random_trajectories(rng, lens, max_edits=6, max_span=20, summary_max=6)
    for tr in trajs:
        live = V.views(tr)
        survivors = set(V.final_walk(tr))
        leaves = {t: (a, b) for t, a, b in OS.diverging_leaves(tr)}
        for t in range(tr.begin + 1, tr.end):
            if t not in survivors:
                assert t not in leaves
                continue
            rec = OS.teacher_prefix(tr, t)
            assert rec == sorted(live[t - 1 - tr.begin])
            before = [j for j in survivors if j < t]
            if before and len(rec) > len(before):
                assert leaves[t] == (t - 1, max(before))
            else:
                assert t not in leaves


def test_leaf_with_empty_final_prefix_is_skipped():
    tr = synth.Trajectory(0, 8, (synth.Edit(4, ((0, 4),)),))
    assert OS.diverging_leaves(tr) == []
    m = mv.ViewMask([tr])
    assert m.stats()["n_leaves"] == 0
    assert all(x.numel() == 0 for x in m.leaves())


@pytest.mark.parametrize("seed", range(20))
def test_library_leaves_bit_exact(seed):
    rng = np.random.default_rng(900 + seed)
    lens = [int(x) for x in rng.integers(1, 400, size=int(rng.integers(1, 5)))]
    trajs = synth.random_trajectories(rng, lens, max_edits=8, max_span=40, summary_max=10)
    want = OS.packed_leaves(trajs)
    for kind in (mv.VIEW_LIVE, mv.VIEW_FINAL):
        m = mv.ViewMask(trajs, kind=kind)
        tok, tea, stu = m.leaves()
        got = list(zip(tok.tolist(), tea.tolist(), stu.tolist()))
        assert got == want
        assert m.stats()["n_leaves"] == len(want)


@pytest.mark.parametrize("seed", range(15))
def test_final_walk_mask_bits(seed):
    """The final-walk mask is the Naive-Compressed conditioning: row r sees the
    surviving keys before it and itself (Pitfall A, Section 3.3)."""
    rng = np.random.default_rng(1300 + seed)
    lens = [int(x) for x in rng.integers(1, 300, size=int(rng.integers(1, 4)))]
    trajs = synth.random_trajectories(rng, lens, max_edits=8, max_span=40, summary_max=10)
    T = trajs[-1].end
    m = mv.ViewMask(trajs, kind=mv.VIEW_FINAL)
    bits = mv.unpack_bits(m.materialize_host(0, T), T)
    want = torch.zeros(T, T, dtype=torch.bool)
    for tr in trajs:
        for r, vis in zip(range(tr.begin, tr.end), V.naive_views(tr, "compressed")):
            want[r, list(vis)] = True
    assert torch.equal(bits, want)
    st = m.stats()
    assert st["visible_pairs"] == int(want.sum())


def test_running_example_final_walk_death():
    traj, _ = trajectory_from(load("running_example.json"))
    m = mv.ViewMask([traj], kind=mv.VIEW_FINAL)
    assert m.death().tolist() == [14, 14, 14, 14, 14, 6, 14, 14, 9, 14, 14, 12, 14, 14]


# ---------------------------------------------------------------------------
# the KL and its gradient
# ---------------------------------------------------------------------------
def _bern_kl(a, b):
    return a * math.log(a / b) + (1 - a) * math.log((1 - a) / (1 - b))


def test_bernoulli_closed_form_and_direction():
    # vocab {0, 1}, one hidden feature: logits (0, x), p_1 = sigmoid(x)
    W = torch.tensor([[0.0], [1.0]], dtype=F64)
    xt, xs = torch.tensor([[1.3], [-0.4]], dtype=F64), torch.tensor([[-0.7], [2.1]], dtype=F64)
    kl, lT, lS = OS.junction_kl(xt, xs, W)
    for i in range(2):
        a = 1 / (1 + math.exp(-float(xt[i, 0])))
        b = 1 / (1 + math.exp(-float(xs[i, 0])))
        assert abs(float(kl[i]) - _bern_kl(a, b)) < 1e-12
        assert abs(float(kl[i]) - _bern_kl(b, a)) > 1e-3   # forward, not reverse
        assert abs(float(lT[i]) - math.log(1 + math.exp(float(xt[i, 0])))) < 1e-12


def test_uniform_teacher():
    gen = torch.Generator().manual_seed(1)
    W = torch.randn(50, 16, generator=gen, dtype=F64)
    hs = torch.randn(3, 16, generator=gen, dtype=F64)
    kl, _, _ = OS.junction_kl(torch.zeros(3, 16, dtype=F64), hs, W)
    logq = torch.log_softmax(hs @ W.T, dim=1)
    want = -math.log(50) - logq.mean(dim=1)
    assert torch.allclose(kl, want, atol=1e-12)


def test_zero_at_equal_and_shifted_logits():
    gen = torch.Generator().manual_seed(2)
    W = torch.randn(40, 8, generator=gen, dtype=F64)
    W[:, 0] = 1.0                      # a feature every logit shares
    h = torch.randn(5, 8, generator=gen, dtype=F64)
    kl, _, _ = OS.junction_kl(h, h, W)
    assert kl.abs().max() < 1e-13
    hs = h.clone()
    hs[:, 0] += 3.7                    # shifts every student logit by 3.7
    kl, lT, lS = OS.junction_kl(h, hs, W)
    assert kl.abs().max() < 1e-12
    assert torch.allclose(lS - lT, torch.full_like(lT, 3.7), atol=1e-12)


@pytest.mark.parametrize("seed", range(5))
def test_nonnegative_and_pinsker(seed):
    gen = torch.Generator().manual_seed(10 + seed)
    W = torch.randn(300, 32, generator=gen, dtype=F64) * 0.3
    ht = torch.randn(64, 32, generator=gen, dtype=F64)
    hs = ht + (0.1 + seed) * torch.randn(64, 32, generator=gen, dtype=F64)
    kl, _, _ = OS.junction_kl(ht, hs, W)
    tv = OS.total_variation(ht, hs, W)
    assert (kl >= 0).all()
    assert (tv <= torch.sqrt(kl / 2) + 1e-12).all()


def test_gradient_finite_differences_and_autograd():
    gen = torch.Generator().manual_seed(3)
    W = torch.randn(30, 6, generator=gen, dtype=F64)
    ht = torch.randn(4, 6, generator=gen, dtype=F64)
    hs = torch.randn(4, 6, generator=gen, dtype=F64)
    dkl = torch.tensor([1.0, -0.5, 2.0, 0.0], dtype=F64)
    g = OS.junction_kl_grad(ht, hs, W, dkl)
    eps = 1e-6
    for i in range(4):
        for k in range(6):
            hp, hm = hs.clone(), hs.clone()
            hp[i, k] += eps
            hm[i, k] -= eps
            fd = (OS.junction_kl(ht, hp, W)[0] - OS.junction_kl(ht, hm, W)[0]) @ dkl / (2 * eps)
            assert abs(float(fd) - float(g[i, k])) < 1e-7
    x = hs.clone().requires_grad_(True)
    logp = torch.log_softmax(ht @ W.T, dim=1)
    loss = (torch.nn.functional.kl_div(torch.log_softmax(x @ W.T, dim=1), logp,
                                       log_target=True, reduction="none").sum(dim=1) * dkl).sum()
    loss.backward()
    assert torch.allclose(x.grad, g, atol=1e-12)


def test_lambda_schedule():
    # Appendix F: linear from 0 to 0.1 over the first 20% of updates, then flat
    assert OS.kl_weight(0, 1000) == 0.0
    assert abs(OS.kl_weight(100, 1000) - 0.05) < 1e-12
    assert OS.kl_weight(200, 1000) == 0.1
    assert OS.kl_weight(999, 1000) == 0.1
    for step in [0, 1, 7, 100, 199, 200, 201, 1000, 5000]:
        for total in [1, 10, 1000]:
            assert abs(mv.sdcc_lambda(step, total) - OS.kl_weight(step, total)) < 1e-6
    assert mv.sdcc_lambda(5, 10, 0.1, 0.0) == pytest.approx(0.1)


@pytest.mark.parametrize("seed", range(15))
def test_library_leaves_and_final_walk_with_restores(seed):
    """With keys that leave and re-enter (offload / retrieve), a surviving
    token diverges when its live prefix and its final-walk prefix differ in
    either direction; the final-walk mask keeps exactly the final walk."""
    rng = np.random.default_rng(2600 + seed)
    lens = [int(x) for x in rng.integers(2, 300, size=int(rng.integers(1, 4)))]
    trajs = synth.random_trajectories(rng, lens, max_edits=10, max_span=40, summary_max=8,
                                      restore_max=30)
    want = OS.packed_leaves(trajs)
    m = mv.ViewMask(trajs, kind=mv.VIEW_FINAL)
    tok, tea, stu = m.leaves()
    assert list(zip(tok.tolist(), tea.tolist(), stu.tolist())) == want
    T = trajs[-1].end
    bits = mv.unpack_bits(m.materialize_host(0, T), T)
    ref = torch.zeros(T, T, dtype=torch.bool)
    for tr in trajs:
        for r, vis in zip(range(tr.begin, tr.end), V.naive_views(tr, "compressed")):
            ref[r, list(vis)] = True
    assert torch.equal(bits, ref)

