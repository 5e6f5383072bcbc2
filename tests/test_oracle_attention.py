"""Pins for the attention oracle: plain causal attention when nothing is
compressed (a library routine), brute force per row, the dense union form,
finite differences, and the two invariants of the conditioning rule."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import views as V
from paper_2609_00865_amd import synth

F64 = torch.float64


def _rand(T, hq, hkv, d, seed):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(T, hq, d, generator=g, dtype=F64)
    k = torch.randn(T, hkv, d, generator=g, dtype=F64)
    v = torch.randn(T, hkv, d, generator=g, dtype=F64)
    do = torch.randn(T, hq, d, generator=g, dtype=F64)
    return q, k, v, do


def _random_trajs(seed, lengths, **kw):
    return synth.random_trajectories(np.random.default_rng(seed), lengths, **kw)


@pytest.mark.parametrize("hq,hkv", [(1, 1), (4, 2), (6, 1)])
def test_no_compression_is_causal_sdpa(hq, hkv):
    """K = 0: every view is the physical prefix, i.e. plain causal attention."""
    T, d = 37, 16
    q, k, v, do = _rand(T, hq, hkv, d, 1)
    traj = [synth.Trajectory(0, T, ())]
    O, L, dq, dk, dv = A.logittree(traj, q, k, v, dout=do)
    qr = q.clone().requires_grad_(True)
    kr = k.clone().requires_grad_(True)
    vr = v.clone().requires_grad_(True)
    G = hq // hkv
    o = torch.nn.functional.scaled_dot_product_attention(
        qr.transpose(0, 1), kr.repeat_interleave(G, 1).transpose(0, 1),
        vr.repeat_interleave(G, 1).transpose(0, 1), is_causal=True).transpose(0, 1)
    (o * do).sum().backward()
    assert torch.allclose(O, o.detach(), atol=1e-12, rtol=0)
    assert torch.allclose(dq, qr.grad, atol=1e-11, rtol=0)
    assert torch.allclose(dk, kr.grad, atol=1e-11, rtol=0)
    assert torch.allclose(dv, vr.grad, atol=1e-11, rtol=0)
    # LSE against the definition
    s = torch.einsum("ihd,jhd->hij", q, k.repeat_interleave(G, 1)) / math.sqrt(d)
    s = s.masked_fill(torch.ones(T, T, dtype=torch.bool).triu(1)[None], float("-inf"))
    assert torch.allclose(L, torch.logsumexp(s, -1), atol=1e-12, rtol=0)


def _brute_rows(trajs, q, k, v):
    """Per row, a Python loop over the keys the definition lets it see."""
    T, hq, d = q.shape
    G = hq // k.shape[1]
    O = np.zeros((T, hq, d))
    L = np.zeros((hq, T))
    qn, kn, vn = q.numpy(), k.numpy(), v.numpy()
    for t in trajs:
        for r in range(t.begin, t.end):
            vis = sorted(V.view_by_definition(t, r))
            for h in range(hq):
                s = [float(np.dot(qn[r, h], kn[j, h // G])) / math.sqrt(d) for j in vis]
                m = max(s)
                w = [math.exp(x - m) for x in s]
                z = sum(w)
                L[h, r] = m + math.log(z)
                O[r, h] = sum(wi / z * vn[j, h // G] for wi, j in zip(w, vis))
    return torch.from_numpy(O), torch.from_numpy(L)


@pytest.mark.parametrize("seed", range(4))
def test_brute_force_rows(seed):
    trajs = _random_trajs(seed, [23, 17, 20], max_edits=4, max_span=5)
    T = trajs[-1].end
    q, k, v, _ = _rand(T, 4, 2, 8, seed)
    O, L = A.logittree(trajs, q, k, v)
    Ob, Lb = _brute_rows(trajs, q, k, v)
    assert torch.allclose(O, Ob, atol=1e-12, rtol=0)
    assert torch.allclose(L, Lb, atol=1e-12, rtol=0)
    Od, Ld = A.dense(trajs, q, k, v)
    assert torch.allclose(Od, Ob, atol=1e-12, rtol=0)
    rows = [0, 5, T - 1, trajs[1].begin + 3]
    Or, Lr = A.rows(trajs, q, k, v, rows)
    assert torch.allclose(Or, Ob[rows], atol=1e-12, rtol=0)
    assert torch.allclose(Lr, Lb[:, rows], atol=1e-12, rtol=0)


@pytest.mark.parametrize("seed", range(3))
def test_logittree_equals_dense_union(seed):
    """Materialisation equivalence (Section 4.3): same outputs and gradients."""
    trajs = _random_trajs(100 + seed, [60, 45], max_edits=5, max_span=12)
    T = trajs[-1].end
    q, k, v, do = _rand(T, 4, 1, 16, seed)
    a = A.logittree(trajs, q, k, v, dout=do)
    b = A.dense(trajs, q, k, v, dout=do)
    for x, y in zip(a, b):
        assert torch.allclose(x, y, atol=1e-12, rtol=0)


@pytest.mark.parametrize("seed", range(4))
def test_logittree_equals_dense_union_with_restores(seed):
    """Keys that leave and re-enter: the per-branch forwards and the masked
    union still agree (each row attends exactly to its view)."""
    trajs = _random_trajs(60 + seed, [90, 70], max_edits=6, max_span=15, restore_max=10)
    T = trajs[-1].end
    q, k, v, do = _rand(T, 2, 1, 8, seed)
    a = A.logittree(trajs, q, k, v, dout=do)
    b = A.dense(trajs, q, k, v, dout=do)
    for x, y in zip(a, b):
        assert torch.allclose(x, y, atol=1e-12, rtol=0)


def test_logittree_row_chunking_and_heads():
    trajs = synth.make_trajectories("tiny", 1)
    q, k, v, do = _rand(512, 2, 1, 8, 5)
    full = A.logittree(trajs, q, k, v, dout=do)
    chunk = A.logittree(trajs, q, k, v, dout=do, row_chunk=37)
    for x, y in zip(full, chunk):
        assert torch.allclose(x, y, atol=1e-12, rtol=0)
    one = A.logittree(trajs, q, k, v, heads=[1])
    assert torch.allclose(one[0][:, 1], full[0][:, 1], atol=1e-13, rtol=0)
    assert torch.all(one[0][:, 0] == 0)


def test_finite_differences():
    trajs = _random_trajs(7, [14, 10], max_edits=3, max_span=4)
    T = trajs[-1].end
    q, k, v, do = _rand(T, 2, 1, 4, 3)
    _, _, dq, dk, dv = A.logittree(trajs, q, k, v, dout=do)

    def f(qq, kk, vv):
        return float((A.logittree(trajs, qq, kk, vv)[0] * do).sum())

    h = 1e-6
    for grad, which in ((dq, 0), (dk, 1), (dv, 2)):
        args = [q, k, v]
        base = args[which]
        for idx in [(0, 0, 0), (3, 1 % base.shape[1], 2), (T - 1, 0, 3), (9, 0, 1), (15, 0, 0)]:
            p = [a.clone() for a in args]
            m = [a.clone() for a in args]
            p[which][idx] += h
            m[which][idx] -= h
            fd = (f(*p) - f(*m)) / (2 * h)
            assert abs(fd - float(grad[idx])) < 1e-7, (which, idx)


def test_eviction_invariance():
    """Rows at or after J_k are blind to E_k; rows before it are not."""
    t = synth.make_trajectories("tiny", 0)[0]
    q, k, v, do = _rand(512, 1, 1, 8, 9)
    O, _ = A.logittree([t], q, k, v)
    ed = t.edits[0]
    ev = [p for b, e in ed.evict for p in range(b, e)]
    k2, v2 = k.clone(), v.clone()
    k2[ev] += torch.randn(len(ev), 1, 8, dtype=F64)
    v2[ev] += 3.0
    O2, _ = A.logittree([t], q, k2, v2)
    J = ed.junction
    assert torch.equal(O[J:], O2[J:])
    assert (O[ev[0]:J] - O2[ev[0]:J]).abs().amax(dim=(1, 2)).min() > 1e-3
    # and no gradient reaches E_k from rows >= J_k
    do2 = do.clone()
    do2[:J] = 0
    _, _, _, dk, dv = A.logittree([t], q, k, v, dout=do2)
    assert torch.all(dk[ev] == 0) and torch.all(dv[ev] == 0)


def test_future_invariance():
    """Rows before p are untouched by anything at or after p (no time travel)."""
    t = synth.make_trajectories("tiny", 1)[0]
    q, k, v, _ = _rand(512, 1, 1, 8, 10)
    O, L = A.logittree([t], q, k, v)
    p = 300
    q2, k2, v2 = q.clone(), k.clone(), v.clone()
    q2[p:] += 1.0
    k2[p:] -= 2.0
    v2[p:] *= 3.0
    O2, L2 = A.logittree([t], q2, k2, v2)
    assert torch.equal(O[:p], O2[:p]) and torch.equal(L[:, :p], L2[:, :p])


def test_pitfall_masks_differ():
    """Negative controls: both pitfalls change the rows the edits touch."""
    t = synth.make_trajectories("tiny", 0)[0]
    q, k, v, _ = _rand(512, 1, 1, 8, 11)
    O, _ = A.logittree([t], q, k, v)
    for kind in ("full", "compressed"):
        M = torch.zeros(512, 512, dtype=torch.bool)
        for r, s in enumerate(V.naive_views(t, kind)):
            M[r, list(s)] = True
        On, _ = A.dense([t], q, k, v, mask=M)
        assert (On - O).abs().max() > 0.1


def test_planted_mistake_in_layers_is_caught(monkeypatch):
    """A layer that forgets its edit (keeps E_k) must fail the brute force pin."""
    trajs = _random_trajs(3, [30], max_edits=3, max_span=6)
    assert any(len(e.evict) for e in trajs[0].edits)
    q, k, v, _ = _rand(30, 1, 1, 4, 2)
    Ob, _ = _brute_rows(trajs, q, k, v)
    real = V.branch_layers

    def leaky(traj):
        out = []
        for first, end, before in real(traj):
            out.append((first, end, list(range(traj.begin, first))))
        return out
    monkeypatch.setattr(V, "branch_layers", leaky)
    O, _ = A.logittree(trajs, q, k, v)
    assert (O - Ob).abs().max() > 1e-3


def test_row_grads_and_row_range_match_full_backward():
    trajs = _random_trajs(21, [40, 33], max_edits=4, max_span=9)
    T = trajs[-1].end
    q, k, v, do = _rand(T, 4, 2, 8, 4)
    _, _, dq, dk, dv = A.logittree(trajs, q, k, v, dout=do)
    rows = [0, 7, 39, 40, 55, T - 1]
    g = A.row_grads(trajs, q, k, v, do, rows)
    assert torch.allclose(g, dq[rows], atol=1e-12, rtol=0)
    # restricting the loss to the rows that see key j reproduces dK_j, dV_j
    death = [x for t in trajs for x in V.death_rows(t)]
    for j in (3, 12, 41, 60):
        _, _, _, dkj, dvj = A.logittree(trajs, q, k, v, dout=do, row_range=(j, death[j]))
        assert torch.allclose(dkj[j], dk[j], atol=1e-12, rtol=0)
        assert torch.allclose(dvj[j], dv[j], atol=1e-12, rtol=0)
