"""Pins of the branch-replicated packing oracle (CPU only).

The running example's packed segments against Table "running-prefixes"; the
packed length identity of Appendix G; owner rows covering each physical row
once, at the position the token had in its live context; the block-diagonal
mask reproducing every view; RoPE against its complex-product form, a hand
example, norm preservation and the relative-position property; multi-layer
exactness of the packed stream against per-branch forwards, with the union
form failing under RoPE at any depth and without positions from the second
layer on (the reason the paper's training loop packs)."""
import math

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import packing as OP
from oracle import views as V
from paper_2609_00865_amd import synth
from tests.fixtures import load, trajectory_from

F64 = torch.float64


def test_running_example_segments():
    fix = load("running_example.json")
    traj, pos = trajectory_from(fix)
    names = {i: n for n, i in pos.items()}
    pk = OP.branch_pack([traj])
    assert len(pk["seg_begin"]) - 1 == 4            # K + 1 branch layers
    assert pk["seg_begin"][-1] == 7 + 9 + 10 + 11
    # each leaf's decoding row r = t - 1 sits in one segment; the segment's
    # prefix up to that slot is the live prefix the table lists (plus s)
    for e in fix["leaves"]:
        r = pos[e["leaf"]] - 1
        slot = [i for i in range(len(pk["src"])) if pk["src"][i] == r and pk["owner"][i]]
        assert len(slot) == 1
        slot = slot[0]
        b = max(x for x in pk["seg_begin"] if x <= slot)
        seq = [names[j] for j in pk["src"][b:slot + 1] if j != pos["s"]]
        assert seq == e["live"]
        assert pk["pos"][slot] == len(e["live"])        # s at position 0
        assert pk["target"][slot] == pos[e["leaf"]]


@pytest.mark.parametrize("seed", range(20))
def test_layout_properties(seed):
    rng = np.random.default_rng(3000 + seed)
    lens = [int(x) for x in rng.integers(1, 200, size=int(rng.integers(1, 4)))]
    trajs = synth.random_trajectories(rng, lens, max_edits=6, max_span=30, summary_max=8)
    T = trajs[-1].end
    pk = OP.branch_pack(trajs)
    N = pk["seg_begin"][-1]
    assert N == sum(len(b) + (e - f) for tr in trajs for f, e, b in V.branch_layers(tr))
    assert N >= T
    own = [s for s, o in zip(pk["src"], pk["owner"]) if o]
    assert sorted(own) == list(range(T))               # every row owned exactly once
    M = OA.visibility(trajs)
    B = OP.block_causal_mask(pk["seg_begin"])
    src = torch.tensor(pk["src"])
    sizes = {tr_r: s for tr in trajs for tr_r, s in zip(range(tr.begin, tr.end), V.view_sizes(tr))}
    for i in range(N):
        if not pk["owner"][i]:
            continue
        r = pk["src"][i]
        seen = torch.zeros(T, dtype=torch.bool)
        seen[src[B[i]]] = True
        assert torch.equal(seen, M[r])                 # the packed row sees exactly View(r)
        assert pk["pos"][i] == sizes[r] - 1            # gap-free logical position


def test_rope_forms_and_properties():
    gen = torch.Generator().manual_seed(0)
    x = torch.randn(50, 3, 16, generator=gen, dtype=F64)
    pos = torch.randint(0, 40000, (50,), generator=gen)
    a = OP.rope(x, pos, 1e6)
    assert torch.allclose(a, OP.rope_complex(x, pos, 1e6), atol=1e-12)
    assert torch.allclose(OP.rope(x, torch.zeros(50), 1e6), x)
    assert torch.allclose(a.norm(dim=-1), x.norm(dim=-1), atol=1e-12)
    assert torch.allclose(OP.rope(a, pos, 1e6, inverse=True), x, atol=1e-10)
    # <R(m) q, R(n) k> = <R(m - n) q, k>
    q, k = x[:25], x[25:]
    m, n = pos[:25], pos[25:]
    lhs = (OP.rope(q, m, 1e4) * OP.rope(k, n, 1e4)).sum(-1)
    rhs = (OP.rope(q, m - n, 1e4) * k).sum(-1)
    assert torch.allclose(lhs, rhs, atol=1e-9)
    # hand example: d = 4, theta = 100, position 1: frequencies 1 and 0.1
    v = torch.tensor([[[1.0, 2.0, 3.0, 4.0]]], dtype=F64)
    got = OP.rope(v, [1], 100.0)[0, 0]
    c1, s1, c2, s2 = math.cos(1), math.sin(1), math.cos(0.1), math.sin(0.1)
    want = [1 * c1 - 3 * s1, 2 * c2 - 4 * s2, 3 * c1 + 1 * s1, 4 * c2 + 2 * s2]
    assert torch.allclose(got, torch.tensor(want, dtype=F64), atol=1e-14)


def _toy(seed, W, H, n_layers):
    gen = torch.Generator().manual_seed(seed)
    d = W // H
    return [{"wq": torch.randn(W, W, generator=gen, dtype=F64) / math.sqrt(W),
             "wk": torch.randn(W, W, generator=gen, dtype=F64) / math.sqrt(W),
             "wv": torch.randn(W, W, generator=gen, dtype=F64) / math.sqrt(W),
             "wo": torch.randn(W, W, generator=gen, dtype=F64) / math.sqrt(W)}
            for _ in range(n_layers)], d


@pytest.mark.parametrize("n_layers", [1, 2, 3])
def test_packed_stream_is_exact_over_layers(n_layers):
    traj, _ = trajectory_from(load("running_example.json"))
    rng = np.random.default_rng(7)
    trajs = [traj] + synth.random_trajectories(rng, [90], max_edits=4, max_span=12)
    trajs[1] = synth.Trajectory(14, 14 + 90, tuple(
        synth.Edit(e.junction + 14, tuple((b + 14, x + 14) for b, x in e.evict),
                   (e.summary[0] + 14, e.summary[1] + 14)) for e in trajs[1].edits))
    T = trajs[-1].end
    W, H = 16, 2
    layers, d = _toy(n_layers, W, H, n_layers)
    x0 = torch.randn(T, W, generator=torch.Generator().manual_seed(1), dtype=F64)
    ref = OP.toy_logittree(trajs, x0, layers, H, d, 1e4)
    got = OP.toy_packed(trajs, x0, layers, H, d, 1e4)
    assert torch.allclose(got, ref, atol=1e-10)
    # The union form: one position per token cannot be right for every row
    # (a key's index in a later row's view shifts once a span before it is
    # evicted), so with RoPE it misses even one layer; without positions it
    # matches one layer and misses a stack (keys past an evicted span carry
    # hidden states computed with the span visible).
    logical = [s - 1 for tr in trajs for s in V.view_sizes(tr)]
    uni = OP.toy_union(trajs, x0, layers, H, d, 1e4, positions=logical)
    assert float((uni - ref).abs().max()) > 1e-3
    ref0 = OP.toy_logittree(trajs, x0, layers, H, d, 0.0)
    assert torch.allclose(OP.toy_packed(trajs, x0, layers, H, d, 0.0), ref0, atol=1e-10)
    err0 = float((OP.toy_union(trajs, x0, layers, H, d, 0.0) - ref0).abs().max())
    if n_layers == 1:
        assert err0 < 1e-10
    else:
        assert err0 > 1e-3


def test_unpack_is_the_adjoint_of_the_gather():
    rng = np.random.default_rng(5)
    trajs = synth.random_trajectories(rng, [120, 80], max_edits=5, max_span=15)
    pk = OP.branch_pack(trajs)
    T, N = trajs[-1].end, pk["seg_begin"][-1]
    gen = torch.Generator().manual_seed(2)
    x = torch.randn(T, 6, generator=gen, dtype=F64)
    g = torch.randn(N, 6, generator=gen, dtype=F64)
    lhs = (x[pk["src"]] * g).sum()
    rhs = (x * OP.unpack_sum(pk, g, T)).sum()
    assert abs(float(lhs - rhs)) < 1e-10


def test_shared_trunk_running_example():
    """Hand-derived from Table "running-prefixes": branch 1 (rows y8..y10)
    shares s, y1..y4 with branch 0 and stores y6 again (its position moves
    from 6 to 5 once y5 is evicted), then its rows; branch 2 shares up to y7
    and stores y10 again; branch 3 shares up to y10."""
    fix = load("running_example.json")
    traj, pos = trajectory_from(fix)
    names = {i: n for n, i in pos.items()}
    pk = OP.shared_trunk_pack([traj])
    assert pk["seg_begin"] == [0, 7, 11, 14, 16]
    assert pk["src"] == [0, 1, 2, 3, 4, 5, 6, 6, 7, 8, 9, 9, 10, 11, 12, 13]
    assert pk["pos"] == [0, 1, 2, 3, 4, 5, 6, 5, 6, 7, 8, 7, 8, 9, 9, 10]
    assert pk["owner"] == [1] * 7 + [0, 1, 1, 1, 0, 1, 1, 1, 1]
    for e in fix["leaves"]:
        r = pos[e["leaf"]] - 1
        slot = [i for i in range(16) if pk["src"][i] == r and pk["owner"][i]]
        assert len(slot) == 1
        seen = [names[pk["src"][j]] for j in pk["views"][slot[0]] if pk["src"][j] != pos["s"]]
        assert seen == e["live"]
        assert pk["pos"][slot[0]] == len(e["live"])


@pytest.mark.parametrize("seed", range(20))
def test_shared_trunk_views(seed):
    """Every slot's view is its branch prefix; owner slots see exactly their
    row's view at its gap-free position; each branch stores only what its
    predecessor does not share, so the stream is no longer than the
    replicated one and each segment starts where the branches diverge."""
    rng = np.random.default_rng(7000 + seed)
    lens = [int(x) for x in rng.integers(1, 200, size=int(rng.integers(1, 4)))]
    trajs = synth.random_trajectories(rng, lens, max_edits=6, max_span=30, summary_max=8,
                                      restore_max=12 if seed % 2 else 0)
    T = trajs[-1].end
    pk = OP.shared_trunk_pack(trajs)
    rep = OP.branch_pack(trajs)
    N = pk["seg_begin"][-1]
    assert T <= N <= rep["seg_begin"][-1]
    own = [s for s, o in zip(pk["src"], pk["owner"]) if o]
    assert sorted(own) == list(range(T))
    M = OA.visibility(trajs)
    sizes = {r: s for tr in trajs for r, s in zip(range(tr.begin, tr.end), V.view_sizes(tr))}
    for i in range(N):
        view_src = [pk["src"][j] for j in pk["views"][i]]
        assert len(view_src) == pk["pos"][i] + 1
        assert view_src[-1] == pk["src"][i] and pk["views"][i][-1] == i
        if pk["owner"][i]:
            r = pk["src"][i]
            seen = torch.zeros(T, dtype=torch.bool)
            seen[view_src] = True
            assert torch.equal(seen, M[r])
            assert pk["pos"][i] == sizes[r] - 1
    # segment k begins where S_k leaves S_{k-1}: at position d_k, with the
    # token S_k[d_k], and its length is |S_k| - d_k
    seg = 0
    for tr in trajs:
        seqs = [list(b) + list(range(f, e)) for f, e, b in V.branch_layers(tr)]
        for k, sq in enumerate(seqs):
            d = 0
            if k > 0:
                prev = seqs[k - 1]
                while d < min(len(sq), len(prev)) and sq[d] == prev[d]:
                    d += 1
            b, e = pk["seg_begin"][seg], pk["seg_begin"][seg + 1]
            assert pk["pos"][b] == d and pk["src"][b] == sq[d] and e - b == len(sq) - d
            seg += 1
    assert seg == len(pk["seg_begin"]) - 1


@pytest.mark.parametrize("n_layers", [1, 2, 3])
def test_shared_trunk_stream_is_exact_over_layers(n_layers):
    traj, _ = trajectory_from(load("running_example.json"))
    rng = np.random.default_rng(8)
    extra = synth.random_trajectories(rng, [90], max_edits=4, max_span=12)[0]
    trajs = [traj, synth.Trajectory(14, 14 + 90, tuple(
        synth.Edit(e.junction + 14, tuple((b + 14, x + 14) for b, x in e.evict),
                   (e.summary[0] + 14, e.summary[1] + 14)) for e in extra.edits))]
    T = trajs[-1].end
    W, H = 16, 2
    layers, d = _toy(10 + n_layers, W, H, n_layers)
    x0 = torch.randn(T, W, generator=torch.Generator().manual_seed(3), dtype=F64)
    for theta in (1e4, 0.0):
        ref = OP.toy_logittree(trajs, x0, layers, H, d, theta)
        got = OP.toy_shared_trunk(trajs, x0, layers, H, d, theta)
        assert torch.allclose(got, ref, atol=1e-10)
    # a planted mistake: sharing one token past the divergence point must fail
    pk = OP.shared_trunk_pack(trajs)
    bad_views = [list(v) for v in pk["views"]]
    moved = 0
    for i in range(len(bad_views)):
        if not pk["owner"][i] and len(bad_views[i]) > 1:
            bad_views[i] = bad_views[i][:-2] + bad_views[i][-1:]   # drop the previous slot
            moved += 1
    assert moved > 0
    assert not torch.equal(OP.views_mask(bad_views), OP.views_mask(pk["views"]))
