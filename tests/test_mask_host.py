"""The library's host mask builder against the oracle's independent replay
(CPU only): key lifetimes bit-exact, the schedule's visibility bits bit-exact,
mask statistics, and every record error path."""
import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import views as V
from paper_2609_00865_amd import mv, synth
from tests.fixtures import load, trajectory_from


def _oracle_death(trajs):
    out = []
    for t in trajs:
        out.extend(V.death_rows(t))
    return torch.tensor(out, dtype=torch.int32)


def _bits_ok(mask, trajs, rows=None):
    T = mask.total_tokens
    M = OA.visibility(trajs)
    if rows is None:
        bits = mv.unpack_bits(mask.materialize_host(0, T), T)
        return torch.equal(bits, M)
    for r0, r1 in rows:
        bits = mv.unpack_bits(mask.materialize_host(r0, r1), T)
        if not torch.equal(bits, M[r0:r1]):
            return False
    return True


@pytest.mark.parametrize("name", ["running_example.json", "blackbox_payloads.json", "weather.json"])
def test_golden_fixtures(name):
    traj, _ = trajectory_from(load(name))
    m = mv.ViewMask([traj])
    assert torch.equal(m.death(), _oracle_death([traj]))
    assert _bits_ok(m, [traj])


def test_running_example_death_row():
    traj, _ = trajectory_from(load("running_example.json"))
    m = mv.ViewMask([traj])
    assert m.death().tolist() == [14, 14, 14, 14, 14, 7, 14, 14, 10, 14, 14, 12, 14, 14]


@pytest.mark.parametrize("seed", range(25))
def test_random_records(seed):
    rng = np.random.default_rng(1000 + seed)
    lens = [int(x) for x in rng.integers(1, 300, size=int(rng.integers(1, 4)))]
    trajs = synth.random_trajectories(rng, lens, max_edits=8, max_span=40, summary_max=20)
    m = mv.ViewMask(trajs)
    assert torch.equal(m.death(), _oracle_death(trajs))
    assert _bits_ok(m, trajs)
    st = m.stats()
    sizes = [s for t in trajs for s in V.view_sizes(t)]
    assert st["visible_pairs"] == sum(sizes)
    assert st["max_view"] == max(sizes)


@pytest.mark.parametrize("workload,seed", [("tiny", 0), ("tiny", 1), ("medium", 0), ("medium", 1)])
def test_workload_masks(workload, seed):
    trajs = synth.make_trajectories(workload, seed)
    m = mv.ViewMask(trajs)
    assert torch.equal(m.death(), _oracle_death(trajs))
    T = m.total_tokens
    if T <= 512:
        assert _bits_ok(m, trajs)
    else:
        rng = np.random.default_rng(seed)
        starts = [0, T - 128] + [int(x) for x in rng.integers(0, T - 128, size=6)]
        assert _bits_ok(m, trajs, rows=[(s, s + 128) for s in starts])
    st = m.stats()
    sizes = [s for t in trajs for s in V.view_sizes(t)]
    assert st["visible_pairs"] == sum(sizes) and st["max_view"] == max(sizes)


@pytest.mark.slow
@pytest.mark.parametrize("workload", ["b4x32k", "long128k"])
def test_large_workload_lifetimes(workload):
    trajs = synth.make_trajectories(workload, 0)
    m = mv.ViewMask(trajs)
    assert torch.equal(m.death(), _oracle_death(trajs))
    st = m.stats()
    sizes = [s for t in trajs for s in V.view_sizes(t)]
    assert st["visible_pairs"] == sum(sizes) and st["max_view"] == max(sizes)
    # the recipe keeps every view well under the long-horizon bound
    assert st["max_view"] < 24576


def test_negative_control_masks_differ():
    """The schedule bits must not be the pitfalls' masks (discrimination)."""
    t = synth.make_trajectories("tiny", 0)[0]
    m = mv.ViewMask([t])
    bits = mv.unpack_bits(m.materialize_host(0, 512), 512)
    for kind in ("full", "compressed"):
        M = torch.zeros(512, 512, dtype=torch.bool)
        for r, s in enumerate(V.naive_views(t, kind)):
            M[r, list(s)] = True
        assert not torch.equal(bits, M)


def _err(trajs, T=None):
    with pytest.raises(mv.MVError) as e:
        mv.ViewMask(trajs, total_tokens=T)
    return e.value


def test_record_errors():
    E, Tr = synth.Edit, synth.Trajectory
    assert _err([Tr(0, 10, (E(5, ((5, 6),)),))]).name == "MV_ERR_BAD_RECORD"          # span reaches junction
    assert _err([Tr(0, 10, (E(4, ((1, 2),)), E(6, ((1, 2),))))]).name == "MV_ERR_BAD_RECORD"  # evicted twice
    assert _err([Tr(0, 10, (E(6, ()), E(6, ())))]).name == "MV_ERR_BAD_RECORD"         # not increasing
    assert _err([Tr(0, 10, (E(0, ()),))]).name == "MV_ERR_BAD_RECORD"                  # junction at begin
    assert _err([Tr(0, 10, (E(10, ()),))]).name == "MV_ERR_BAD_RECORD"                 # junction at end
    assert _err([Tr(0, 10, (E(8, ((3, 5), (4, 6))),))]).name == "MV_ERR_BAD_RECORD"    # overlapping spans
    assert _err([Tr(0, 10, (E(8, ((4, 6), (1, 2))),))]).name == "MV_ERR_BAD_RECORD"    # unsorted spans
    assert _err([Tr(0, 10, (E(8, ((2, 4),), (3, 5)),))]).name == "MV_ERR_BAD_RECORD"   # summary meets E_k
    assert _err([Tr(0, 10, (E(8, ((2, 4),), (9, 12)),))]).name == "MV_ERR_BAD_RECORD"  # summary outside
    assert _err([Tr(0, 5), Tr(6, 9)]).name == "MV_ERR_BAD_RECORD"                      # gap in packing
    assert _err([Tr(0, 5)], T=6).name == "MV_ERR_BAD_RECORD"                           # does not cover T
    assert _err([Tr(0, 10, (E(8, ((1, 1),)),))]).name == "MV_ERR_BAD_RECORD"           # empty span
    msg = str(_err([Tr(0, 10, (E(4, ((1, 2),)), E(6, ((1, 2),))))]))
    assert "not live" in msg
    # restores: only a token that is out of the view may come back, not in the
    # edit that evicts it, and only from before the junction
    assert _err([Tr(0, 10, (E(4, (), restore=((1, 2),)),))]).name == "MV_ERR_BAD_RECORD"
    assert _err([Tr(0, 10, (E(4, ((1, 2),), restore=((1, 2),)),))]).name == "MV_ERR_BAD_RECORD"
    assert _err([Tr(0, 10, (E(4, ((1, 2),)), E(6, (), restore=((1, 3),))))]).name == "MV_ERR_BAD_RECORD"
    assert _err([Tr(0, 10, (E(4, ((1, 2),)), E(6, (), restore=((7, 8),))))]).name == "MV_ERR_BAD_RECORD"
    assert _err([Tr(0, 10, (E(4, ((1, 2),)), E(6, (), restore=((1, 2),)),
                            E(8, (), restore=((1, 2),))))]).name == "MV_ERR_BAD_RECORD"


def test_empty_edit_and_summary_only_edits():
    trajs = [synth.Trajectory(0, 40, (synth.Edit(10, (), (10, 14)), synth.Edit(20, ((0, 3),))))]
    m = mv.ViewMask(trajs)
    assert torch.equal(m.death(), _oracle_death(trajs))
    assert _bits_ok(m, trajs)


def test_schedule_statistics_are_consistent():
    m = mv.ViewMask(synth.make_trajectories("medium", 0))
    st = m.stats()
    nq = (8192 + 127) // 128
    causal = sum((min(8192, (q + 1) * 128) - 1) // 64 + 1 for q in range(nq))
    assert st["tiles_full"] + st["tiles_partial"] + st["tiles_skipped"] == causal
    assert st["tiles_skipped"] > 0.3 * causal


@pytest.mark.parametrize("T", [1, 63, 64, 65, 129, 257, 300])
def test_ragged_tail_tiles_are_never_full(T):
    """A key tile that runs past the last token is always partial: full tiles
    skip the predicate and would otherwise admit padding keys."""
    m = mv.ViewMask([synth.Trajectory(0, T, ())])
    st = m.stats()
    n_qt = (T + 127) // 128
    causal = sum((min(T, (q + 1) * 128) - 1) // 64 + 1 for q in range(n_qt))
    # with no edits a tile is full iff it is complete and lies below the diagonal
    full = sum(1 for q in range(n_qt) for kt in range((min(T, (q + 1) * 128) - 1) // 64 + 1)
               if kt * 64 + 64 <= T and kt * 64 + 63 <= q * 128)
    assert st["tiles_full"] == full
    assert st["tiles_full"] + st["tiles_partial"] == causal
    assert _bits_ok(m, [synth.Trajectory(0, T, ())])


def test_restore_hand_example():
    """y1, y2 evicted at row 4; y1 restored at row 7: rows 4-6 see neither,
    rows 7-9 see y1 again (at its own position), y2 never comes back."""
    E, Tr = synth.Edit, synth.Trajectory
    trajs = [Tr(0, 10, (E(4, ((1, 3),)), E(7, (), restore=((1, 2),))))]
    m = mv.ViewMask(trajs)
    assert m.death().tolist() == [10, 4, 4] + [10] * 7
    ptr, iv = m.intervals()
    assert ptr.tolist() == [0, 0, 1] + [1] * 8 and iv.tolist() == [[7, 10]]
    assert V.lifetimes(trajs[0])[1] == [(1, 4), (7, 10)]
    assert _bits_ok(m, trajs)
    views = V.views(trajs[0])
    assert views[5] == frozenset({0, 3, 4, 5}) and views[8] == frozenset({0, 1, 3, 4, 5, 6, 7, 8})
    assert m.stats()["visible_pairs"] == sum(len(v) for v in views)


@pytest.mark.parametrize("seed", range(25))
def test_random_records_with_restores(seed):
    rng = np.random.default_rng(7000 + seed)
    lens = [int(x) for x in rng.integers(2, 300, size=int(rng.integers(1, 4)))]
    trajs = synth.random_trajectories(rng, lens, max_edits=10, max_span=40, summary_max=10,
                                      restore_max=30)
    m = mv.ViewMask(trajs)
    assert torch.equal(m.death(), _oracle_death(trajs))
    ptr, iv = m.intervals()
    want = [ivs[1:] for tr in trajs for ivs in V.lifetimes(tr)]
    got = [iv[ptr[j]:ptr[j + 1]].tolist() for j in range(trajs[-1].end)]
    assert got == [[list(x) for x in w] for w in want]
    assert _bits_ok(m, trajs)
    sizes = [s for t in trajs for s in V.view_sizes(t)]
    st = m.stats()
    assert st["visible_pairs"] == sum(sizes) and st["max_view"] == max(sizes)

