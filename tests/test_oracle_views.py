"""Pins for the oracle's view replay: the paper's worked examples, the direct
set definition, and the budget identities of Appendix B.3."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import views as V
from paper_2609_00865_amd import synth
from tests.fixtures import load, trajectory_from


def _running_example_ok(views_fn, final_fn):
    fix = load("running_example.json")
    traj, pos = trajectory_from(fix)
    vs = views_fn(traj)
    final = set(final_fn(traj))
    for leaf in fix["leaves"]:
        row = pos[leaf["leaf"]] - 1                  # logits for y_t come from row t-1
        live = {fix["tokens"][j] for j in vs[row]} - {"s"}
        fin = {fix["tokens"][j] for j in final if j <= row} - {"s"}
        if live != set(leaf["live"]) or fin != set(leaf["final"]):
            return False
        if live - fin != set(leaf["diverges_by"]):
            return False
    return True


def test_running_example_table():
    assert _running_example_ok(V.views, V.final_walk)


def test_running_example_full_mask():
    """The 14 x 14 mask the table implies (prompt included), row by row."""
    fix = load("running_example.json")
    traj, _ = trajectory_from(fix)
    expect = {r: set(range(r + 1)) for r in range(7)}
    expect.update({7: {0, 1, 2, 3, 4, 6, 7}, 8: {0, 1, 2, 3, 4, 6, 7, 8},
                   9: {0, 1, 2, 3, 4, 6, 7, 8, 9}, 10: {0, 1, 2, 3, 4, 6, 7, 9, 10},
                   11: {0, 1, 2, 3, 4, 6, 7, 9, 10, 11}, 12: {0, 1, 2, 3, 4, 6, 7, 9, 10, 12},
                   13: {0, 1, 2, 3, 4, 6, 7, 9, 10, 12, 13}})
    assert [set(s) for s in V.views(traj)] == [expect[r] for r in range(14)]
    assert V.death_rows(traj) == [14, 14, 14, 14, 14, 7, 14, 14, 10, 14, 14, 12, 14, 14]


def test_planted_mistakes_fail_the_table(monkeypatch):
    """An off-by-one junction, a dropped edit and the two pitfalls all fail."""
    late = lambda t: [frozenset(V.view_by_definition(t, r - 1) | {r}) if r > t.begin
                      else frozenset({r}) for r in range(t.begin, t.end)]
    assert not _running_example_ok(late, V.final_walk)
    assert not _running_example_ok(lambda t: V.naive_views(t, "full"), V.final_walk)
    assert not _running_example_ok(lambda t: V.naive_views(t, "compressed"), V.final_walk)

    def drop_last(t):
        return V.views(synth.Trajectory(t.begin, t.end, t.edits[:-1]))
    assert not _running_example_ok(drop_last, V.final_walk)


def test_blackbox_payload_rows():
    fix = load("blackbox_payloads.json")
    traj, pos = trajectory_from(fix)
    vs = V.views(traj)
    for row in fix["payload_rows"]:
        assert {fix["tokens"][j] for j in vs[pos[row["row"]]]} == set(row["view"])
    # the harness-written summary does not see the span evicted at its own junction
    assert pos["y2"] not in vs[pos["summary"]]


def test_weather_rows():
    fix = load("weather.json")
    traj, pos = trajectory_from(fix)
    names = fix["tokens"]
    vs = V.views(traj)
    comp = V.naive_views(traj, "compressed")
    full = V.naive_views(traj, "full")
    for row in fix["rows"]:
        r = pos[row["row"]]
        assert {names[j] for j in vs[r]} == set(row["rollout_sees"])
        if "naive_compressed_sees" in row:
            assert {names[j] for j in comp[r]} == set(row["naive_compressed_sees"])
        if "naive_full_sees" in row:
            assert {names[j] for j in full[r]} == set(row["naive_full_sees"])


def _check_against_definition(trajs):
    for t in trajs:
        vs = V.views(t)
        death = V.death_rows(t)
        for r in range(t.begin, t.end):
            d = V.view_by_definition(t, r)
            assert vs[r - t.begin] == d
            assert len(d) == V.view_sizes(t)[r - t.begin]
        life = V.lifetimes(t)
        for j in range(t.begin, t.end):
            seen = [r for r in range(t.begin, t.end) if j in vs[r - t.begin]]
            ivs = life[j - t.begin]
            assert seen == [r for b, e in ivs for r in range(b, e)]
            assert ivs[0][0] == j and death[j - t.begin] == ivs[0][1]


@pytest.mark.parametrize("seed", range(20))
def test_replay_matches_definition(seed):
    rng = np.random.default_rng(seed)
    trajs = synth.random_trajectories(rng, [int(x) for x in rng.integers(3, 40, size=3)])
    _check_against_definition(trajs)


@settings(max_examples=60, deadline=None)
@given(st.integers(0, 2**31 - 1), st.lists(st.integers(1, 30), min_size=1, max_size=3))
def test_replay_matches_definition_hypothesis(seed, lengths):
    rng = np.random.default_rng(seed)
    _check_against_definition(synth.random_trajectories(rng, lengths, max_edits=5))


@pytest.mark.parametrize("seed", range(20))
def test_replay_matches_definition_with_restores(seed):
    rng = np.random.default_rng(100 + seed)
    trajs = synth.random_trajectories(rng, [int(x) for x in rng.integers(3, 60, size=3)],
                                      max_edits=8, max_span=10, restore_max=8)
    _check_against_definition(trajs)
    for t in trajs:
        live = V.views(t)
        for j, ivs in zip(range(t.begin, t.end), V.lifetimes(t)):
            rows = {r for r in range(t.begin, t.end) if j in live[r - t.begin]}
            assert rows == {r for b, e in ivs for r in range(b, e)}
            assert all(e < b2 for (_, e), (b2, _) in zip(ivs, ivs[1:]))   # disjoint, gaps


def test_restore_re_enters_in_physical_order():
    t = synth.Trajectory(0, 9, (synth.Edit(3, ((0, 2),)), synth.Edit(6, (), restore=((1, 2),))))
    rows = {r: list(lv) for r, lv in V.replay(t)}
    assert rows[5] == [2, 3, 4, 5]
    assert rows[6] == [1, 2, 3, 4, 5, 6]          # y1 back at its own slot
    with pytest.raises(V.BadRecord):
        list(V.replay(synth.Trajectory(0, 9, (synth.Edit(3, (), restore=((1, 2),)),))))


def _budget(t):
    layers = V.branch_layers(t)
    L = t.end - t.begin
    evicted = set()
    for e in t.edits:
        for b, x in e.evict:
            evicted.update(range(b, x))
    C = len(V.final_walk(t))
    ells = [len(before) + (end - first) for first, end, before in layers]
    return L, C, ells, layers, evicted


@pytest.mark.parametrize("workload,seed", [("tiny", 0), ("tiny", 1), ("medium", 0), ("medium", 1)])
def test_budget_identities(workload, seed):
    """C = L - |U E_k|; l_i <= L; l_{K+1} = C; sum l_i > L for K >= 1 (App. B.3).

    The appendix also states C <= l_i; with l_i the length of layer i's own
    sequence that fails for an early, short layer (here l_1 = J_1 < C), so it
    is not asserted.
    """
    for t in synth.make_trajectories(workload, seed):
        L, C, ells, layers, evicted = _budget(t)
        assert C == L - len(evicted)
        assert len(ells) == len(t.edits) + 1
        assert all(l <= L for l in ells)
        assert ells[-1] == C
        assert sum(ells) > L
        # each layer's last row sees exactly the layer's sequence
        sizes = V.view_sizes(t)
        for (first, end, before), l in zip(layers, ells):
            assert sizes[end - 1 - t.begin] == l


def test_budget_equality_without_edits():
    t = synth.Trajectory(0, 50, ())
    L, C, ells, _, _ = _budget(t)
    assert ells == [L] and C == L


def test_workload_records_are_valid_and_shaped():
    """Every generated record replays, and the recipes' stated shapes hold."""
    for wl, kw in [("tiny", {}), ("medium", {})]:
        for seed in (0, 1):
            trajs = synth.make_trajectories(wl, seed)
            T, _ = V.packed(trajs)
            assert T == synth.ATTN_WORKLOADS[wl].total_tokens
            for t in trajs:
                V.death_rows(t)             # raises on an invalid record
    t = synth.make_trajectories("tiny", 0)[0]
    assert [e.junction for e in t.edits] == [192, 384]
    assert all(sum(b - a for a, b in e.evict) == 96 for e in t.edits)


def test_bad_records_raise():
    with pytest.raises(V.BadRecord):
        V.death_rows(synth.Trajectory(0, 10, (synth.Edit(5, ((5, 6),)),)))   # evicts the junction row
    with pytest.raises(V.BadRecord):
        V.death_rows(synth.Trajectory(0, 10, (synth.Edit(4, ((1, 2),)), synth.Edit(6, ((1, 2),)))))
    with pytest.raises(V.BadRecord):
        V.death_rows(synth.Trajectory(0, 10, (synth.Edit(6, ()), synth.Edit(6, ()))))
    with pytest.raises(V.BadRecord):
        V.packed([synth.Trajectory(0, 5), synth.Trajectory(6, 9)])
