"""Live views by replaying the eviction record (test infrastructure only).

The paper's policy conditions step t on the physical history with exactly the
edits fired by step t applied (Eq. "live-view", Section 3.2).  The record of a
rollout is the physical union plus the ordered edits (J_k, E_k) (Appendix E.1;
Definition "trajectory tree", Appendix B.1).

Reading used throughout (the paper's Table "running-prefixes" fixes it): rows
are physical positions, the logits for token y_t come from row t-1, and edit k
is applied *before* row J_k is evaluated; rows < J_k still see E_k, rows >= J_k
do not.  Summary tokens are ordinary tokens born at their own row.

Trajectories are any objects with ``begin``, ``end`` and ``edits``; an edit has
``junction`` and ``evict`` (iterable of half-open physical spans), and
optionally ``restore``: spans evicted by earlier edits that are live again
from the junction on (an offload / retrieve memory, where a token can leave
the view and re-enter it, Appendix E).  A restored token re-enters at its own
physical position, so the live list stays in physical order.
"""
from __future__ import annotations

from typing import Dict, Iterator, List, Sequence, Tuple


class BadRecord(ValueError):
    """The eviction record cannot describe a rollout."""


def _evicted_positions(edit) -> List[int]:
    out: List[int] = []
    for b, e in edit.evict:
        out.extend(range(int(b), int(e)))
    return out


def _restored_positions(edit) -> List[int]:
    out: List[int] = []
    for b, e in getattr(edit, "restore", ()):
        out.extend(range(int(b), int(e)))
    return out


def _edits_by_row(traj) -> Dict[int, tuple]:
    by_row: Dict[int, tuple] = {}
    last = None
    for ed in traj.edits:
        J = int(ed.junction)
        if not (traj.begin < J < traj.end):
            raise BadRecord(f"junction {J} outside ({traj.begin}, {traj.end})")
        if last is not None and J <= last:
            raise BadRecord("junctions must be strictly increasing")
        last = J
        by_row[J] = (_evicted_positions(ed), _restored_positions(ed))
    return by_row


def replay(traj) -> Iterator[Tuple[int, List[int]]]:
    """Yield (row, live list) for every row of one trajectory, in order.

    The live list is the ordered context the policy held while evaluating the
    row (the row itself included).  The yielded list is the replay's working
    state: copy it if it must outlive the iteration step.
    """
    by_row = _edits_by_row(traj)
    live: Dict[int, None] = {}          # insertion-ordered set
    for r in range(traj.begin, traj.end):
        evict, restore = by_row.get(r, ((), ()))
        for p in evict:
            if p not in live:
                raise BadRecord(f"edit at row {r} evicts {p}, which is not live")
            del live[p]
        if restore:
            for p in restore:
                if p in live or not (traj.begin <= p < r) or p in evict:
                    raise BadRecord(f"edit at row {r} restores {p}, which is not evicted")
                live[p] = None
            live = dict.fromkeys(sorted(live))
        live[r] = None
        yield r, live


def views(traj) -> List[frozenset]:
    """View(r) as a set, for every row (small trajectories only)."""
    return [frozenset(lv) for _, lv in replay(traj)]


def view_sizes(traj) -> List[int]:
    """|View(r)| for every row."""
    return [len(lv) for _, lv in replay(traj)]


def death_rows(traj) -> List[int]:
    """For every key of the trajectory, the first row that no longer sees it.

    This is omega(j) of Eq. "4d-mask-def" (Section 4.2) with +infinity written
    as the trajectory's end (for a key that re-enters, the end of its first
    live interval; see ``lifetimes``).  Derived from the record by replaying
    the live set: the row at which the key first leaves it.
    """
    return [iv[0][1] for iv in lifetimes(traj)]


def lifetimes(traj) -> List[List[Tuple[int, int]]]:
    """For every key, the maximal runs of rows [b, e) whose view holds it,
    replayed edit by edit (the same checks as ``replay``)."""
    by_row = _edits_by_row(traj)
    out: List[List[Tuple[int, int]]] = [[] for _ in range(traj.end - traj.begin)]
    open_at: Dict[int, int] = {}
    for r in range(traj.begin, traj.end):
        evict, restore = by_row.get(r, ((), ()))
        for p in evict:
            if p not in open_at:
                raise BadRecord(f"edit at row {r} evicts {p}, which is not live")
            out[p - traj.begin].append((open_at.pop(p), r))
        for p in restore:
            if p in open_at or not (traj.begin <= p < r) or p in evict:
                raise BadRecord(f"edit at row {r} restores {p}, which is not evicted")
            open_at[p] = r
        open_at[r] = r
    for p, b in open_at.items():
        out[p - traj.begin].append((b, traj.end))
    for iv in out:
        iv.sort()
    return out


def view_by_definition(traj, r: int) -> frozenset:
    """View(r) straight from the definition, without incremental state.

    Key j is visible to row r iff j <= r and the last edit fired by row r
    (J_k <= r) that names j does not evict it.
    """
    gone = set()
    for ed in sorted(traj.edits, key=lambda e: int(e.junction)):
        if int(ed.junction) <= r:
            gone.update(_evicted_positions(ed))
            gone.difference_update(_restored_positions(ed))
    return frozenset(j for j in range(traj.begin, r + 1) if j not in gone)


def branch_layers(traj) -> List[Tuple[int, int, List[int]]]:
    """The K+1 branch layers of the trajectory tree (Appendix B.1).

    Layer k holds the rows [J_k, J_{k+1}) (J_0 = begin, J_{K+1} = end).  Each
    entry is (first row, end row, keys live just before the first row is
    appended), so the layer's sequence is ``keys ++ range(first, end)`` and
    ordinary causal attention over it gives every row of the layer its view
    (Section 4.1: each branch is forwarded as its own sequence).
    """
    bounds = [traj.begin] + [int(e.junction) for e in traj.edits] + [traj.end]
    starts = set(bounds[:-1])
    layers = []
    cur = None
    for r, live in replay(traj):
        if r in starts:
            if cur is not None:
                layers.append(cur)
            before = [p for p in live if p != r]
            cur = [r, r, before]
        cur[1] = r + 1
    layers.append(cur)
    return [tuple(x) for x in layers]


def final_walk(traj) -> List[int]:
    """The final compressed walk: what survives every edit (Eq. "live-vs-final")."""
    last = None
    for _, lv in replay(traj):
        last = lv
    return list(last) if last is not None else []


def naive_views(traj, kind: str) -> List[frozenset]:
    """The two pitfalls' conditioning sets, for negative-control tests.

    ``full``:       the physical prefix H_{<=r} (Pitfall B, Eq. "pitfall-B-symptom").
    ``compressed``: the prefix of the final compressed walk (Pitfall A,
                    Eq. "pitfall-A-symptom"): every edit applied, even future ones.
    """
    if kind == "full":
        return [frozenset(range(traj.begin, r + 1)) for r in range(traj.begin, traj.end)]
    if kind == "compressed":
        kept = set(final_walk(traj))
        return [frozenset(j for j in range(traj.begin, r + 1) if j in kept or j == r)
                for r in range(traj.begin, traj.end)]
    raise ValueError(kind)


def packed(trajs: Sequence) -> Tuple[int, List]:
    """Check that trajectories tile [0, T) back-to-back; return T."""
    pos = 0
    for t in trajs:
        if t.begin != pos or t.end <= t.begin:
            raise BadRecord("trajectories must tile [0, T) in order")
        pos = t.end
    return pos, list(trajs)
