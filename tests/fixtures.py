"""Turn the paper's worked examples under tests/golden/ into trajectories."""
import json
import os

from paper_2609_00865_amd.synth import Edit, Trajectory

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def trajectory_from(fix):
    """One trajectory over the fixture's token names, positions 0..n-1."""
    pos = {t: i for i, t in enumerate(fix["tokens"])}
    edits = []
    for e in fix["edits"]:
        J = e["junction"]
        J = pos[J] if isinstance(J, str) else int(J)
        ev = sorted(pos[t] for t in e["evict"])
        spans = []
        for p in ev:
            if spans and spans[-1][1] == p:
                spans[-1] = (spans[-1][0], p + 1)
            else:
                spans.append((p, p + 1))
        edits.append(Edit(J, tuple(spans)))
    return Trajectory(0, len(fix["tokens"]), tuple(edits)), pos
