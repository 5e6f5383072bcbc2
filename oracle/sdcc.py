"""SDCC junction KL (test infrastructure only).

Self-distillation for conditioning consistency (Section 5.1) adds, at every
diverging leaf p, the forward KL between the policy under the live prefix
z_p (teacher, gradient stopped) and the policy under the final-walk prefix x_p
(student), Eq. "soft_loss":

    KL_p = sum_v P(v | z_p) (log P(v | z_p) - log Q(v | x_p)).

Leaves (Eq. "sdcc-contexts"; Definition "trajectory tree", Appendix B.1): a
token y_t of the final compressed walk whose live prefix differs from its
final-walk prefix.  Both prefixes are physical positions: the live prefix of
y_t is View(t-1) (the row that decoded y_t, Eq. "live-view"), the final-walk
prefix is the set of surviving positions before t.  The teacher row is t-1 of
a live-view pass; the student row is the last surviving position before t in
a final-walk pass.  A token whose final-walk prefix is empty has no student
row and carries no KL term.

The policy head is the same softmax(W h) as the token log-prob, so with
teacher and student hidden states hT, hS:

    KL = sum_v p_v (zT_v - zS_v) - lseT + lseS,   p = softmax(zT), zX = W hX,

and since the teacher is stop-gradient the derivative into the student
hidden state is the textbook cross-entropy gradient (q - p)^T W (q =
softmax(zS)).  All arithmetic in fp64 unless the caller asks otherwise.
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import torch

from oracle import views as V


def diverging_leaves(traj) -> List[Tuple[int, int, int]]:
    """(token, teacher row, student row) for every diverging leaf, in order.

    Straight from the definition: compare the replayed live view of row t-1
    with the surviving positions before t.
    """
    live = V.views(traj)
    survivors = sorted(V.final_walk(traj))
    alive = set(survivors)
    out = []
    for t in range(traj.begin + 1, traj.end):
        if t not in alive:
            continue
        final_prefix = frozenset(j for j in survivors if j < t)
        if not final_prefix:
            continue
        if live[t - 1 - traj.begin] != final_prefix:
            out.append((t, t - 1, max(final_prefix)))
    return out


def teacher_prefix(traj, t: int) -> List[int]:
    """The teacher context of Eq. "teacher-reconstruction", built the other way
    round: start from the final-walk prefix of y_t and re-insert, at their
    original slots, every evicted position still live when y_t was decoded
    (the spans active at t, Appendix "variational", the set A(p))."""
    survivors = [j for j in sorted(V.final_walk(traj)) if j < t]
    active = []
    for ed in traj.edits:
        if int(ed.junction) >= t:            # fired after row t-1 was evaluated
            for b, e in ed.evict:
                active.extend(j for j in range(int(b), int(e)) if j < t)
    return sorted(set(survivors) | set(active))


def packed_leaves(trajs: Sequence) -> List[Tuple[int, int, int]]:
    out = []
    for tr in trajs:
        out.extend(diverging_leaves(tr))
    return out


def junction_kl(h_teacher, h_student, weight, dtype=torch.float64):
    """Per-leaf KL(p || q), lseT, lseS for matching rows of h_teacher, h_student."""
    W = weight.to(dtype)
    zT = h_teacher.to(dtype) @ W.T
    zS = h_student.to(dtype) @ W.T
    lT = torch.logsumexp(zT, dim=1)
    lS = torch.logsumexp(zS, dim=1)
    logp = zT - lT[:, None]
    logq = zS - lS[:, None]
    kl = (logp.exp() * (logp - logq)).sum(dim=1)
    return kl, lT, lS


def junction_kl_grad(h_teacher, h_student, weight, dkl, dtype=torch.float64):
    """d(sum_p dkl_p KL_p)/d h_student = dkl_p (q - p)^T W (teacher stop-grad)."""
    W = weight.to(dtype)
    p = torch.softmax(h_teacher.to(dtype) @ W.T, dim=1)
    q = torch.softmax(h_student.to(dtype) @ W.T, dim=1)
    return dkl.to(dtype)[:, None] * ((q - p) @ W)


def total_variation(h_teacher, h_student, weight, dtype=torch.float64):
    """||p - q||_TV per leaf (the left side of Proposition "pinsker-bound")."""
    W = weight.to(dtype)
    p = torch.softmax(h_teacher.to(dtype) @ W.T, dim=1)
    q = torch.softmax(h_student.to(dtype) @ W.T, dim=1)
    return 0.5 * (p - q).abs().sum(dim=1)


def kl_weight(step: int, total_steps: int, lambda_max: float = 0.1,
              warmup_frac: float = 0.2) -> float:
    """The lambda schedule of the training recipe (Appendix F): a linear ramp
    from 0 over the first warmup_frac of training, then lambda_max."""
    warm = warmup_frac * total_steps
    if warm <= 0 or step >= warm:
        return lambda_max
    return lambda_max * max(step, 0) / warm
