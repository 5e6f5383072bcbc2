"""View-masked attention, the slow and obvious way (test infrastructure only).

Two independent forms of the same function:

* ``logittree``: for every branch layer of every trajectory, build the layer's
  own sequence (keys live before the layer, then the layer's rows) and run
  ordinary causal softmax attention on it, keeping only the layer's rows.  This
  is LogitTree (Section 4.1, Eq. "logittree-def"; per-branch loss mask keeps
  each row on exactly one branch).  Gradients come from autograd through every
  branch, with shared Q/K/V leaves accumulating across branches (Proposition
  "sft_tree", Appendix C.1).
* ``dense``: one T x T boolean mask built from the replayed views and a masked
  softmax over the packed union (Eq. "4d-mask-def", Section 4.2).  Tiny inputs.

By the materialisation-equivalence theorem (Section 4.3; Appendix C.3) the two
agree up to floating-point association order.

Shapes: q [T, Hq, d], k/v [T, Hkv, d]; query head h reads KV head h // (Hq/Hkv).
Outputs: O [T, Hq, d] and LSE [Hq, T] (natural log); softmax scale 1/sqrt(d)
unless given.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import torch

from . import views as _views


def _expand_kv(x: torch.Tensor, hq: int) -> torch.Tensor:
    g = hq // x.shape[1]
    return x.repeat_interleave(g, dim=1)


def _check(q, k, v):
    T, hq, d = q.shape
    if k.shape != v.shape or k.shape[0] != T or k.shape[2] != d or hq % k.shape[1]:
        raise ValueError("bad attention shapes")


def logittree(trajs: Sequence, q, k, v, scale: Optional[float] = None,
              dtype=torch.float64, dout=None, heads: Optional[Sequence[int]] = None,
              row_chunk: int = 4096, row_range: Optional[tuple] = None):
    """Forward (and backward when ``dout`` is given) in LogitTree form.

    ``heads`` restricts the computation to a subset of query heads (their KV
    heads follow); ``row_range`` = (r0, r1) keeps only the loss of rows in
    [r0, r1), exactly as a per-branch loss mask would.  Entries outside the
    selection are left zero.  Returns (O, LSE) or (O, LSE, dQ, dK, dV), all in
    ``dtype``.  Because row i only ever reads View(i), restricting the rows to
    those that see key j yields the exact dK_j and dV_j.
    """
    _check(q, k, v)
    T, hq, d = q.shape
    hkv = k.shape[1]
    heads = list(range(hq)) if heads is None else list(heads)
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else scale
    G = hq // hkv

    qf = q.detach().to(dtype)
    kf = k.detach().to(dtype)
    vf = v.detach().to(dtype)
    want_grad = dout is not None
    if want_grad:
        qf.requires_grad_(True)
        kf.requires_grad_(True)
        vf.requires_grad_(True)
        dof = dout.detach().to(dtype)
    hsel = torch.tensor(heads, dtype=torch.long)
    ksel = hsel // G

    O = torch.zeros(T, hq, d, dtype=dtype)
    LSE = torch.zeros(hq, T, dtype=dtype)
    _, trajs = _views.packed(trajs)
    r0, r1 = (0, T) if row_range is None else (int(row_range[0]), int(row_range[1]))
    for traj in trajs:
        if traj.end <= r0 or traj.begin >= r1:
            continue
        for first, end, before in _views.branch_layers(traj):
            nb = len(before)
            lo, hi = max(first, r0), min(end, r1)
            for c0 in range(lo, hi, row_chunk):
                c1 = min(hi, c0 + row_chunk)
                keys = torch.tensor(before + list(range(first, c1)), dtype=torch.long)
                qs = qf[c0:c1][:, hsel]                 # [n, h, d]
                ks = kf[keys][:, ksel]                   # [m, h, d]
                vs = vf[keys][:, ksel]
                s = torch.einsum("nhd,mhd->hnm", qs, ks) * scale
                # causal inside the layer's own sequence: row c0+i sits at
                # sequence index nb + (c0 - first) + i
                qi = nb + (c0 - first) + torch.arange(c1 - c0)
                kj = torch.arange(len(keys))
                s = s.masked_fill(kj[None, None, :] > qi[None, :, None], float("-inf"))
                lse = torch.logsumexp(s, dim=-1)        # [h, n]
                p = torch.exp(s - lse[..., None])
                o = torch.einsum("hnm,mhd->nhd", p, vs)
                if want_grad:
                    (o * dof[c0:c1][:, hsel]).sum().backward()
                O[c0:c1, hsel] = o.detach()
                LSE[hsel, c0:c1] = lse.detach()
    if not want_grad:
        return O, LSE
    return O, LSE, qf.grad, kf.grad, vf.grad


def visibility(trajs: Sequence) -> torch.Tensor:
    """T x T boolean matrix: entry (i, j) is True iff key j is in View(i)."""
    T, trajs = _views.packed(trajs)
    M = torch.zeros(T, T, dtype=torch.bool)
    for traj in trajs:
        for r, lv in _views.replay(traj):
            M[r, torch.tensor(list(lv), dtype=torch.long)] = True
    return M


def dense(trajs: Sequence, q, k, v, scale: Optional[float] = None,
          dtype=torch.float64, dout=None, mask: Optional[torch.Tensor] = None):
    """Dense masked softmax over the packed union (tiny inputs only).

    ``mask`` overrides the visibility matrix (negative controls pass the
    pitfalls' masks here).
    """
    _check(q, k, v)
    T, hq, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else scale
    M = visibility(trajs) if mask is None else mask
    qf = q.detach().to(dtype).requires_grad_(dout is not None)
    kf = k.detach().to(dtype).requires_grad_(dout is not None)
    vf = v.detach().to(dtype).requires_grad_(dout is not None)
    ke, ve = _expand_kv(kf, hq), _expand_kv(vf, hq)
    s = torch.einsum("ihd,jhd->hij", qf, ke) * scale
    s = s.masked_fill(~M[None], float("-inf"))
    lse = torch.logsumexp(s, dim=-1)
    p = torch.exp(s - lse[..., None])
    o = torch.einsum("hij,jhd->ihd", p, ve)
    if dout is None:
        return o.detach(), lse.detach()
    (o * dout.to(dtype)).sum().backward()
    return o.detach(), lse.detach(), qf.grad, kf.grad, vf.grad


def rows(trajs: Sequence, q, k, v, sample_rows: Sequence[int],
         heads: Optional[Sequence[int]] = None, scale: Optional[float] = None,
         dtype=torch.float64):
    """Output and LSE of selected rows, each from its own view (forward only).

    Row r mixes the values of exactly View(r), found by replaying the record.
    Returns O [len(rows), len(heads), d] and LSE [len(heads), len(rows)].
    """
    _check(q, k, v)
    T, hq, d = q.shape
    G = hq // k.shape[1]
    heads = list(range(hq)) if heads is None else list(heads)
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else scale
    want = {}
    for i, r in enumerate(sample_rows):
        want.setdefault(int(r), []).append(i)
    O = torch.zeros(len(sample_rows), len(heads), d, dtype=dtype)
    LSE = torch.zeros(len(heads), len(sample_rows), dtype=dtype)
    _, trajs = _views.packed(trajs)
    for traj in trajs:
        todo = [r for r in want if traj.begin <= r < traj.end]
        if not todo:
            continue
        last = max(todo)
        for r, lv in _views.replay(traj):
            if r in want:
                keys = torch.tensor(list(lv), dtype=torch.long)
                for hi, h in enumerate(heads):
                    qv = q[r, h].to(dtype)
                    kk = k[keys, h // G].to(dtype)
                    vv = v[keys, h // G].to(dtype)
                    s = (kk @ qv) * scale
                    lse = torch.logsumexp(s, 0)
                    o = torch.exp(s - lse) @ vv
                    for i in want[r]:
                        O[i, hi] = o
                        LSE[hi, i] = lse
            if r == last:
                break
    return O, LSE


def row_grads(trajs: Sequence, q, k, v, dout, sample_rows: Sequence[int],
              heads: Optional[Sequence[int]] = None, scale: Optional[float] = None,
              dtype=torch.float64):
    """dQ of selected rows, each from its own view.

    Row i's output depends on q_i only through its own softmax over View(i),
    so dQ_i = scale * sum_j P_ij (dP_ij - D_i) k_j with dP_ij = <dO_i, v_j> and
    D_i = <dO_i, O_i> needs nothing but that view.
    Returns dQ [len(rows), len(heads), d].
    """
    _check(q, k, v)
    T, hq, d = q.shape
    G = hq // k.shape[1]
    heads = list(range(hq)) if heads is None else list(heads)
    scale = 1.0 / math.sqrt(d) if scale is None or scale <= 0 else scale
    want = {}
    for i, r in enumerate(sample_rows):
        want.setdefault(int(r), []).append(i)
    dQ = torch.zeros(len(sample_rows), len(heads), d, dtype=dtype)
    _, trajs = _views.packed(trajs)
    for traj in trajs:
        todo = [r for r in want if traj.begin <= r < traj.end]
        if not todo:
            continue
        last = max(todo)
        for r, lv in _views.replay(traj):
            if r in want:
                keys = torch.tensor(list(lv), dtype=torch.long)
                for hi, h in enumerate(heads):
                    kk = k[keys, h // G].to(dtype)
                    vv = v[keys, h // G].to(dtype)
                    s = (kk @ q[r, h].to(dtype)) * scale
                    p = torch.softmax(s, 0)
                    do = dout[r, h].to(dtype)
                    dp = vv @ do
                    Di = torch.dot(p @ vv, do)
                    g = scale * ((p * (dp - Di)) @ kk)
                    for i in want[r]:
                        dQ[i, hi] = g
            if r == last:
                break
    return dQ
