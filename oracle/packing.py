"""Branch-replicated packing, per-branch position ids, rotary embedding and a
multi-layer exactness check (test infrastructure only).

The training loop of the paper does not run the physical-union form of Eq.
"4d-mask-def" directly: it materialises one copy of each shared-trunk token
per branch, packs the copies into one sequence under a block-diagonal causal
mask and restarts position ids per branch (Appendix G; Section 6.1's note on
the 4D mask's implementation).  Each copy's hidden state is then computed
from its branch-local prefix alone, which is what makes a stack of layers
exact (the union form is exact for one layer only: a key between an evicted
span and its junction carries, from the second layer on, a hidden state
computed with the span visible).

Layout.  For every trajectory, for every branch layer k (rows [J_k, J_{k+1}),
Appendix B.1), one segment = the keys live just before J_k in physical order,
followed by the rows J_k .. J_{k+1}-1.  Per packed slot:
  src     physical token the slot copies,
  pos     its index inside the segment (the position the token had in the
          live context when the layer's rows were decoded),
  owner   1 for the layer's own rows (they carry their row's loss), 0 for the
          copies of trunk tokens,
  target  the physical row whose token the slot predicts (src + 1 for an
          owner slot that is not its trajectory's last row), else -1.
The packed length is sum over layers of l_k >= L (Appendix G).

Rotary embedding (reading: the rotate-half form with base theta, as the
Qwen3 family uses): for i < d/2, f_i = theta^(-2i/d), a = pos * f_i,
  y_i = x_i cos a - x_{i+d/2} sin a,  y_{i+d/2} = x_{i+d/2} cos a + x_i sin a.

Shared trunk (LogitTree with the trunk's keys and values cached, Section
4.1): branch k stores only the suffix of S_k after the prefix it shares with
S_{k-1}; its rows attend to that prefix where an earlier branch stored it.

Toy model for the exactness check: n_layers of multi-head attention with RoPE
on q and k and a residual, x <- x + Attn(x) Wo, no other sublayers.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence

import torch

from . import views as V


def branch_pack(trajs: Sequence) -> Dict[str, list]:
    src: List[int] = []
    pos: List[int] = []
    owner: List[int] = []
    target: List[int] = []
    seg_begin: List[int] = [0]
    for tr in trajs:
        for first, end, before in V.branch_layers(tr):
            seq = list(before) + list(range(first, end))
            for p, j in enumerate(seq):
                src.append(j)
                pos.append(p)
                own = j >= first
                owner.append(1 if own else 0)
                target.append(j + 1 if own and j + 1 < tr.end else -1)
            seg_begin.append(len(src))
    return {"src": src, "pos": pos, "owner": owner, "target": target, "seg_begin": seg_begin}


def shared_trunk_pack(trajs: Sequence) -> Dict[str, list]:
    """LogitTree with the shared trunk cached (Section 4.1): consecutive branch
    sequences S_{k-1}, S_k agree on their first d_k tokens (the tokens before
    the first one edit k removes), at the same positions; branch k stores only
    S_k[d_k:] and reads its prefix from the slots of earlier branches.

    Returns the layout of ``branch_pack`` plus ``views``: for every slot, the
    slots holding S_k[0 .. pos] of its branch k (what its row attends to)."""
    src: List[int] = []
    pos: List[int] = []
    owner: List[int] = []
    target: List[int] = []
    views: List[List[int]] = []
    seg_begin: List[int] = [0]
    for tr in trajs:
        prev_seq: List[int] = []
        prev_slots: List[int] = []
        for k, (first, end, before) in enumerate(V.branch_layers(tr)):
            seq = list(before) + list(range(first, end))
            d = 0
            if k > 0:
                while d < min(len(seq), len(prev_seq)) and seq[d] == prev_seq[d]:
                    d += 1
            slots = prev_slots[:d]
            for p in range(d, len(seq)):
                j = seq[p]
                slots.append(len(src))
                src.append(j)
                pos.append(p)
                own = j >= first
                owner.append(1 if own else 0)
                target.append(j + 1 if own and j + 1 < tr.end else -1)
                views.append(list(slots))
            seg_begin.append(len(src))
            prev_seq, prev_slots = seq, slots
    return {"src": src, "pos": pos, "owner": owner, "target": target,
            "seg_begin": seg_begin, "views": views}


def views_mask(views: Sequence[Sequence[int]]) -> torch.Tensor:
    """N x N: slot i sees slot j iff j is in views[i]."""
    n = len(views)
    M = torch.zeros(n, n, dtype=torch.bool)
    for i, vs in enumerate(views):
        M[i, list(vs)] = True
    return M


def block_causal_mask(seg_begin: Sequence[int]) -> torch.Tensor:
    """N x N: slot i sees slot j iff both lie in one segment and j <= i."""
    n = seg_begin[-1]
    M = torch.zeros(n, n, dtype=torch.bool)
    for b, e in zip(seg_begin[:-1], seg_begin[1:]):
        M[b:e, b:e] = torch.tril(torch.ones(e - b, e - b, dtype=torch.bool))
    return M


def rope(x: torch.Tensor, pos, theta: float, inverse: bool = False) -> torch.Tensor:
    """x [N, H, d] rotated by each row's position (inverse: by minus it)."""
    N, H, d = x.shape
    half = d // 2
    xd = x.to(torch.float64)
    p = torch.as_tensor(pos, dtype=torch.float64).reshape(N, 1)
    i = torch.arange(half, dtype=torch.float64)
    a = p * theta ** (-2.0 * i / d)                  # [N, half]
    if inverse:
        a = -a
    c, s = torch.cos(a)[:, None, :], torch.sin(a)[:, None, :]
    lo, hi = xd[..., :half], xd[..., half:]
    return torch.cat([lo * c - hi * s, hi * c + lo * s], dim=-1)


def rope_complex(x: torch.Tensor, pos, theta: float) -> torch.Tensor:
    """The same rotation written as a complex product (pairs (i, i + d/2))."""
    N, H, d = x.shape
    half = d // 2
    z = torch.complex(x[..., :half].to(torch.float64), x[..., half:].to(torch.float64))
    p = torch.as_tensor(pos, dtype=torch.float64).reshape(N, 1, 1)
    f = torch.tensor([theta ** (-2.0 * i / d) for i in range(half)], dtype=torch.float64)
    w = torch.polar(torch.ones_like(p * f), p * f)
    r = z * w
    return torch.cat([r.real, r.imag], dim=-1)


def _attend(x, mask, pos, params, n_heads, head_dim, theta):
    """One residual attention layer over rows x [n, W] with a boolean mask."""
    q = (x @ params["wq"]).reshape(-1, n_heads, head_dim)
    k = (x @ params["wk"]).reshape(-1, n_heads, head_dim)
    v = (x @ params["wv"]).reshape(-1, n_heads, head_dim)
    if theta > 0:
        q, k = rope(q, pos, theta), rope(k, pos, theta)
    s = torch.einsum("ihd,jhd->hij", q, k) / math.sqrt(head_dim)
    s = s.masked_fill(~mask[None], float("-inf"))
    o = torch.einsum("hij,jhd->ihd", torch.softmax(s, dim=-1), v)
    return x + o.reshape(x.shape[0], -1) @ params["wo"]


def toy_logittree(trajs, x0, layers, n_heads, head_dim, theta) -> torch.Tensor:
    """Every branch layer forwarded as its own sequence through the whole
    stack (Section 4.1); each physical row keeps the output of its own layer."""
    out = torch.zeros(x0.shape, dtype=torch.float64)
    for tr in trajs:
        for first, end, before in V.branch_layers(tr):
            seq = list(before) + list(range(first, end))
            n = len(seq)
            x = x0.to(torch.float64)[seq]
            mask = torch.tril(torch.ones(n, n, dtype=torch.bool))
            for prm in layers:
                x = _attend(x, mask, list(range(n)), prm, n_heads, head_dim, theta)
            out[first:end] = x[len(before):]
    return out


def toy_packed(trajs, x0, layers, n_heads, head_dim, theta) -> torch.Tensor:
    """The packed stream: copies gathered by src, one forward under the
    block-diagonal mask with per-branch positions, owner rows scattered back."""
    pk = branch_pack(trajs)
    x = x0.to(torch.float64)[pk["src"]]
    mask = block_causal_mask(pk["seg_begin"])
    for prm in layers:
        x = _attend(x, mask, pk["pos"], prm, n_heads, head_dim, theta)
    out = torch.zeros(x0.shape, dtype=torch.float64)
    own = torch.tensor(pk["owner"], dtype=torch.bool)
    out[torch.tensor(pk["src"])[own]] = x[own]
    return out


def toy_shared_trunk(trajs, x0, layers, n_heads, head_dim, theta) -> torch.Tensor:
    """The shared-trunk stream: each branch's new tokens gathered once, one
    forward in which every slot attends to its branch prefix, owner rows
    scattered back."""
    pk = shared_trunk_pack(trajs)
    x = x0.to(torch.float64)[pk["src"]]
    mask = views_mask(pk["views"])
    for prm in layers:
        x = _attend(x, mask, pk["pos"], prm, n_heads, head_dim, theta)
    out = torch.zeros(x0.shape, dtype=torch.float64)
    own = torch.tensor(pk["owner"], dtype=torch.bool)
    out[torch.tensor(pk["src"])[own]] = x[own]
    return out


def toy_union(trajs, x0, layers, n_heads, head_dim, theta, positions=None) -> torch.Tensor:
    """The physical-union form over every layer (exact for one layer only)."""
    from .attention import visibility
    M = visibility(trajs)
    T = x0.shape[0]
    pos = list(range(T)) if positions is None else positions
    x = x0.to(torch.float64)
    for prm in layers:
        x = _attend(x, M, pos, prm, n_heads, head_dim, theta)
    return x


def unpack_sum(pack: Dict[str, list], g: torch.Tensor, T: int) -> torch.Tensor:
    """Gradient of a packed tensor back to the physical tokens: the sum over
    each token's copies (the adjoint of the gather by src)."""
    out = torch.zeros((T,) + tuple(g.shape[1:]), dtype=torch.float64)
    out.index_add_(0, torch.tensor(pack["src"]), g.to(torch.float64))
    return out
