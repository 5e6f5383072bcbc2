"""Seeded synthetic inputs for the view-masked attention and the token log-prob.

This module only *draws* inputs; it holds none of the method's arithmetic (no
views, no key lifetimes, no masks, no softmax).  Both the HIP library's callers
and the CPU oracle's tests take their inputs from here, so both sides see the
same bytes.

A trajectory is described the way the paper's rollout record describes it
(Appendix E.1, "one record per rollout", and Definition "trajectory tree" in
Appendix B.1): a physical token range plus an ordered list of edits
``(J_k, E_k)``.  Positions are *query rows*: edit k is applied before row
``J_k`` is evaluated, so rows ``>= J_k`` no longer see ``E_k``.  Summary blocks
are ordinary tokens born at ``[J_k, J_k + s_k)`` (the harness-written summary of
the black-box figure sits in the post-edit view); they are carried as metadata.

Workload recipes (structure drawn with ``numpy.random.default_rng``):

* ``tiny``     1 x 512 tokens, 1/1 heads, d=64, fp32; junctions 192 and 384,
               each evicting one run of 96 consecutive live non-summary tokens
               (start uniform over valid starts); 32 summary tokens per edit.
* ``medium``   1 x 8192, 16/4 heads, d=128, bf16; 6 junctions drawn uniformly
               (spacing >= 256) in [512, N-256); each edit evicts 1-4 disjoint
               runs of the live view totalling U[0.3, 0.6] of it; 256 summary.
* ``b4x32k``   4 x 32768, 28/4 heads, d=128, bf16; 16 junctions per trajectory
               in [2560, N-1024), spacing >= 1024; one run of U[512, 4096]
               live non-prompt tokens; summary U[256, 1024]; the first 2048
               tokens of each trajectory are never evicted.
* ``long128k`` 1 x 131072, 64/8 heads, d=128, bf16; 40 junctions in
               [2560, N-2048), spacing >= 2048; one run of U[0.5, 0.8] of the
               live non-prompt history; summary U[512, 2048]; prompt 2048.
* ``lmhead``   32768 tokens, hidden 3584, vocab 152064; h ~ N(0,1),
               W ~ N(0, 0.02^2), targets uniform, logp_old ~ N(-2, 1),
               dlogp ~ N(0, 1), eps = 0.2.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

Span = Tuple[int, int]


@dataclass(frozen=True)
class Edit:
    junction: int                 # J_k: first row evaluated under the post-edit view
    evict: Tuple[Span, ...]       # E_k as disjoint, sorted, half-open physical spans
    summary: Span = (0, 0)        # metadata only; (b, b) means none
    restore: Tuple[Span, ...] = ()  # earlier-evicted spans live again from J_k on


@dataclass(frozen=True)
class Trajectory:
    begin: int
    end: int
    edits: Tuple[Edit, ...] = ()


@dataclass(frozen=True)
class AttnWorkload:
    name: str
    n_traj: int
    traj_len: int
    n_heads_q: int
    n_heads_kv: int
    head_dim: int
    dtype: str                    # dtype the inputs are drawn in ("fp32" or "bf16")

    @property
    def total_tokens(self) -> int:
        return self.n_traj * self.traj_len


@dataclass(frozen=True)
class LogprobWorkload:
    name: str
    n_tokens: int
    hidden: int
    vocab: int
    eps_low: float = 0.2
    eps_high: float = 0.2


ATTN_WORKLOADS = {
    "tiny": AttnWorkload("tiny", 1, 512, 1, 1, 64, "fp32"),
    "medium": AttnWorkload("medium", 1, 8192, 16, 4, 128, "bf16"),
    "b4x32k": AttnWorkload("b4x32k", 4, 32768, 28, 4, 128, "bf16"),
    "long128k": AttnWorkload("long128k", 1, 131072, 64, 8, 128, "bf16"),
}
LOGPROB_WORKLOADS = {
    "lmhead": LogprobWorkload("lmhead", 32768, 3584, 152064),
}
_WORKLOAD_INDEX = {"tiny": 0, "medium": 1, "b4x32k": 2, "long128k": 3, "lmhead": 4}


# --------------------------------------------------------------------------
# small sampling helpers
# --------------------------------------------------------------------------
def _composition(rng: np.random.Generator, total: int, parts: int) -> List[int]:
    """Uniform random split of ``total`` into ``parts`` non-negative integers."""
    if parts == 1:
        return [total]
    cuts = np.sort(rng.choice(total + parts - 1, size=parts - 1, replace=False))
    edges = np.concatenate(([-1], cuts, [total + parts - 1]))
    return [int(x) for x in (np.diff(edges) - 1)]


def _spread_junctions(rng, lo: int, hi: int, k: int, gap: int) -> List[int]:
    """k sorted junctions in [lo, hi) with consecutive spacing >= gap (sort-then-shift)."""
    room = (hi - lo) - (k - 1) * gap
    if room < k:
        raise ValueError("junction range too small")
    base = np.sort(rng.choice(room, size=k, replace=False))
    return [int(lo + b + i * gap) for i, b in enumerate(base)]


def _to_spans(positions: Sequence[int]) -> Tuple[Span, ...]:
    """Group sorted physical positions into maximal half-open runs."""
    spans: List[Span] = []
    for p in (int(x) for x in positions):
        if spans and spans[-1][1] == p:
            spans[-1] = (spans[-1][0], p + 1)
        else:
            spans.append((p, p + 1))
    return tuple(spans)


class _LiveTracker:
    """Which physical tokens of one trajectory the generator has not yet evicted.

    Used only to draw *valid* eviction sets (every evicted token must still be
    live when its edit fires); the oracle re-derives views on its own.
    """

    def __init__(self, begin: int, end: int):
        self.begin = begin
        self.alive = np.ones(end - begin, dtype=bool)
        self.protected = np.zeros(end - begin, dtype=bool)

    def live_before(self, junction: int) -> np.ndarray:
        idx = np.nonzero(self.alive[: junction - self.begin])[0]
        return idx + self.begin

    def kill(self, positions: Sequence[int]) -> None:
        for p in positions:
            assert self.alive[p - self.begin]
            self.alive[p - self.begin] = False

    def dead_before(self, junction: int) -> np.ndarray:
        idx = np.nonzero(~self.alive[: junction - self.begin])[0]
        return idx + self.begin

    def revive(self, positions: Sequence[int]) -> None:
        for p in positions:
            assert not self.alive[p - self.begin]
            self.alive[p - self.begin] = True

    def protect(self, b: int, e: int) -> None:
        self.protected[b - self.begin: e - self.begin] = True

    def is_protected(self, positions: np.ndarray) -> np.ndarray:
        return self.protected[positions - self.begin]


def _valid_run_starts(ok: np.ndarray, n: int) -> np.ndarray:
    """Start indices i such that ok[i:i+n] is all True."""
    if n <= 0 or n > len(ok):
        return np.zeros(0, dtype=np.int64)
    c = np.concatenate(([0], np.cumsum(ok.astype(np.int64))))
    full = (c[n:] - c[:-n]) == n
    return np.nonzero(full)[0]


# --------------------------------------------------------------------------
# per-workload edit recipes
# --------------------------------------------------------------------------
def _edits_tiny(rng, begin: int, length: int) -> Tuple[Edit, ...]:
    tr = _LiveTracker(begin, begin + length)
    edits = []
    for j in (192, 384):
        J = begin + j
        view = tr.live_before(J)
        ok = ~tr.is_protected(view)            # summaries are not evictable here
        starts = _valid_run_starts(ok, 96)
        s = int(rng.choice(starts))
        run = view[s: s + 96]
        tr.kill(run)
        summ = (J, J + 32)
        tr.protect(*summ)
        edits.append(Edit(J, _to_spans(run), summ))
    return tuple(edits)


def _edits_medium(rng, begin: int, length: int) -> Tuple[Edit, ...]:
    tr = _LiveTracker(begin, begin + length)
    edits = []
    for J in _spread_junctions(rng, begin + 512, begin + length - 256, 6, 256):
        view = tr.live_before(J)
        nv = len(view)
        n_runs = int(rng.integers(1, 5))
        frac = float(rng.uniform(0.3, 0.6))
        x = max(n_runs, int(round(frac * nv)))
        lens = [1 + p for p in _composition(rng, x - n_runs, n_runs)]
        keep = nv - x
        gaps = _composition(rng, keep - (n_runs - 1), n_runs + 1)
        for i in range(1, n_runs):
            gaps[i] += 1                        # runs stay separate
        pos, evicted = 0, []
        for i in range(n_runs):
            pos += gaps[i]
            evicted.extend(view[pos: pos + lens[i]].tolist())
            pos += lens[i]
        tr.kill(evicted)
        edits.append(Edit(J, _to_spans(sorted(evicted)), (J, J + 256)))
    return tuple(edits)


def _edits_prompted(rng, begin: int, length: int, n_edits: int, lo: int,
                    hi_margin: int, gap: int, run_len, summ_rng) -> Tuple[Edit, ...]:
    tr = _LiveTracker(begin, begin + length)
    tr.protect(begin, begin + 2048)
    edits = []
    for J in _spread_junctions(rng, begin + lo, begin + length - hi_margin, n_edits, gap):
        view = tr.live_before(J)
        cand = view[~tr.is_protected(view)]     # prompt tokens are never evicted
        n = min(run_len(rng, len(cand)), len(cand))
        evicted: List[int] = []
        if n > 0:
            s = int(rng.integers(0, len(cand) - n + 1))
            evicted = cand[s: s + n].tolist()
            tr.kill(evicted)
        s_len = int(rng.integers(summ_rng[0], summ_rng[1] + 1))
        edits.append(Edit(J, _to_spans(evicted), (J, J + s_len)))
    return tuple(edits)


def _edits_b4x32k(rng, begin: int, length: int) -> Tuple[Edit, ...]:
    return _edits_prompted(rng, begin, length, 16, 2560, 1024, 1024,
                           lambda r, n: int(r.integers(512, 4097)), (256, 1024))


def _edits_long128k(rng, begin: int, length: int) -> Tuple[Edit, ...]:
    return _edits_prompted(rng, begin, length, 40, 2560, 2048, 2048,
                           lambda r, n: int(round(float(r.uniform(0.5, 0.8)) * n)),
                           (512, 2048))


_RECIPES = {"tiny": _edits_tiny, "medium": _edits_medium,
            "b4x32k": _edits_b4x32k, "long128k": _edits_long128k}


def make_trajectories(workload: str, seed: int = 0) -> List[Trajectory]:
    """The packed trajectories of an attention workload (back-to-back)."""
    wl = ATTN_WORKLOADS[workload]
    rng = np.random.default_rng([_WORKLOAD_INDEX[workload], seed])
    out = []
    for t in range(wl.n_traj):
        b = t * wl.traj_len
        out.append(Trajectory(b, b + wl.traj_len, _RECIPES[workload](rng, b, wl.traj_len)))
    return out


def random_trajectories(rng: np.random.Generator, lengths: Sequence[int],
                        max_edits: int = 4, max_span: int = 6,
                        summary_max: int = 3, restore_max: int = 0) -> List[Trajectory]:
    """Small random trajectories for property tests (any valid record).

    With restore_max > 0 an edit may also bring back up to that many tokens
    evicted by earlier edits (offload / retrieve, keys with several live
    intervals); a token is never evicted and restored by the same edit."""
    out, b = [], 0
    for n in lengths:
        tr = _LiveTracker(b, b + n)
        k = int(rng.integers(0, max_edits + 1)) if n > 2 else 0
        js = sorted(set(int(x) for x in rng.integers(b + 1, b + n, size=k))) if k else []
        edits = []
        for J in js:
            dead = tr.dead_before(J)
            n_rs = int(rng.integers(0, min(restore_max, len(dead)) + 1)) if restore_max else 0
            rs = sorted(rng.choice(dead, size=n_rs, replace=False).tolist()) if n_rs else []
            view = tr.live_before(J)
            n_ev = int(rng.integers(0, min(max_span, len(view)) + 1))
            ev = sorted(rng.choice(view, size=n_ev, replace=False).tolist()) if n_ev else []
            tr.kill(ev)
            tr.revive(rs)
            s = int(rng.integers(0, summary_max + 1))
            edits.append(Edit(J, _to_spans(ev), (J, min(J + s, b + n)), _to_spans(rs)))
        out.append(Trajectory(b, b + n, tuple(edits)))
        b += n
    return out


# --------------------------------------------------------------------------
# tensors
# --------------------------------------------------------------------------
def tensor_seed(workload: str, seed: int) -> int:
    return 1_000_003 * (_WORKLOAD_INDEX.get(workload, 7) + 1) + seed


def make_attn_tensors(workload: str, seed: int = 0, device: str = "cpu",
                      dtype: Optional[torch.dtype] = None,
                      total_tokens: Optional[int] = None):
    """q, k, v, dout ~ N(0, 1) drawn from a seeded torch generator on ``device``.

    Inputs drawn as fp32 are rounded once to bf16 (round-to-nearest-even) when
    ``dtype`` is bf16: the kernels compute in bf16, and the oracle is fed the
    same rounded values.  CPU and GPU generators draw different streams, so a
    test that needs the oracle on GPU-drawn tensors copies them to the host.
    """
    wl = ATTN_WORKLOADS[workload]
    T = total_tokens if total_tokens is not None else wl.total_tokens
    gen = torch.Generator(device=device)
    gen.manual_seed(tensor_seed(workload, seed))
    out_dtype = dtype if dtype is not None else torch.bfloat16
    shapes = [(T, wl.n_heads_q, wl.head_dim), (T, wl.n_heads_kv, wl.head_dim),
              (T, wl.n_heads_kv, wl.head_dim), (T, wl.n_heads_q, wl.head_dim)]
    out = []
    for s in shapes:
        x = torch.randn(s, generator=gen, device=device, dtype=torch.float32)
        out.append(x.to(out_dtype))
    return tuple(out)


def make_logprob_inputs(n_tokens: int, hidden: int, vocab: int, seed: int = 0,
                        device: str = "cpu", workload: str = "lmhead"):
    """hidden (bf16), weight (bf16), target (int32), logp_old (fp32), dlogp (fp32)."""
    gen = torch.Generator(device=device)
    gen.manual_seed(tensor_seed(workload, seed))
    h = torch.randn((n_tokens, hidden), generator=gen, device=device).to(torch.bfloat16)
    w = (0.02 * torch.randn((vocab, hidden), generator=gen, device=device)).to(torch.bfloat16)
    tgt = torch.randint(0, vocab, (n_tokens,), generator=gen, device=device, dtype=torch.int64)
    old = -2.0 + torch.randn((n_tokens,), generator=gen, device=device)
    g = torch.randn((n_tokens,), generator=gen, device=device)
    return h, w, tgt.to(torch.int32), old.float(), g.float()


def make_grpo_inputs(lengths: Sequence[int], seed: int = 0, logp_noise: float = 0.1,
                     ref_noise: float = 0.05, mask_frac: float = 0.8):
    """Per-token inputs of the GRPO loss for trajectories of the given lengths:
    traj_ptr int32 [n+1], reward fp32 [n] (EM in {0, 0.2, 1}, as the recipe's
    exact-match reward with a format bonus), logp fp32 [T] ~ -2 + N(0, 1),
    logp_old = logp + N(0, logp_noise^2) (so both clip edges and the interior
    occur), logp_ref = logp + N(0, ref_noise^2), loss mask uint8 with the
    given fraction of ones."""
    gen = torch.Generator().manual_seed(tensor_seed("grpo", seed))
    ptr = [0]
    for n in lengths:
        ptr.append(ptr[-1] + int(n))
    T = ptr[-1]
    pick = torch.randint(0, 3, (len(lengths),), generator=gen)
    reward = torch.tensor([0.0, 0.2, 1.0])[pick]
    logp = -2.0 + torch.randn(T, generator=gen)
    old = logp + logp_noise * torch.randn(T, generator=gen)
    ref = logp + ref_noise * torch.randn(T, generator=gen)
    mask = (torch.rand(T, generator=gen) < mask_frac).to(torch.uint8)
    return (torch.tensor(ptr, dtype=torch.int32), reward.float(), logp.float(), old.float(),
            ref.float(), mask)

