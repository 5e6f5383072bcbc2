"""Python binding of libmv: argument marshalling only.

Every computation runs in libmv (the HIP kernels and the C++ mask builder);
this module turns trajectories and torch tensors into the C ABI's plain
pointers and sizes, allocates outputs and workspaces with torch, and raises
``MVError`` on any non-OK status.  If libmv.so has not been built the import
fails loudly: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmv.so")


class MVError(RuntimeError):
    def __init__(self, status: int, name: str, message: str):
        super().__init__(f"{name}: {message}")
        self.status = status
        self.name = name


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"libmv.so not found at {_LIB_PATH}; run "
                          "`python -m paper_2609_00865_amd.build` (or __graft_entry__.build())")
    return ctypes.CDLL(_LIB_PATH)


_lib = _load()


class Span(ctypes.Structure):
    _fields_ = [("begin", ctypes.c_int32), ("end", ctypes.c_int32)]


class EditC(ctypes.Structure):
    _fields_ = [("junction", ctypes.c_int32), ("n_evict", ctypes.c_int32),
                ("evict", ctypes.POINTER(Span)), ("summary", Span),
                ("n_restore", ctypes.c_int32), ("restore", ctypes.POINTER(Span))]


class TrajectoryC(ctypes.Structure):
    _fields_ = [("begin", ctypes.c_int32), ("end", ctypes.c_int32),
                ("n_edits", ctypes.c_int32), ("edits", ctypes.POINTER(EditC))]


class MaskStats(ctypes.Structure):
    _fields_ = [("visible_pairs", ctypes.c_int64), ("total_tokens", ctypes.c_int32),
                ("max_view", ctypes.c_int32), ("n_segments", ctypes.c_int32),
                ("tiles_full", ctypes.c_int32), ("tiles_partial", ctypes.c_int32),
                ("tiles_skipped", ctypes.c_int32), ("bwd_items", ctypes.c_int32),
                ("bwd_partial_slots", ctypes.c_int32), ("n_leaves", ctypes.c_int32),
                ("fwd_tile_pairs", ctypes.c_int64), ("bwd_tile_pairs", ctypes.c_int64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class AttnShape(ctypes.Structure):
    _fields_ = [("total_tokens", ctypes.c_int32), ("n_heads_q", ctypes.c_int32),
                ("n_heads_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float)]


class LogprobShape(ctypes.Structure):
    _fields_ = [("n_tokens", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("eps_low", ctypes.c_float),
                ("eps_high", ctypes.c_float)]


class PackStats(ctypes.Structure):
    _fields_ = [("total_tokens", ctypes.c_int32), ("n_packed", ctypes.c_int32),
                ("n_segments", ctypes.c_int32), ("max_copies", ctypes.c_int32),
                ("causal_pairs", ctypes.c_int64)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


class KLShape(ctypes.Structure):
    _fields_ = [("n_leaves", ctypes.c_int32), ("hidden", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("n_rows_teacher", ctypes.c_int32),
                ("n_rows_student", ctypes.c_int32)]


class GrpoShape(ctypes.Structure):
    _fields_ = [("n_tokens", ctypes.c_int32), ("n_traj", ctypes.c_int32),
                ("group_size", ctypes.c_int32), ("eps_low", ctypes.c_float),
                ("eps_high", ctypes.c_float), ("beta", ctypes.c_float),
                ("adv_eps", ctypes.c_float)]


GRPO_STATS = ["loss", "logdiff", "clip_frac_low", "clip_frac_high", "kl_ref", "ratio_mean",
              "n_loss_tokens", "adv_abs_mean"]

_vp, _sz, _i32, _f32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_float
_P = ctypes.POINTER


def _sig(name, res, *args):
    fn = getattr(_lib, name)
    fn.restype = res
    fn.argtypes = list(args)
    return fn


mv_status_string = _sig("mv_status_string", ctypes.c_char_p, ctypes.c_int)
mv_last_error = _sig("mv_last_error", ctypes.c_char_p)
mv_version = _sig("mv_version", _i32)
mv_build_view_mask = _sig("mv_build_view_mask", ctypes.c_int, _P(TrajectoryC), _i32, _i32,
                          _P(_vp))
mv_build_view_mask_tiled = _sig("mv_build_view_mask_tiled", ctypes.c_int, _P(TrajectoryC), _i32,
                                _i32, _i32, _i32, _P(_vp))
TILE_Q, TILE_K = 128, 64   # the forward / dQ tile shape the kernels are built for
mv_build_view_mask_kind = _sig("mv_build_view_mask_kind", ctypes.c_int, _P(TrajectoryC), _i32,
                               _i32, _i32, _P(_vp))
mv_view_mask_leaves = _sig("mv_view_mask_leaves", ctypes.c_int, _vp, _vp, _vp, _vp, _i32,
                           _P(_i32))
mv_view_mask_intervals = _sig("mv_view_mask_intervals", ctypes.c_int, _vp, _vp, _vp, _i32,
                              _P(_i32))
mv_view_mask_device_bytes = _sig("mv_view_mask_device_bytes", _sz, _vp)
mv_view_mask_upload = _sig("mv_view_mask_upload", ctypes.c_int, _vp, _vp, _sz, _vp)
mv_view_mask_stats = _sig("mv_view_mask_stats", ctypes.c_int, _vp, _P(MaskStats))
mv_view_mask_death = _sig("mv_view_mask_death", ctypes.c_int, _vp, _vp)
mv_view_mask_materialize = _sig("mv_view_mask_materialize", ctypes.c_int, _vp, _i32, _i32, _vp,
                                _vp)
mv_view_mask_materialize_host = _sig("mv_view_mask_materialize_host", ctypes.c_int, _vp, _i32,
                                     _i32, _vp)
mv_view_mask_free = _sig("mv_view_mask_free", None, _vp)
mv_attn_fwd = _sig("mv_attn_fwd", ctypes.c_int, _vp, _P(AttnShape), _vp, _vp, _vp, _vp, _vp,
                   _vp)
mv_attn_bwd_workspace_bytes = _sig("mv_attn_bwd_workspace_bytes", _sz, _vp, _P(AttnShape))
mv_attn_bwd = _sig("mv_attn_bwd", ctypes.c_int, _vp, _P(AttnShape), _vp, _vp, _vp, _vp, _vp,
                   _vp, _vp, _vp, _vp, _vp, _sz, _vp)
mv_attn_bwd_noalloc = _sig("mv_attn_bwd_noalloc", ctypes.c_int, _vp, _P(AttnShape), _vp, _vp, _vp,
                           _vp, _vp, _vp, _vp, _vp, _vp, _vp)
mv_token_logprob_workspace_bytes = _sig("mv_token_logprob_workspace_bytes", _sz,
                                        _P(LogprobShape))
mv_token_logprob = _sig("mv_token_logprob", ctypes.c_int, _P(LogprobShape), _vp, _vp, _vp, _vp,
                        _vp, _vp, _vp, _vp, _vp, _sz, _vp)
mv_token_logprob_bwd_workspace_bytes = _sig("mv_token_logprob_bwd_workspace_bytes", _sz,
                                            _P(LogprobShape))
mv_token_logprob_bwd = _sig("mv_token_logprob_bwd", ctypes.c_int, _P(LogprobShape), _vp, _vp,
                            _vp, _vp, _vp, _vp, _vp, _sz, _vp)
mv_token_logprob_dweight = _sig("mv_token_logprob_dweight", ctypes.c_int, _P(LogprobShape), _vp,
                                _vp, _sz, _vp, _vp)
mv_token_logprob_bad_targets = _sig("mv_token_logprob_bad_targets", ctypes.c_int, _vp, _P(_i32),
                                    _vp)
mv_ppo_clip_dlogp = _sig("mv_ppo_clip_dlogp", ctypes.c_int, _i32, _vp, _vp, _f32, _f32, _f32,
                         _vp, _vp)
mv_build_branch_pack = _sig("mv_build_branch_pack", ctypes.c_int, _P(TrajectoryC), _i32, _i32,
                            _P(_vp))
mv_build_shared_trunk_pack = _sig("mv_build_shared_trunk_pack", ctypes.c_int, _P(TrajectoryC), _i32,
                                  _i32, _P(_vp))
mv_branch_pack_stats = _sig("mv_branch_pack_stats", ctypes.c_int, _vp, _P(PackStats))
mv_branch_pack_layout = _sig("mv_branch_pack_layout", ctypes.c_int, _vp, _vp, _vp, _vp, _vp, _vp)
mv_branch_pack_mask = _sig("mv_branch_pack_mask", _vp, _vp)
mv_branch_pack_device_bytes = _sig("mv_branch_pack_device_bytes", _sz, _vp)
mv_branch_pack_upload = _sig("mv_branch_pack_upload", ctypes.c_int, _vp, _vp, _sz, _vp)
mv_branch_pack_free = _sig("mv_branch_pack_free", None, _vp)
mv_pack_rows = _sig("mv_pack_rows", ctypes.c_int, _vp, _vp, _i32, _vp, _vp)
mv_unpack_rows_sum = _sig("mv_unpack_rows_sum", ctypes.c_int, _vp, _vp, _i32, _i32, _vp, _vp)
mv_rope = _sig("mv_rope", ctypes.c_int, _vp, _vp, _i32, _i32, _f32, _i32, _vp, _vp)
mv_pack_rows_rope = _sig("mv_pack_rows_rope", ctypes.c_int, _vp, _vp, _i32, _i32, _f32, _vp, _vp)
mv_unpack_rows_sum_rope = _sig("mv_unpack_rows_sum_rope", ctypes.c_int, _vp, _vp, _i32, _i32,
                               _f32, _i32, _vp, _vp)
mv_grpo_loss_workspace_bytes = _sig("mv_grpo_loss_workspace_bytes", _sz, _P(GrpoShape))
mv_grpo_loss = _sig("mv_grpo_loss", ctypes.c_int, _P(GrpoShape), _vp, _vp, _vp, _vp, _vp, _vp,
                    _vp, _vp, _vp, _vp, _sz, _vp)
mv_token_logprob_grpo_workspace_bytes = _sig("mv_token_logprob_grpo_workspace_bytes", _sz,
                                             _P(LogprobShape), _P(GrpoShape))
mv_token_logprob_grpo = _sig("mv_token_logprob_grpo", ctypes.c_int, _P(LogprobShape),
                             _P(GrpoShape), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                             _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp)
mv_sdcc_kl_workspace_bytes = _sig("mv_sdcc_kl_workspace_bytes", _sz, _P(KLShape))
mv_sdcc_kl = _sig("mv_sdcc_kl", ctypes.c_int, _P(KLShape), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                  _vp, _sz, _vp)
mv_sdcc_kl_bwd_workspace_bytes = _sig("mv_sdcc_kl_bwd_workspace_bytes", _sz, _P(KLShape))
mv_sdcc_kl_bwd = _sig("mv_sdcc_kl_bwd", ctypes.c_int, _P(KLShape), _vp, _vp, _vp, _vp, _vp, _vp,
                      _vp, _vp, _vp, _vp, _sz, _vp)
mv_sdcc_lambda = _sig("mv_sdcc_lambda", _f32, _i32, _i32, _f32, _f32)

mv_profile_enable = _sig("mv_profile_enable", ctypes.c_int, _i32)
mv_profile_read = _sig("mv_profile_read", ctypes.c_int, ctypes.c_char_p, _P(ctypes.c_double),
                       _P(_i32))

EXPORTED = ["mv_status_string", "mv_last_error", "mv_version", "mv_build_view_mask",
            "mv_view_mask_device_bytes", "mv_view_mask_upload", "mv_view_mask_stats",
            "mv_view_mask_death", "mv_view_mask_materialize", "mv_view_mask_materialize_host",
            "mv_view_mask_free", "mv_attn_fwd", "mv_attn_bwd_workspace_bytes", "mv_attn_bwd",
            "mv_token_logprob_workspace_bytes", "mv_token_logprob",
            "mv_token_logprob_bwd_workspace_bytes", "mv_token_logprob_bwd", "mv_ppo_clip_dlogp",
            "mv_build_view_mask_kind", "mv_view_mask_leaves", "mv_sdcc_kl_workspace_bytes",
            "mv_sdcc_kl", "mv_sdcc_kl_bwd_workspace_bytes", "mv_sdcc_kl_bwd", "mv_sdcc_lambda",
            "mv_grpo_loss_workspace_bytes", "mv_grpo_loss", "mv_build_branch_pack",
            "mv_branch_pack_stats", "mv_branch_pack_layout", "mv_branch_pack_mask",
            "mv_branch_pack_device_bytes", "mv_branch_pack_upload", "mv_branch_pack_free",
            "mv_pack_rows", "mv_unpack_rows_sum", "mv_rope", "mv_token_logprob_dweight",
            "mv_view_mask_intervals", "mv_token_logprob_bad_targets", "mv_attn_bwd_noalloc",
            "mv_build_shared_trunk_pack", "mv_token_logprob_grpo_workspace_bytes",
            "mv_token_logprob_grpo", "mv_pack_rows_rope", "mv_unpack_rows_sum_rope",
            "mv_build_view_mask_tiled",
            "mv_profile_enable", "mv_profile_read"]

VIEW_LIVE, VIEW_FINAL = 0, 1


def check(status: int) -> None:
    if status != 0:
        raise MVError(status, mv_status_string(status).decode(), mv_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _aligned_buffer(nbytes: int, device) -> tuple:
    """A uint8 device tensor and the first 256-byte aligned address inside it."""
    buf = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    addr = (buf.data_ptr() + 255) & ~255
    return buf, addr


# ---------------------------------------------------------------------------
# view mask
# ---------------------------------------------------------------------------
def _trajectories_c(trajectories: Sequence):
    """ctypes array of mv_trajectory plus the arrays it points into."""
    keep = []
    trajs = (TrajectoryC * len(trajectories))()
    for ti, t in enumerate(trajectories):
        edits = (EditC * max(1, len(t.edits)))()
        for ei, e in enumerate(t.edits):
            spans = (Span * max(1, len(e.evict)))()
            for si, (b, x) in enumerate(e.evict):
                spans[si] = Span(int(b), int(x))
            keep.append(spans)
            rest = tuple(getattr(e, "restore", ()))
            rspans = (Span * max(1, len(rest)))()
            for si, (b, x) in enumerate(rest):
                rspans[si] = Span(int(b), int(x))
            keep.append(rspans)
            summ = getattr(e, "summary", (0, 0))
            edits[ei] = EditC(int(e.junction), len(e.evict), spans,
                              Span(int(summ[0]), int(summ[1])), len(rest), rspans)
        keep.append(edits)
        trajs[ti] = TrajectoryC(int(t.begin), int(t.end), len(t.edits), edits)
    return trajs, keep

class ViewMask:
    """Owns a libmv mask object built from trajectories (host), optionally uploaded."""

    def __init__(self, trajectories: Sequence, total_tokens: Optional[int] = None,
                 kind: int = 0):
        trajs, keep = _trajectories_c(trajectories)
        T = total_tokens if total_tokens is not None else int(trajectories[-1].end)
        handle = ctypes.c_void_p()
        check(mv_build_view_mask_kind(trajs, len(trajectories), T, int(kind),
                                      ctypes.byref(handle)))
        self._h = handle
        self._owned = True
        self.total_tokens = T
        self._dev = None

    @classmethod
    def _borrowed(cls, handle, total_tokens: int, owner) -> "ViewMask":
        """A mask owned by another library object (kept alive through `owner`)."""
        m = cls.__new__(cls)
        m._h = ctypes.c_void_p(handle)
        m._owned = False
        m._owner = owner
        m.total_tokens = total_tokens
        m._dev = None
        return m

    def __del__(self, _free=mv_view_mask_free):
        h = getattr(self, "_h", None)
        if h is not None and h.value and getattr(self, "_owned", False):
            _free(h)
        self._h = None

    @property
    def handle(self):
        return self._h

    def stats(self) -> dict:
        s = MaskStats()
        check(mv_view_mask_stats(self._h, ctypes.byref(s)))
        return s.as_dict()

    def death(self) -> torch.Tensor:
        out = torch.empty(self.total_tokens, dtype=torch.int32)
        check(mv_view_mask_death(self._h, _ptr(out)))
        return out

    def leaves(self):
        """(tokens, teacher_rows, student_rows): int32 host tensors, one entry per leaf."""
        n = ctypes.c_int32()
        check(mv_view_mask_leaves(self._h, None, None, None, 0, ctypes.byref(n)))
        out = [torch.empty(n.value, dtype=torch.int32) for _ in range(3)]
        check(mv_view_mask_leaves(self._h, _ptr(out[0]), _ptr(out[1]), _ptr(out[2]), n.value,
                                  ctypes.byref(n)))
        return tuple(out)

    def intervals(self):
        """(iv_ptr [T + 1], iv [n, 2]): further live intervals of restored keys."""
        n = ctypes.c_int32()
        ptr = torch.empty(self.total_tokens + 1, dtype=torch.int32)
        check(mv_view_mask_intervals(self._h, _ptr(ptr), None, 0, ctypes.byref(n)))
        iv = torch.empty(max(1, 2 * n.value), dtype=torch.int32)
        check(mv_view_mask_intervals(self._h, None, _ptr(iv), n.value, ctypes.byref(n)))
        return ptr, iv[:2 * n.value].view(-1, 2)

    def device_bytes(self) -> int:
        return int(mv_view_mask_device_bytes(self._h))

    def upload(self, device="cuda", stream=None) -> "ViewMask":
        buf, addr = _aligned_buffer(self.device_bytes(), device)
        check(mv_view_mask_upload(self._h, ctypes.c_void_p(addr), self.device_bytes(),
                                  _stream(stream)))
        self._dev = buf
        return self

    def materialize(self, row_begin: int, row_end: int, stream=None) -> torch.Tensor:
        words = (self.total_tokens + 31) // 32
        out = torch.empty((row_end - row_begin) * words, dtype=torch.int32, device="cuda")
        check(mv_view_mask_materialize(self._h, row_begin, row_end, _ptr(out), _stream(stream)))
        return out.view(row_end - row_begin, words)

    def materialize_host(self, row_begin: int, row_end: int) -> torch.Tensor:
        words = (self.total_tokens + 31) // 32
        out = torch.empty((row_end - row_begin) * words, dtype=torch.int32)
        check(mv_view_mask_materialize_host(self._h, row_begin, row_end, _ptr(out)))
        return out.view(row_end - row_begin, words)


def unpack_bits(words: torch.Tensor, total_tokens: int) -> torch.Tensor:
    """[rows, ceil(T/32)] int32 words -> [rows, T] bool (bit j%32 of word j//32)."""
    w = words.to(torch.int64) & 0xFFFFFFFF
    shifts = torch.arange(32, dtype=torch.int64, device=w.device)
    bits = (w[..., None] >> shifts) & 1
    return bits.reshape(words.shape[0], -1)[:, :total_tokens].bool()


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------
def _attn_shape(mask: ViewMask, q, k, scale):
    T, hq, d = q.shape
    return AttnShape(T, hq, k.shape[1], d, float(scale) if scale else 0.0)


def _need_bf16_cuda(*ts):
    for t in ts:
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
            raise ValueError("expected contiguous bf16 CUDA tensors")


def attn_fwd(mask: ViewMask, q, k, v, scale: Optional[float] = None, stream=None):
    _need_bf16_cuda(q, k, v)
    shape = _attn_shape(mask, q, k, scale)
    o = torch.empty_like(q)
    lse = torch.empty((q.shape[1], q.shape[0]), dtype=torch.float32, device=q.device)
    check(mv_attn_fwd(mask.handle, ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                      _ptr(lse), _stream(stream)))
    return o, lse


def attn_bwd_workspace(mask: ViewMask, q, k, scale=None) -> torch.Tensor:
    shape = _attn_shape(mask, q, k, scale)
    n = int(mv_attn_bwd_workspace_bytes(mask.handle, ctypes.byref(shape)))
    return torch.empty(n, dtype=torch.uint8, device=q.device)


def attn_bwd(mask: ViewMask, q, k, v, o, dout, lse, scale: Optional[float] = None,
             workspace: Optional[torch.Tensor] = None, stream=None):
    _need_bf16_cuda(q, k, v, o, dout)
    shape = _attn_shape(mask, q, k, scale)
    ws = workspace if workspace is not None else attn_bwd_workspace(mask, q, k, scale)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    check(mv_attn_bwd(mask.handle, ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                      _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(ws),
                      ws.numel(), _stream(stream)))
    return dq, dk, dv


# Bytes of the static scratch mv_attn_bwd_noalloc works in (mv.h)
ATTN_BWD_NOALLOC_SCRATCH_BYTES = 64 << 20


def attn_bwd_noalloc(mask: ViewMask, q, k, v, o, dout, lse, scale: Optional[float] = None,
                     stream=None, out=None):
    """The backward through mv_attn_bwd_noalloc (no workspace).  `out` =
    (dq, dk, dv) preallocated by the caller; otherwise torch allocates them."""
    _need_bf16_cuda(q, k, v, o, dout)
    shape = _attn_shape(mask, q, k, scale)
    dq, dk, dv = out if out is not None else (torch.empty_like(q), torch.empty_like(k),
                                              torch.empty_like(v))
    check(mv_attn_bwd_noalloc(mask.handle, ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v),
                              _ptr(o), _ptr(dout), _ptr(lse), _ptr(dq), _ptr(dk), _ptr(dv),
                              _stream(stream)))
    return dq, dk, dv


# ---------------------------------------------------------------------------
# token log-prob
# ---------------------------------------------------------------------------
def _lp_shape(hidden, weight, eps_low, eps_high):
    return LogprobShape(hidden.shape[0], hidden.shape[1], weight.shape[0], float(eps_low),
                        float(eps_high))


def token_logprob_workspace(hidden, weight) -> torch.Tensor:
    s = _lp_shape(hidden, weight, 0.2, 0.2)
    n = int(mv_token_logprob_workspace_bytes(ctypes.byref(s)))
    return torch.empty(n, dtype=torch.uint8, device=hidden.device)


def token_logprob(hidden, weight, target, logp_old=None, eps_low=0.2, eps_high=0.2,
                  workspace=None, stream=None):
    _need_bf16_cuda(hidden, weight)
    s = _lp_shape(hidden, weight, eps_low, eps_high)
    T = hidden.shape[0]
    dev = hidden.device
    logp = torch.empty(T, dtype=torch.float32, device=dev)
    lse = torch.empty(T, dtype=torch.float32, device=dev)
    ratio = clipped = None
    if logp_old is not None:
        ratio = torch.empty(T, dtype=torch.float32, device=dev)
        clipped = torch.empty(T, dtype=torch.float32, device=dev)
    ws = workspace if workspace is not None else token_logprob_workspace(hidden, weight)
    check(mv_token_logprob(ctypes.byref(s), _ptr(hidden), _ptr(weight), _ptr(target),
                           _ptr(logp_old), _ptr(logp), _ptr(ratio), _ptr(clipped), _ptr(lse),
                           _ptr(ws), ws.numel(), _stream(stream)))
    return logp, ratio, clipped, lse


def token_logprob_bwd_workspace(hidden, weight) -> torch.Tensor:
    s = _lp_shape(hidden, weight, 0.2, 0.2)
    n = int(mv_token_logprob_bwd_workspace_bytes(ctypes.byref(s)))
    return torch.empty(n, dtype=torch.uint8, device=hidden.device)


def token_logprob_bwd(hidden, weight, target, lse, dlogp, workspace=None, stream=None):
    _need_bf16_cuda(hidden, weight)
    s = _lp_shape(hidden, weight, 0.2, 0.2)
    dh = torch.empty_like(hidden)
    ws = workspace if workspace is not None else token_logprob_bwd_workspace(hidden, weight)
    check(mv_token_logprob_bwd(ctypes.byref(s), _ptr(hidden), _ptr(weight), _ptr(target),
                               _ptr(lse), _ptr(dlogp), _ptr(dh), _ptr(ws), ws.numel(),
                               _stream(stream)))
    return dh


def token_logprob_dweight(hidden, weight, workspace, stream=None):
    """dW = G^T H (fp32 [V, H]) from the G that token_logprob_bwd left in `workspace`."""
    _need_bf16_cuda(hidden, weight)
    s = _lp_shape(hidden, weight, 0.2, 0.2)
    dw = torch.empty(weight.shape, dtype=torch.float32, device=hidden.device)
    check(mv_token_logprob_dweight(ctypes.byref(s), _ptr(hidden), _ptr(workspace),
                                   workspace.numel(), _ptr(dw), _stream(stream)))
    return dw


def token_logprob_bad_targets(workspace, stream=None) -> int:
    """Target ids outside [-1, vocab) that the last token_logprob /
    token_logprob_bwd call on `workspace` met (waits for the stream)."""
    n = ctypes.c_int32()
    check(mv_token_logprob_bad_targets(_ptr(workspace), ctypes.byref(n), _stream(stream)))
    return n.value


def ppo_clip_dlogp(ratio, adv, eps_low=0.2, eps_high=0.2, scale=1.0, stream=None):
    out = torch.empty_like(ratio)
    check(mv_ppo_clip_dlogp(ratio.numel(), _ptr(ratio), _ptr(adv), eps_low, eps_high, scale,
                            _ptr(out), _stream(stream)))
    return out


# ---------------------------------------------------------------------------
# branch-replicated packing
# ---------------------------------------------------------------------------
class BranchPack:
    """Owns a libmv branch packing built from trajectories."""

    def __init__(self, trajectories: Sequence, total_tokens: Optional[int] = None,
                 shared_trunk: bool = False):
        trajs, keep = _trajectories_c(trajectories)
        T = total_tokens if total_tokens is not None else int(trajectories[-1].end)
        handle = ctypes.c_void_p()
        build = mv_build_shared_trunk_pack if shared_trunk else mv_build_branch_pack
        check(build(trajs, len(trajectories), T, ctypes.byref(handle)))
        self._h = handle
        self.total_tokens = T
        st = self.stats()
        self.n_packed = st["n_packed"]
        self.n_segments = st["n_segments"]
        self.mask = ViewMask._borrowed(mv_branch_pack_mask(handle), self.n_packed, self)
        self._dev = None

    def __del__(self, _free=mv_branch_pack_free):
        h = getattr(self, "_h", None)
        if h is not None and h.value:
            _free(h)
            self._h = None

    def stats(self) -> dict:
        s = PackStats()
        check(mv_branch_pack_stats(self._h, ctypes.byref(s)))
        return s.as_dict()

    def layout(self) -> dict:
        N = self.n_packed
        out = {"src": torch.empty(N, dtype=torch.int32), "pos": torch.empty(N, dtype=torch.int32),
               "owner": torch.empty(N, dtype=torch.uint8),
               "target": torch.empty(N, dtype=torch.int32),
               "seg_begin": torch.empty(self.n_segments + 1, dtype=torch.int32)}
        check(mv_branch_pack_layout(self._h, _ptr(out["src"]), _ptr(out["pos"]),
                                    _ptr(out["owner"]), _ptr(out["target"]),
                                    _ptr(out["seg_begin"])))
        return out

    def upload(self, device="cuda", stream=None) -> "BranchPack":
        n = int(mv_branch_pack_device_bytes(self._h))
        buf, addr = _aligned_buffer(n, device)
        check(mv_branch_pack_upload(self._h, ctypes.c_void_p(addr), n, _stream(stream)))
        self._dev = buf
        self.mask.upload(device, stream)
        return self

    @property
    def handle(self):
        return self._h


def pack_rows(pack: BranchPack, x, stream=None):
    """x [T, ...] bf16 -> [n_packed, ...] gathered by each slot's physical token."""
    _need_bf16_cuda(x)
    W = x[0].numel()
    out = torch.empty((pack.n_packed,) + tuple(x.shape[1:]), dtype=x.dtype, device=x.device)
    check(mv_pack_rows(pack.handle, _ptr(x), W, _ptr(out), _stream(stream)))
    return out


def unpack_rows_sum(pack: BranchPack, g, out_fp32: bool = False, stream=None):
    """g [n_packed, ...] bf16 -> [T, ...]: each token's copies summed (fp32 accumulation)."""
    _need_bf16_cuda(g)
    W = g[0].numel()
    out = torch.empty((pack.total_tokens,) + tuple(g.shape[1:]),
                      dtype=torch.float32 if out_fp32 else g.dtype, device=g.device)
    check(mv_unpack_rows_sum(pack.handle, _ptr(g), W, 1 if out_fp32 else 0, _ptr(out),
                             _stream(stream)))
    return out


def rope(pack: BranchPack, x, theta: float = 1e6, inverse: bool = False, out=None, stream=None):
    """Rotary embedding of x [n_packed, H, d] bf16 by each slot's position id."""
    _need_bf16_cuda(x)
    out = torch.empty_like(x) if out is None else out
    check(mv_rope(pack.handle, _ptr(x), x.shape[1], x.shape[2], float(theta),
                  -1 if inverse else 1, _ptr(out), _stream(stream)))
    return out


def pack_rows_rope(pack: BranchPack, x, theta: float = 1e6, stream=None):
    """x [T, H, d] bf16 -> [n_packed, H, d]: gathered by each slot's physical
    token and rotated by the slot's position id in the same pass."""
    _need_bf16_cuda(x)
    out = torch.empty((pack.n_packed,) + tuple(x.shape[1:]), dtype=x.dtype, device=x.device)
    check(mv_pack_rows_rope(pack.handle, _ptr(x), x.shape[1], x.shape[2], float(theta),
                            _ptr(out), _stream(stream)))
    return out


def unpack_rows_sum_rope(pack: BranchPack, g, theta: float = 1e6, out_fp32: bool = False,
                         stream=None):
    """g [n_packed, H, d] bf16 -> [T, H, d]: each copy rotated back by its
    slot's position and the copies of a token summed (fp32), in one pass."""
    _need_bf16_cuda(g)
    out = torch.empty((pack.total_tokens,) + tuple(g.shape[1:]),
                      dtype=torch.float32 if out_fp32 else g.dtype, device=g.device)
    check(mv_unpack_rows_sum_rope(pack.handle, _ptr(g), g.shape[1], g.shape[2], float(theta),
                                  1 if out_fp32 else 0, _ptr(out), _stream(stream)))
    return out


# ---------------------------------------------------------------------------
# GRPO loss and drift diagnostics
# ---------------------------------------------------------------------------
def grpo_loss(traj_ptr, reward, logp, logp_old, logp_ref=None, loss_mask=None, group_size=16,
              eps_low=0.2, eps_high=0.28, beta=0.0, adv_eps=1e-6, workspace=None, stream=None):
    """(advantage [n_traj], dlogp [T], stats fp32 [8] in GRPO_STATS order), all on device."""
    T, n_traj = logp.numel(), reward.numel()
    s = GrpoShape(T, n_traj, int(group_size), float(eps_low), float(eps_high), float(beta),
                  float(adv_eps))
    dev = logp.device
    adv = torch.empty(n_traj, dtype=torch.float32, device=dev)
    dlogp = torch.empty(T, dtype=torch.float32, device=dev)
    stats = torch.empty(8, dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = torch.empty(int(mv_grpo_loss_workspace_bytes(ctypes.byref(s))),
                                dtype=torch.uint8, device=dev)
    check(mv_grpo_loss(ctypes.byref(s), _ptr(traj_ptr), _ptr(reward), _ptr(logp),
                       _ptr(logp_old), _ptr(logp_ref), _ptr(loss_mask), _ptr(adv), _ptr(dlogp),
                       _ptr(stats), _ptr(workspace), workspace.numel(), _stream(stream)))
    return adv, dlogp, stats


def token_logprob_grpo_workspace(hidden, weight, n_traj, group_size=16) -> torch.Tensor:
    s = _lp_shape(hidden, weight, 0.2, 0.2)
    g = GrpoShape(hidden.shape[0], int(n_traj), int(group_size), 0.2, 0.2, 0.0, 1e-6)
    n = int(mv_token_logprob_grpo_workspace_bytes(ctypes.byref(s), ctypes.byref(g)))
    return torch.empty(n, dtype=torch.uint8, device=hidden.device)


def token_logprob_grpo(hidden, weight, target, logp_old, traj_ptr, reward, logp_ref=None,
                       loss_mask=None, group_size=16, eps_low=0.2, eps_high=0.28, beta=0.0,
                       adv_eps=1e-6, workspace=None, stream=None):
    """token_logprob and grpo_loss in one forward (the loss fused into the
    log-prob's combine pass): (logp, ratio, clipped, lse, advantage, dlogp,
    stats fp32 [8] in GRPO_STATS order), all on device.  The same clip pair
    serves the ratio output and the loss."""
    _need_bf16_cuda(hidden, weight)
    T, n_traj = hidden.shape[0], reward.numel()
    s = _lp_shape(hidden, weight, eps_low, eps_high)
    g = GrpoShape(T, n_traj, int(group_size), float(eps_low), float(eps_high), float(beta),
                  float(adv_eps))
    dev = hidden.device
    f = lambda n: torch.empty(n, dtype=torch.float32, device=dev)
    logp, ratio, clipped, lse, dlogp = f(T), f(T), f(T), f(T), f(T)
    adv, stats = f(n_traj), f(8)
    if workspace is None:
        workspace = torch.empty(
            int(mv_token_logprob_grpo_workspace_bytes(ctypes.byref(s), ctypes.byref(g))),
            dtype=torch.uint8, device=dev)
    check(mv_token_logprob_grpo(ctypes.byref(s), ctypes.byref(g), _ptr(hidden), _ptr(weight),
                                _ptr(target), _ptr(logp_old), _ptr(traj_ptr), _ptr(reward),
                                _ptr(logp_ref), _ptr(loss_mask), _ptr(logp), _ptr(ratio),
                                _ptr(clipped), _ptr(lse), _ptr(adv), _ptr(dlogp), _ptr(stats),
                                _ptr(workspace), workspace.numel(), _stream(stream)))
    return logp, ratio, clipped, lse, adv, dlogp, stats


# ---------------------------------------------------------------------------
# SDCC junction KL
# ---------------------------------------------------------------------------
def _kl_shape(h_teacher, rows_teacher, h_student, weight):
    return KLShape(rows_teacher.numel(), weight.shape[1], weight.shape[0], h_teacher.shape[0],
                   h_student.shape[0])


def _need_rows(*ts):
    for t in ts:
        if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous():
            raise ValueError("expected contiguous int32 CUDA row indices")


def sdcc_kl(h_teacher, rows_teacher, h_student, rows_student, weight, workspace=None,
            stream=None):
    """Per-leaf KL(p_teacher || q_student) and both log-partition values."""
    _need_bf16_cuda(h_teacher, h_student, weight)
    _need_rows(rows_teacher, rows_student)
    s = _kl_shape(h_teacher, rows_teacher, h_student, weight)
    n, dev = rows_teacher.numel(), weight.device
    kl, lse_t, lse_s = (torch.empty(n, dtype=torch.float32, device=dev) for _ in range(3))
    if workspace is None:
        workspace = torch.empty(int(mv_sdcc_kl_workspace_bytes(ctypes.byref(s))),
                                dtype=torch.uint8, device=dev)
    check(mv_sdcc_kl(ctypes.byref(s), _ptr(h_teacher), _ptr(rows_teacher), _ptr(h_student),
                     _ptr(rows_student), _ptr(weight), _ptr(kl), _ptr(lse_t), _ptr(lse_s),
                     _ptr(workspace), workspace.numel(), _stream(stream)))
    return kl, lse_t, lse_s


def sdcc_kl_bwd(h_teacher, rows_teacher, h_student, rows_student, weight, lse_t, lse_s, dkl,
                workspace=None, stream=None):
    """Gradient of sum_p dkl[p] KL_p into the student hidden row of each leaf: bf16 [n, H]."""
    _need_bf16_cuda(h_teacher, h_student, weight)
    _need_rows(rows_teacher, rows_student)
    s = _kl_shape(h_teacher, rows_teacher, h_student, weight)
    n, dev = rows_teacher.numel(), weight.device
    dh = torch.empty((n, weight.shape[1]), dtype=torch.bfloat16, device=dev)
    if workspace is None:
        workspace = torch.empty(int(mv_sdcc_kl_bwd_workspace_bytes(ctypes.byref(s))),
                                dtype=torch.uint8, device=dev)
    check(mv_sdcc_kl_bwd(ctypes.byref(s), _ptr(h_teacher), _ptr(rows_teacher), _ptr(h_student),
                         _ptr(rows_student), _ptr(weight), _ptr(lse_t), _ptr(lse_s), _ptr(dkl),
                         _ptr(dh), _ptr(workspace), workspace.numel(), _stream(stream)))
    return dh


def sdcc_lambda(step: int, total_steps: int, lambda_max: float = 0.1,
                warmup_frac: float = 0.2) -> float:
    return float(mv_sdcc_lambda(int(step), int(total_steps), float(lambda_max),
                                float(warmup_frac)))


# ---------------------------------------------------------------------------
# kernel timing
# ---------------------------------------------------------------------------
KERNELS = ["attn_fwd", "attn_bwd_dkdv", "attn_bwd_reduce", "attn_bwd_dq",
           "lm_logits", "lm_target", "lm_combine", "lm_wt", "lm_grad", "lm_dh", "lm_dw",
           "kl_logits", "kl_combine", "kl_wt", "kl_grad", "kl_dh",
           "grpo", "grpo_prep", "grpo_finish", "pack", "unpack", "rope", "pack_rope",
           "unpack_rope",
           "materialize", "ppo_clip"]


def profile_enable(on: bool = True) -> None:
    check(mv_profile_enable(1 if on else 0))


def profile_read(kernel: str):
    """(total ms, launches) of the named kernel since profiling was enabled."""
    ms = ctypes.c_double()
    n = ctypes.c_int32()
    check(mv_profile_read(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
