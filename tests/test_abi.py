"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, sizes its workspaces, and rejects bad arguments before launching."""
import ctypes
import os
import re

import pytest
import torch

from paper_2609_00865_amd import mv, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mv.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mv_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(mv._LIB_PATH)
    names = _declared()
    assert len(names) >= 19
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(mv.EXPORTED) == names


def test_version_and_status_strings():
    assert mv.mv_version() >> 16 == 1
    assert mv.mv_status_string(0) == b"MV_OK"
    assert mv.mv_status_string(3) == b"MV_ERR_SHAPE"


FAKE = ctypes.c_void_p(1 << 20)      # aligned, non-null, never dereferenced


def _shape(T=512, hq=1, hkv=1, d=64, scale=0.0):
    return mv.AttnShape(T, hq, hkv, d, scale)


def _mask():
    return mv.ViewMask(synth.make_trajectories("tiny", 0))


def _status(s):
    return mv.mv_status_string(s).decode()


def test_attention_argument_errors():
    m = _mask()
    fwd = lambda sh, *p: _status(mv.mv_attn_fwd(m.handle, ctypes.byref(sh), *p))
    ok = [FAKE] * 5 + [None]
    assert fwd(_shape(T=511), *ok) == "MV_ERR_SHAPE"
    assert fwd(_shape(hq=3, hkv=2), *ok) == "MV_ERR_SHAPE"
    assert fwd(_shape(d=96), *ok) == "MV_ERR_UNSUPPORTED"
    assert fwd(_shape(), None, FAKE, FAKE, FAKE, FAKE, None) == "MV_ERR_INVALID_ARG"
    assert fwd(_shape(), ctypes.c_void_p((1 << 20) + 2), FAKE, FAKE, FAKE, FAKE, None) == "MV_ERR_INVALID_ARG"
    # valid request, but the mask was never uploaded: refused before any launch
    assert fwd(_shape(), *ok) == "MV_ERR_STATE"
    assert "uploaded" in mv.mv_last_error().decode()


def test_attention_tensor_size_limit():
    """The kernels address each tensor with 32-bit byte offsets: a Q of 4 GiB
    or more is refused (262144 tokens x 64 heads x 128 x 2 B = 2^32 B)."""
    big = mv.ViewMask([synth.Trajectory(0, 262144, ())])
    fwd = lambda sh: _status(mv.mv_attn_fwd(big.handle, ctypes.byref(sh), *([FAKE] * 5), None))
    assert fwd(_shape(T=262144, hq=64, hkv=8, d=128)) == "MV_ERR_UNSUPPORTED"
    assert "4 GiB" in mv.mv_last_error().decode()
    # one token fewer fits: the request gets as far as the upload check
    small = mv.ViewMask([synth.Trajectory(0, 262143, ())])
    sh = _shape(T=262143, hq=64, hkv=8, d=128)
    assert _status(mv.mv_attn_fwd(small.handle, ctypes.byref(sh), *([FAKE] * 5), None)) == "MV_ERR_STATE"


def test_backward_workspace_errors():
    m = _mask()
    sh = _shape()
    need = mv.mv_attn_bwd_workspace_bytes(m.handle, ctypes.byref(sh))
    assert need >= 512 * 4
    st = mv.mv_attn_bwd(m.handle, ctypes.byref(sh), *([FAKE] * 10), need - 1, None)
    assert _status(st) == "MV_ERR_WORKSPACE"
    assert mv.mv_attn_bwd_workspace_bytes(m.handle, ctypes.byref(_shape(d=96))) == 0


def test_noalloc_backward_scratch_limit():
    """mv_attn_bwd_noalloc refuses, before anything is enqueued, a backward
    whose workspace exceeds its static scratch (the 4 x 32K batch needs
    ~840 MiB); the 8K trajectory's (~37.5 MiB) fits and gets as far as the
    upload check."""
    big = mv.ViewMask(synth.make_trajectories("b4x32k", 0))
    sh = _shape(T=big.total_tokens, hq=28, hkv=4, d=128)
    assert mv.mv_attn_bwd_workspace_bytes(big.handle, ctypes.byref(sh)) > \
        mv.ATTN_BWD_NOALLOC_SCRATCH_BYTES
    st = mv.mv_attn_bwd_noalloc(big.handle, ctypes.byref(sh), *([FAKE] * 9), None)
    assert _status(st) == "MV_ERR_WORKSPACE"
    assert "scratch" in mv.mv_last_error().decode()
    med = mv.ViewMask(synth.make_trajectories("medium", 0))
    sh = _shape(T=med.total_tokens, hq=16, hkv=4, d=128)
    assert 0 < mv.mv_attn_bwd_workspace_bytes(med.handle, ctypes.byref(sh)) <= \
        mv.ATTN_BWD_NOALLOC_SCRATCH_BYTES
    st = mv.mv_attn_bwd_noalloc(med.handle, ctypes.byref(sh), *([FAKE] * 9), None)
    assert _status(st) == "MV_ERR_STATE"


def test_logprob_argument_errors():
    s = mv.LogprobShape(16, 100, 50, 0.2, 0.2)
    assert _status(mv.mv_token_logprob(ctypes.byref(s), *([FAKE] * 9), 1 << 30, None)) == "MV_ERR_UNSUPPORTED"
    s = mv.LogprobShape(16, 128, 50, 0.2, 0.2)
    need = mv.mv_token_logprob_workspace_bytes(ctypes.byref(s))
    assert need > 0
    args = [FAKE] * 9
    assert _status(mv.mv_token_logprob(ctypes.byref(s), *args, need - 1, None)) == "MV_ERR_WORKSPACE"
    # ratio requested without logp_old
    a2 = [FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE]
    assert _status(mv.mv_token_logprob(ctypes.byref(s), *a2, need, None)) == "MV_ERR_INVALID_ARG"
    bad = mv.LogprobShape(16, 128, 50, 1.5, 0.2)
    assert _status(mv.mv_token_logprob(ctypes.byref(bad), *args, need, None)) == "MV_ERR_INVALID_ARG"
    nb = mv.mv_token_logprob_bwd_workspace_bytes(ctypes.byref(s))
    assert nb >= 16 * 256 * 2
    assert _status(mv.mv_token_logprob_bwd(ctypes.byref(s), *([FAKE] * 7), nb - 1, None)) == "MV_ERR_WORKSPACE"


def test_sdcc_argument_errors():
    s = mv.KLShape(8, 100, 50, 16, 16)
    assert _status(mv.mv_sdcc_kl(ctypes.byref(s), *([FAKE] * 9), 1 << 30, None)) == "MV_ERR_UNSUPPORTED"
    s = mv.KLShape(8, 128, 50, -1, 16)
    assert _status(mv.mv_sdcc_kl(ctypes.byref(s), *([FAKE] * 9), 1 << 30, None)) == "MV_ERR_SHAPE"
    s = mv.KLShape(8, 128, 50, 16, 16)
    need = mv.mv_sdcc_kl_workspace_bytes(ctypes.byref(s))
    assert need > 0
    assert _status(mv.mv_sdcc_kl(ctypes.byref(s), *([FAKE] * 9), need - 1, None)) == "MV_ERR_WORKSPACE"
    a = [FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE]
    assert _status(mv.mv_sdcc_kl(ctypes.byref(s), *a, need, None)) == "MV_ERR_INVALID_ARG"
    nb = mv.mv_sdcc_kl_bwd_workspace_bytes(ctypes.byref(s))
    assert nb >= 8 * 256 * 2
    assert _status(mv.mv_sdcc_kl_bwd(ctypes.byref(s), *([FAKE] * 10), nb - 1, None)) == "MV_ERR_WORKSPACE"
    empty = mv.KLShape(0, 128, 50, 0, 0)
    assert _status(mv.mv_sdcc_kl(ctypes.byref(empty), *([None] * 9), 0, None)) == "MV_OK"
    h = ctypes.c_void_p()
    assert _status(mv.mv_build_view_mask_kind(None, 0, 10, 0, ctypes.byref(h))) == "MV_ERR_INVALID_ARG"


def test_mask_buffer_errors():
    m = _mask()
    assert _status(mv.mv_view_mask_upload(m.handle, None, 1 << 20, None)) == "MV_ERR_INVALID_ARG"
    assert _status(mv.mv_view_mask_upload(m.handle, ctypes.c_void_p((1 << 20) + 16), 1 << 20, None)) == "MV_ERR_INVALID_ARG"
    assert _status(mv.mv_view_mask_upload(m.handle, FAKE, m.device_bytes() - 1, None)) == "MV_ERR_WORKSPACE"
    assert _status(mv.mv_view_mask_materialize(m.handle, 0, 513, FAKE, None)) == "MV_ERR_INVALID_ARG"
    assert _status(mv.mv_view_mask_materialize(m.handle, 0, 10, FAKE, None)) == "MV_ERR_STATE"
    assert _status(mv.mv_ppo_clip_dlogp(-1, FAKE, FAKE, 0.2, 0.2, 1.0, FAKE, None)) == "MV_ERR_INVALID_ARG"
    h = ctypes.c_void_p()
    assert _status(mv.mv_build_view_mask(None, 0, 10, ctypes.byref(h))) == "MV_ERR_INVALID_ARG"


def test_tiled_builder_accepts_only_the_kernels_tiles():
    """The builder that names a tile shape builds the same mask for the
    kernels' own shape and refuses any other before building anything."""
    trajs = synth.make_trajectories("tiny", 0)
    tc, keep = mv._trajectories_c(trajs)
    T = trajs[-1].end
    h = ctypes.c_void_p()
    assert _status(mv.mv_build_view_mask_tiled(tc, len(trajs), T, mv.TILE_Q, mv.TILE_K,
                                               ctypes.byref(h))) == "MV_OK"
    st = mv.MaskStats()
    assert _status(mv.mv_view_mask_stats(h, ctypes.byref(st))) == "MV_OK"
    assert st.visible_pairs == mv.ViewMask(trajs).stats()["visible_pairs"]
    mv.mv_view_mask_free(h)
    for tq, tk in ((64, 64), (128, 128), (256, 64), (0, 0)):
        h2 = ctypes.c_void_p()
        assert _status(mv.mv_build_view_mask_tiled(tc, len(trajs), T, tq, tk,
                                                   ctypes.byref(h2))) == "MV_ERR_UNSUPPORTED"
        assert not h2.value
        assert b"unsupported" in mv.mv_last_error()


def test_binding_has_no_fallback():
    """The binding is marshalling only: it never imports the oracle."""
    src = open(os.path.join(ROOT, "paper_2609_00865_amd", "mv.py")).read()
    assert "oracle" not in src.replace("no fallback", "")
    for name in os.listdir(os.path.join(ROOT, "paper_2609_00865_amd")):
        if name.endswith(".py"):
            text = open(os.path.join(ROOT, "paper_2609_00865_amd", name)).read()
            assert "import oracle" not in text and "from oracle" not in text, name
