"""The library's branch-replicated packing (host part) against the oracle's,
bit-exact, and its error paths (CPU only)."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import packing as OP
from paper_2609_00865_amd import mv, synth
from tests.fixtures import load, trajectory_from


def _check(trajs):
    pk = mv.BranchPack(trajs)
    want = OP.branch_pack(trajs)
    got = pk.layout()
    for k in ("src", "pos", "owner", "target", "seg_begin"):
        assert got[k].tolist() == want[k], k
    st = pk.stats()
    N = want["seg_begin"][-1]
    assert st["n_packed"] == N and st["total_tokens"] == trajs[-1].end
    lens = np.diff(want["seg_begin"])
    assert st["causal_pairs"] == int((lens * (lens + 1) // 2).sum())
    counts = np.bincount(want["src"], minlength=trajs[-1].end)
    assert st["max_copies"] == int(counts.max())
    # the packed mask is block-diagonal causal: bit-exact against the oracle's
    bits = mv.unpack_bits(pk.mask.materialize_host(0, N), N)
    assert torch.equal(bits, OP.block_causal_mask(want["seg_begin"]))
    return pk


def test_running_example():
    traj, _ = trajectory_from(load("running_example.json"))
    pk = _check([traj])
    assert pk.n_packed == 37 and pk.n_segments == 4


@pytest.mark.parametrize("seed", range(15))
def test_random_records(seed):
    rng = np.random.default_rng(4000 + seed)
    lens = [int(x) for x in rng.integers(1, 400, size=int(rng.integers(1, 4)))]
    _check(synth.random_trajectories(rng, lens, max_edits=8, max_span=40, summary_max=10))


@pytest.mark.parametrize("seed", range(10))
def test_random_records_with_restores(seed):
    rng = np.random.default_rng(5000 + seed)
    lens = [int(x) for x in rng.integers(2, 300, size=int(rng.integers(1, 4)))]
    _check(synth.random_trajectories(rng, lens, max_edits=8, max_span=40, summary_max=8,
                                     restore_max=25))


def test_no_edits_is_the_identity_layout():
    trajs = [synth.Trajectory(0, 50, ()), synth.Trajectory(50, 51, ())]
    pk = _check(trajs)
    lay = pk.layout()
    assert lay["src"].tolist() == list(range(51))
    assert lay["pos"].tolist() == list(range(50)) + [0]


def test_errors_without_gpu():
    trajs, _ = mv._trajectories_c([synth.Trajectory(0, 10, (synth.Edit(5, ((7, 8),)),))])
    h = ctypes.c_void_p()
    st = mv.mv_build_branch_pack(trajs, 1, 10, ctypes.byref(h))
    assert mv.mv_status_string(st).decode() == "MV_ERR_BAD_RECORD"   # span after its junction
    pk = mv.BranchPack([synth.Trajectory(0, 10, ())])
    fake = ctypes.c_void_p(1 << 20)
    st = mv.mv_pack_rows(pk.handle, fake, 64, fake, None)
    assert mv.mv_status_string(st).decode() == "MV_ERR_STATE"          # not uploaded
    st = mv.mv_branch_pack_upload(pk.handle, ctypes.c_void_p((1 << 20) + 16), 1 << 20, None)
    assert mv.mv_status_string(st).decode() == "MV_ERR_INVALID_ARG"
    n = mv.mv_branch_pack_device_bytes(pk.handle)
    st = mv.mv_branch_pack_upload(pk.handle, fake, n - 1, None)
    assert mv.mv_status_string(st).decode() == "MV_ERR_WORKSPACE"


def _check_shared(trajs):
    pk = mv.BranchPack(trajs, shared_trunk=True)
    want = OP.shared_trunk_pack(trajs)
    got = pk.layout()
    for k in ("src", "pos", "owner", "target", "seg_begin"):
        assert got[k].tolist() == want[k], k
    N = want["seg_begin"][-1]
    st = pk.stats()
    assert st["n_packed"] == N
    bits = mv.unpack_bits(pk.mask.materialize_host(0, N), N)
    ref = OP.views_mask(want["views"])
    assert torch.equal(bits, ref)
    assert st["causal_pairs"] == int(ref.sum())
    return pk


def test_shared_trunk_running_example():
    traj, _ = trajectory_from(load("running_example.json"))
    pk = _check_shared([traj])
    assert pk.n_packed == 16 and pk.n_segments == 4


@pytest.mark.parametrize("seed", range(12))
def test_shared_trunk_random_records(seed):
    rng = np.random.default_rng(6000 + seed)
    lens = [int(x) for x in rng.integers(1, 400, size=int(rng.integers(1, 4)))]
    _check_shared(synth.random_trajectories(rng, lens, max_edits=8, max_span=40, summary_max=10,
                                            restore_max=25 if seed % 3 == 0 else 0))


def test_shared_trunk_without_edits_is_the_physical_stream():
    trajs = [synth.Trajectory(0, 50, ()), synth.Trajectory(50, 51, ())]
    pk = _check_shared(trajs)
    assert pk.layout()["src"].tolist() == list(range(51))
