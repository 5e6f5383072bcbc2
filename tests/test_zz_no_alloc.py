"""mv_attn_bwd_noalloc, the attention backward that allocates nothing (its
workspace is a static scratch array on each GPU), against mv_attn_bwd on the
same inputs: every output bit-identical, on two calls in a row, the second
with a smaller input (the scratch keeps the first call's contents)."""
import numpy as np
import pytest
import torch

from paper_2609_00865_amd import mv, synth

pytestmark = pytest.mark.gpu


def _case(kind, seed):
    if kind == "medium":
        trajs = synth.make_trajectories("medium", seed)
        q, k, v, do = synth.make_attn_tensors("medium", seed)
    else:
        rng = np.random.default_rng(seed)
        trajs = synth.random_trajectories(rng, [300, 477, 223], max_edits=6, max_span=80,
                                          summary_max=30)
        T = trajs[-1].end
        gen = torch.Generator().manual_seed(seed)
        q, do = (torch.randn(T, 4, 128, generator=gen).to(torch.bfloat16) for _ in range(2))
        k, v = (torch.randn(T, 2, 128, generator=gen).to(torch.bfloat16) for _ in range(2))
    return trajs, q, k, v, do


def test_noalloc_backward_matches_workspace_backward():
    for kind, seed in (("medium", 0), ("ragged", 3)):
        trajs, q, k, v, do = _case(kind, seed)
        print(f"[gpu] noalloc backward {kind} seed {seed} T={q.shape[0]} Hq={q.shape[1]}",
              flush=True)
        m = mv.ViewMask(trajs).upload()
        qd, kd, vd, dd = (x.cuda().contiguous() for x in (q, k, v, do))
        o, lse = mv.attn_fwd(m, qd, kd, vd)
        need = int(mv.mv_attn_bwd_workspace_bytes(m.handle,
                                                  mv._attn_shape(m, qd, kd, None)))
        assert 0 < need <= mv.ATTN_BWD_NOALLOC_SCRATCH_BYTES
        ref = mv.attn_bwd(m, qd, kd, vd, o, dd, lse)
        got = mv.attn_bwd_noalloc(m, qd, kd, vd, o, dd, lse)
        torch.cuda.synchronize()
        for name, a, b in zip(("dQ", "dK", "dV"), got, ref):
            assert torch.equal(a, b), f"{kind}: {name} differs from mv_attn_bwd"
