"""GPU parity of both packings of the branch layers (replicated trunk, and
shared trunk: each branch stores only what it does not share with the one
before it) -- gather, its adjoint, rotary embedding by per-branch positions,
attention over the packed stream -- against the oracle, through the C ABI;
plus a two-layer model run on each packed stream against per-branch forwards
of the whole stack.

Gates: the gather is bit-exact; fp32 sums of the copies 1e-6 relative; bf16
outputs as everywhere else (2e-2 + 2^-8 |ref| elementwise, 1e-2 relative
Frobenius); the rotation is computed in fp32 from exact angles, so its error
beyond the final bf16 rounding stays below 1e-5 x max|x|.  The two-layer
model keeps bf16 activations between layers (as a bf16 model does): its gate
is a relative Frobenius error of 2e-2, and the union form must miss it by far.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import packing as OP
from paper_2609_00865_amd import mv, synth
from tests.parity import assert_bf16_close, errors

pytestmark = pytest.mark.gpu
F64 = torch.float64
BF = torch.bfloat16


def _pack(trajs, shared):
    return mv.BranchPack(trajs, shared_trunk=shared).upload()


def _layout(trajs, shared):
    return OP.shared_trunk_pack(trajs) if shared else OP.branch_pack(trajs)


SHARED = pytest.mark.parametrize("shared", [False, True], ids=["replicated", "shared_trunk"])


def _records(seed, lens=(300, 257, 180)):
    rng = np.random.default_rng(seed)
    return synth.random_trajectories(rng, list(lens), max_edits=6, max_span=40, summary_max=12)


@SHARED
def test_pack_and_unpack(shared):
    trajs = _records(1)
    pk = _pack(trajs, shared)
    lay = _layout(trajs, shared)
    T, N = trajs[-1].end, pk.n_packed
    print(f"[gpu] pack rows T={T} N={N}", flush=True)
    gen = torch.Generator().manual_seed(3)
    x = torch.randn(T, 3, 64, generator=gen).to(BF)
    got = mv.pack_rows(pk, x.cuda()).cpu()
    assert torch.equal(got, x[lay["src"]])
    g = torch.randn(N, 3, 64, generator=gen).to(BF)
    ref = OP.unpack_sum(lay, g, T)
    s32 = mv.unpack_rows_sum(pk, g.cuda(), out_fp32=True).cpu()
    s16 = mv.unpack_rows_sum(pk, g.cuda()).cpu()
    torch.cuda.synchronize()
    rel = float(((s32.double() - ref).abs() / ref.abs().clamp(min=1e-3)).max())
    assert rel < 1e-6, rel
    assert_bf16_close(s16, ref, "unpack bf16")


@SHARED
@pytest.mark.parametrize("d,theta", [(64, 1e4), (128, 1e6)])
def test_rope(d, theta, shared):
    trajs = _records(2, lens=(900, 400))
    pk = _pack(trajs, shared)
    lay = _layout(trajs, shared)
    N = pk.n_packed
    print(f"[gpu] rope N={N} d={d}", flush=True)
    gen = torch.Generator().manual_seed(4)
    x = torch.randn(N, 4, d, generator=gen).to(BF)
    xd = x.cuda()
    y = mv.rope(pk, xd, theta).cpu()
    back = mv.rope(pk, y.cuda(), theta, inverse=True).cpu()
    inplace = xd.clone()
    mv.rope(pk, inplace, theta, out=inplace)
    torch.cuda.synchronize()
    ref = OP.rope(x, lay["pos"], theta)
    excess = float(((y.double() - ref).abs() - 2.0 ** -8 * ref.abs()).max())
    assert excess <= 1e-5 * float(x.abs().max()), excess
    assert torch.equal(inplace.cpu(), y)
    assert_bf16_close(back, x.double(), "rope round trip")


@SHARED
@pytest.mark.parametrize("d,theta,H", [(64, 1e4, 3), (128, 1e6, 5)])
def test_fused_gather_rope_and_adjoint(d, theta, H, shared):
    """The gather with the rotation fused into it against the oracle's gather
    then rotation; its adjoint (inverse rotation of each copy, summed) against
    the oracle's inverse rotation then sum over copies.  The head count is not
    a multiple of the kernel's 4-head blocks."""
    trajs = _records(5, lens=(700, 333))
    pk = _pack(trajs, shared)
    lay = _layout(trajs, shared)
    T, N = trajs[-1].end, pk.n_packed
    print(f"[gpu] fused gather+rope T={T} N={N} H={H} d={d}", flush=True)
    gen = torch.Generator().manual_seed(6)
    x = torch.randn(T, H, d, generator=gen).to(BF)
    got = mv.pack_rows_rope(pk, x.cuda(), theta).cpu()
    ref = OP.rope(x[lay["src"]], lay["pos"], theta)
    excess = float(((got.double() - ref).abs() - 2.0 ** -8 * ref.abs()).max())
    assert excess <= 1e-5 * float(x.abs().max()), excess
    g = torch.randn(N, H, d, generator=gen).to(BF)
    gd = g.cuda()
    s32 = mv.unpack_rows_sum_rope(pk, gd, theta, out_fp32=True).cpu()
    s16 = mv.unpack_rows_sum_rope(pk, gd, theta).cpu()
    again = mv.unpack_rows_sum_rope(pk, gd, theta, out_fp32=True).cpu()
    torch.cuda.synchronize()
    assert torch.equal(s32, again)
    back = OP.unpack_sum(lay, OP.rope(g, lay["pos"], theta, inverse=True), T)
    # fp32 rotation and sums: error well under 1e-5 of the largest term
    err = float((s32.double() - back).abs().max())
    assert err <= 1e-5 * float(g.abs().max()) * max(int(np.bincount(lay["src"]).max()), 1), err
    assert_bf16_close(s16, back, "unpack+rope bf16")


@SHARED
@pytest.mark.parametrize("workload", ["tiny", "medium"])
def test_packed_attention_forward_backward(shared, workload):
    """One layer over the packed stream: owner rows give every row's view
    output; the copies' gradients summed back give the per-branch dK, dV
    (with the shared trunk a trunk slot gathers the gradients of every branch
    that reads it)."""
    trajs = synth.make_trajectories(workload, 0)
    q, k, v, do = synth.make_attn_tensors(workload, 0)
    if workload == "tiny":
        q = q.repeat(1, 2, 1).contiguous()
        do = do.repeat(1, 2, 1).contiguous()
    pk = _pack(trajs, shared)
    lay = pk.layout()
    own = lay["owner"].bool()
    print(f"[gpu] packed attention T={q.shape[0]} N={pk.n_packed}", flush=True)
    qp, kp, vp = (mv.pack_rows(pk, x.cuda()) for x in (q, k, v))
    dop = mv.pack_rows(pk, do.cuda())
    dop[~own.cuda()] = 0                       # only a row's own copy carries its loss
    o, lse = mv.attn_fwd(pk.mask, qp, kp, vp)
    dq, dk, dv = mv.attn_bwd(pk.mask, qp, kp, vp, o, dop, lse)
    dK = mv.unpack_rows_sum(pk, dk, out_fp32=True).cpu()
    dV = mv.unpack_rows_sum(pk, dv, out_fp32=True).cpu()
    torch.cuda.synchronize()
    O, L, dQ, rdK, rdV = OA.logittree(trajs, q.to(F64), k.to(F64), v.to(F64), dout=do.to(F64),
                                      row_chunk=1024)
    src = lay["src"].long()
    o_own = torch.zeros_like(O)
    o_own[src[own]] = o.cpu()[own].double()
    assert_bf16_close(o_own, O, "packed O (owner rows)")
    dq_own = torch.zeros_like(dQ)
    dq_own[src[own]] = dq.cpu()[own].double()
    assert_bf16_close(dq_own, dQ, "packed dQ (owner rows)")
    # summed over copies: a bf16 rounding per copy, then fp32 sums
    assert_bf16_close(dK, rdK, "packed dK summed over copies")
    assert_bf16_close(dV, rdV, "packed dV summed over copies")


@SHARED
def test_packed_attention_with_re_entering_keys(shared):
    """Packing a record whose keys leave and re-enter: every layer's segment
    copies the keys live at its start (restored ones at their own slots)."""
    rng = np.random.default_rng(41)
    trajs = synth.random_trajectories(rng, [600, 333], max_edits=8, max_span=60,
                                      summary_max=10, restore_max=50)
    T = trajs[-1].end
    gen = torch.Generator().manual_seed(41)
    q = torch.randn(T, 2, 64, generator=gen).to(BF)
    k, v = (torch.randn(T, 1, 64, generator=gen).to(BF) for _ in range(2))
    pk = _pack(trajs, shared)
    lay = pk.layout()
    own = lay["owner"].bool()
    print(f"[gpu] packed attention with restores T={T} N={pk.n_packed}", flush=True)
    o, _ = mv.attn_fwd(pk.mask, *(mv.pack_rows(pk, x.cuda()) for x in (q, k, v)))
    torch.cuda.synchronize()
    O, _ = OA.logittree(trajs, q.to(F64), k.to(F64), v.to(F64))
    got = torch.zeros_like(O)
    got[lay["src"].long()[own]] = o.cpu()[own].double()
    assert_bf16_close(got, O, "packed O with restores")


def _bf(x):
    return x.to(BF)


@SHARED
def test_two_layer_model_on_the_packed_stream(shared):
    trajs = synth.make_trajectories("tiny", 1)
    T = trajs[-1].end
    W, H, d, theta, n_layers = 128, 2, 64, 1e4, 2
    gen = torch.Generator().manual_seed(11)
    layers = [{n: _bf(torch.randn(W, W, generator=gen) / math.sqrt(W)).double()
               for n in ("wq", "wk", "wv", "wo")} for _ in range(n_layers)]
    x0 = _bf(torch.randn(T, W, generator=gen)).double()
    ref = OP.toy_logittree(trajs, x0, layers, H, d, theta)
    uni = OP.toy_union(trajs, x0, layers, H, d, theta)
    pk = _pack(trajs, shared)
    print(f"[gpu] two-layer model T={T} N={pk.n_packed} shared={shared}", flush=True)
    x = mv.pack_rows(pk, _bf(x0).cuda())
    for prm in layers:
        w = {n: t.float().cuda() for n, t in prm.items()}
        xf = x.float()
        q = _bf(xf @ w["wq"]).reshape(-1, H, d).contiguous()
        k = _bf(xf @ w["wk"]).reshape(-1, H, d).contiguous()
        v = _bf(xf @ w["wv"]).reshape(-1, H, d).contiguous()
        q, k = mv.rope(pk, q, theta), mv.rope(pk, k, theta)
        o, _ = mv.attn_fwd(pk.mask, q, k, v)
        x = _bf(xf + o.float().reshape(-1, W) @ w["wo"])
    torch.cuda.synchronize()
    lay = pk.layout()
    own = lay["owner"].bool()
    got = torch.zeros(T, W, dtype=F64)
    got[lay["src"].long()[own]] = x.cpu()[own].double()
    _, rel, _ = errors(got, ref)
    _, rel_uni, _ = errors(uni, ref)
    print(f"two-layer: packed rel_fro={rel:.3e}  union-form rel_fro={rel_uni:.3e}", flush=True)
    assert rel <= 2e-2
    assert rel_uni >= 10 * rel
