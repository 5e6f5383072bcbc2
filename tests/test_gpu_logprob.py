"""GPU parity of the fused LM-head log-prob / ratio / clip and its backward
(C ABI -> HIP kernels) against the oracle."""
import math

import pytest
import torch

from oracle import logprob as OL
from paper_2609_00865_amd import mv, synth
from tests.parity import assert_bf16_close, assert_rel_close

pytestmark = pytest.mark.gpu
F64 = torch.float64


def _inputs(T, H, V, seed, skip_every=0):
    """Inputs with every skip_every-th token (the last of each run, so a
    single token stays scored) marked as one without loss."""
    h, w, y, old, g = synth.make_logprob_inputs(T, H, V, seed)
    if skip_every:
        y[skip_every - 1::skip_every] = -1
    return h, w, y, old, g


def _gpu(h, w, y, old, g, eps_lo=0.2, eps_hi=0.2):
    print(f"[gpu] logprob T={h.shape[0]} H={h.shape[1]} V={w.shape[0]}", flush=True)
    hd, wd, yd, od, gd = h.cuda(), w.cuda(), y.cuda(), old.cuda(), g.cuda()
    logp, ratio, clipped, lse = mv.token_logprob(hd, wd, yd, od, eps_lo, eps_hi)
    dh = mv.token_logprob_bwd(hd, wd, yd, lse, gd)
    torch.cuda.synchronize()
    return logp.cpu(), ratio.cpu(), clipped.cpu(), lse.cpu(), dh.cpu()


def _check(h, w, y, old, g, what, eps_lo=0.2, eps_hi=0.2):
    logp, ratio, clipped, lse, dh = _gpu(h, w, y, old, g, eps_lo, eps_hi)
    rl, rr, rc, rlse = OL.token_logprob(h, w, y, old, eps_lo, eps_hi)
    assert_rel_close(logp[y >= 0], rl[y >= 0], f"{what} logp")
    assert torch.all(logp[y < 0] == 0)
    assert_rel_close(lse, rlse, f"{what} lse")
    assert_rel_close(ratio, rr, f"{what} ratio", rel=2e-3)
    assert_rel_close(clipped, rc, f"{what} clipped", rel=2e-3)
    ref_dh = OL.token_logprob_bwd(h, w, y, g)
    assert_bf16_close(dh, ref_dh, f"{what} dH")
    return logp, ratio, clipped


@pytest.mark.parametrize("T,H,V", [(300, 256, 1000), (257, 128, 600), (64, 192, 256),
                                   (1, 64, 17)])
def test_small_ragged(T, H, V):
    inputs = _inputs(T, H, V, 1, skip_every=7)
    assert (inputs[2] >= 0).any()
    _check(*inputs, f"lp{T}x{H}x{V}")


def test_out_of_range_targets_are_skipped_and_counted():
    """Ids outside [-1, vocab) are never used as an index: their tokens are
    scored as tokens without loss (logp 0, ratio 1, zero dH) and counted in
    the workspace's status word; the other tokens are unaffected."""
    T, H, V = 200, 128, 1000
    h, w, y, old, g = _inputs(T, H, V, 12)
    bad = {3: V, 50: V + 12345, 77: -2, 199: 2 ** 31 - 1}
    for t, val in bad.items():
        y[t] = val
    y[10] = -1                          # the ordinary convention: not counted
    print(f"[gpu] logprob out-of-range targets T={T} H={H} V={V}", flush=True)
    hd, wd, yd, od, gd = h.cuda(), w.cuda(), y.cuda(), old.cuda(), g.cuda()
    ws_f = mv.token_logprob_workspace(hd, wd)
    ws_b = mv.token_logprob_bwd_workspace(hd, wd)
    logp, ratio, clipped, lse = mv.token_logprob(hd, wd, yd, od, workspace=ws_f)
    dh = mv.token_logprob_bwd(hd, wd, yd, lse, gd, workspace=ws_b)
    assert mv.token_logprob_bad_targets(ws_f) == len(bad)
    assert mv.token_logprob_bad_targets(ws_b) == len(bad)
    logp, ratio, clipped, dh = logp.cpu(), ratio.cpu(), clipped.cpu(), dh.cpu()
    skip = torch.tensor(sorted(list(bad) + [10]))
    assert torch.all(logp[skip] == 0) and torch.all(ratio[skip] == 1)
    assert torch.all(clipped[skip] == 1) and torch.all(dh[skip].float() == 0)
    y_ref = y.clone()
    y_ref[skip] = -1
    rl, rr, rc, rlse = OL.token_logprob(h, w, y_ref, old)
    keep = y_ref >= 0
    assert_rel_close(logp[keep], rl[keep], "bad-id case logp")
    assert_rel_close(ratio, rr, "bad-id case ratio", rel=2e-3)
    assert_bf16_close(dh, OL.token_logprob_bwd(h, w, y_ref, g), "bad-id case dH")
    # a later call on the same workspace starts from zero
    mv.token_logprob(hd, wd, y_ref.cuda(), od, workspace=ws_f)
    assert mv.token_logprob_bad_targets(ws_f) == 0


def test_clip_edges_exercised():
    """Behaviour log-probs near the recomputed ones, so both clip edges and the
    unclipped interior occur (the benchmark's draw clips every token)."""
    T, H, V = 512, 256, 3000
    h, w, y, _, g = _inputs(T, H, V, 2)
    ref, _, _, _ = OL.token_logprob(h, w, y)
    gen = torch.Generator().manual_seed(3)
    old = (ref + 0.1 * torch.randn(T, generator=gen, dtype=F64)).float()
    logp, ratio, clipped = _check(h, w, y, old, g, "clip", 0.2, 0.28)
    assert (clipped == 0.8).any() and (clipped == 1.28).any()
    assert ((clipped > 0.8) & (clipped < 1.28)).sum() > T // 2


def test_uniform_special_case():
    T, H, V = 96, 128, 777
    h, w, y, old, g = _inputs(T, H, V, 4)
    w[:] = w[0]
    logp, _, _, lse, dh = _gpu(h, w, y, old, g)
    assert torch.allclose(logp, torch.full_like(logp, -math.log(V)), rtol=1e-4, atol=0)
    assert dh.float().abs().max() < 1e-3


def test_ppo_clip_dlogp():
    gen = torch.Generator().manual_seed(5)
    ratio = torch.exp(0.4 * torch.randn(1000, generator=gen))
    adv = torch.randn(1000, generator=gen)
    got = mv.ppo_clip_dlogp(ratio.cuda(), adv.cuda(), 0.2, 0.28, 1.0).cpu()
    ref = OL.ppo_clip_dlogp(ratio, adv, 0.2, 0.28)
    assert torch.allclose(got.double(), ref, atol=1e-6, rtol=1e-6)


@pytest.mark.slow
def test_full_size_sampled():
    """32768 tokens x 3584 hidden x 152064 vocab; 48 sampled tokens."""
    wl = synth.LOGPROB_WORKLOADS["lmhead"]
    h, w, y, old, g = synth.make_logprob_inputs(wl.n_tokens, wl.hidden, wl.vocab, 0, device="cuda")
    print("[gpu] lmhead full size", flush=True)
    logp, ratio, clipped, lse = mv.token_logprob(h, w, y, old)
    dh = mv.token_logprob_bwd(h, w, y, lse, g)
    torch.cuda.synchronize()
    idx = torch.tensor([0, 1, 255, 256, 4095, 16384, wl.n_tokens - 1] +
                       list(range(100, 32768, 800)))
    hc, wc, yc, oc, gc = h.cpu(), w.cpu(), y.cpu(), old.cpu(), g.cpu()
    rl, rr, rc, rlse = OL.token_logprob(hc[idx], wc, yc[idx], oc[idx], dtype=torch.float32)
    assert_rel_close(logp.cpu()[idx], rl, "lmhead logp")
    assert_rel_close(lse.cpu()[idx], rlse, "lmhead lse")
    assert_rel_close(ratio.cpu()[idx], rr, "lmhead ratio", rel=2e-3)
    assert_rel_close(clipped.cpu()[idx], rc, "lmhead clipped", rel=2e-3)
    ref_dh = OL.token_logprob_bwd(hc[idx], wc, yc[idx], gc[idx], dtype=torch.float32)
    assert_bf16_close(dh.cpu()[idx], ref_dh, "lmhead dH")


@pytest.mark.parametrize("T,H,V", [(300, 256, 1000), (2000, 512, 3000)])
def test_repeat_is_bit_identical(T, H, V):
    """Fixed-order reductions throughout (per-chunk partials merged in chunk
    order, the split dH summed in split order, no atomics): a second forward
    and backward reproduce every bit.  Both shapes split dH over the
    vocabulary and have ragged token and vocabulary tiles."""
    h, w, y, old, g = _inputs(T, H, V, 9, skip_every=11)
    first = _gpu(h, w, y, old, g)
    second = _gpu(h, w, y, old, g)
    for a, b in zip(first, second):
        assert torch.equal(a, b)


@pytest.mark.parametrize("T,H,V", [(300, 256, 1000), (257, 192, 600), (64, 128, 256),
                                   (1, 64, 17)])
def test_dweight_small_ragged(T, H, V):
    h, w, y, old, g = _inputs(T, H, V, 6, skip_every=5)
    print(f"[gpu] dweight T={T} H={H} V={V}", flush=True)
    hd, wd, yd, gd = h.cuda(), w.cuda(), y.cuda(), g.cuda()
    _, _, _, lse = mv.token_logprob(hd, wd, yd)
    ws = mv.token_logprob_bwd_workspace(hd, wd)
    mv.token_logprob_bwd(hd, wd, yd, lse, gd, workspace=ws)
    dw = mv.token_logprob_dweight(hd, wd, ws).cpu()
    torch.cuda.synchronize()
    ref = OL.token_logprob_dweight(h, w, y, g)
    assert_bf16_close(dw, ref, f"dW {T}x{H}x{V}")
    # every row of G sums to zero, so do the columns of dW over the vocabulary
    assert float(dw.double().sum(dim=0).abs().max()) < 1e-2 * float(ref.abs().max()) + 1e-3


@pytest.mark.slow
def test_dweight_full_width():
    """320 tokens (a ragged last k slice) at the full 3584 x 152064 head; the
    targets' rows and every 6007th row checked (fp32 oracle)."""
    wl = synth.LOGPROB_WORKLOADS["lmhead"]
    T = 320
    h, w, y, old, g = synth.make_logprob_inputs(T, wl.hidden, wl.vocab, 3)
    print("[gpu] dweight full width", flush=True)
    hd, wd, yd, gd = h.cuda(), w.cuda(), y.cuda(), g.cuda()
    _, _, _, lse = mv.token_logprob(hd, wd, yd)
    ws = mv.token_logprob_bwd_workspace(hd, wd)
    mv.token_logprob_bwd(hd, wd, yd, lse, gd, workspace=ws)
    dw = mv.token_logprob_dweight(hd, wd, ws)
    torch.cuda.synchronize()
    rows = torch.tensor(sorted(set(y[:40].long().tolist()) | set(range(0, wl.vocab, 6007))))
    ref = OL.token_logprob_dweight(h, w, y, g, dtype=torch.float32)[rows]
    assert_bf16_close(dw.cpu()[rows], ref, "dW full width (sampled rows)")
