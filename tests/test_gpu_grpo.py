"""GPU parity of the GRPO token loss, its per-token gradient and the drift
diagnostics (C ABI -> HIP kernels) against the oracle.

Gates: advantages, gradient and the mean statistics 1e-5 relative to their
scale (fp32 per-token arithmetic, fp32 per-block sums of 256 terms, fp64
across blocks).  The clip decision is taken in fp32 by the kernel and in fp64
by the oracle: a token whose ratio lies within 1e-5 of a clip edge may fall on
either side, so its gradient is accepted on either branch and the clip
fractions may differ by the count of such tokens.
"""
import numpy as np
import pytest
import torch

from oracle import grpo as OG
from paper_2609_00865_amd import mv, synth

pytestmark = pytest.mark.gpu
F64 = torch.float64


def _run(lengths, G, seed, beta=0.001, eps=(0.2, 0.28), use_ref=True, use_mask=True,
         noise=0.1):
    ptr, r, lp, old, ref, mask = synth.make_grpo_inputs(lengths, seed, logp_noise=noise)
    print(f"[gpu] grpo T={lp.numel()} n_traj={len(lengths)} G={G}", flush=True)
    ref = ref if use_ref else None
    mask = mask if use_mask else None
    dev = [None if x is None else x.cuda() for x in (ptr, r, lp, old, ref, mask)]
    adv, dlogp, stats = mv.grpo_loss(*dev, group_size=G, eps_low=eps[0], eps_high=eps[1],
                                     beta=beta if use_ref else 0.0)
    again = mv.grpo_loss(*dev, group_size=G, eps_low=eps[0], eps_high=eps[1],
                         beta=beta if use_ref else 0.0)
    torch.cuda.synchronize()
    for a, b in zip((adv, dlogp, stats), again):
        assert torch.equal(a, b)          # fixed-order reductions
    ref_out = OG.grpo_loss(ptr.tolist(), r, lp, old, ref, mask, G, eps[0], eps[1],
                           beta if use_ref else 0.0)
    return adv.cpu(), dlogp.cpu(), stats.cpu(), ref_out


def _check(adv, dlogp, stats, ref, what):
    assert torch.allclose(adv.double(), ref["advantage"], rtol=1e-5, atol=1e-5), what
    rho = ref["ratio"]
    amb = ((rho - 0.8).abs() < 1e-5) | ((rho - 1.28).abs() < 1e-5)
    n = float(ref["stats"]["n_loss_tokens"])
    scale = float(ref["dlogp"].abs().max()) or 1.0
    err = (dlogp.double() - ref["dlogp"]).abs()
    ok = err <= 1e-5 * scale
    assert bool(ok[~amb].all()), f"{what}: dlogp max err {float(err[~amb].max()):.3e}"
    st = ref["stats"]
    got = dict(zip(mv.GRPO_STATS, stats.tolist()))
    print(f"{what}: {got} ambiguous={int(amb.sum())}", flush=True)
    assert got["n_loss_tokens"] == n
    for k in ("loss", "logdiff", "kl_ref", "ratio_mean", "adv_abs_mean"):
        tol = 1e-5 * max(1.0, abs(float(st[k])))
        assert abs(got[k] - float(st[k])) <= tol, (what, k, got[k], float(st[k]))
    slack = float(amb.sum()) / max(n, 1.0) + 1e-6
    for k in ("clip_frac_low", "clip_frac_high"):
        assert abs(got[k] - float(st[k])) <= slack, (what, k)


@pytest.mark.parametrize("seed", [0, 1])
def test_ragged_groups(seed):
    rng = np.random.default_rng(seed)
    lengths = [int(x) for x in rng.integers(0, 700, size=32)]     # includes empty ones
    out = _run(lengths, 16, seed)
    _check(*out, f"grpo/{seed}")
    st = out[3]["stats"]
    assert float(st["clip_frac_low"]) > 0 and float(st["clip_frac_high"]) > 0


def test_no_reference_no_mask_group_of_one():
    _check(*_run([5, 300, 1, 257], 1, 3, use_ref=False, use_mask=False), "grpo-g1")


def test_single_token_and_wide_ratios():
    _check(*_run([1, 2], 2, 4, noise=1.0), "grpo-tiny")


def test_bench_shape():
    """The recipe's shape: 4 prompts x 16 samples, 512 tokens each (32768)."""
    _check(*_run([512] * 64, 16, 5), "grpo-64x512")
