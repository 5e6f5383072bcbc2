"""Comparison helpers for GPU-vs-oracle parity.

Floating-point gates (bf16 outputs and gradients):
  * |gpu - ref| <= 2e-2 + 2^-8 |ref| elementwise: the 2e-2 absolute bound on
    the computation plus the half-ulp of the one round-to-nearest-even to
    bf16 that storing the output costs (half an ulp of x is at most
    2^-8 |x|; at |x| >= 8 it alone exceeds 2e-2), and
  * ||gpu - ref||_F <= 1e-2 * ||ref||_F (relative Frobenius), which stays
    meaningful where the absolute gate is loose (long rows have small |O|).
Both sides read the same bf16 input values; the oracle runs in fp64 (fp32 for
the largest samples).
"""
import torch

ATOL_BF16 = 2e-2
REL_FRO = 1e-2
LOGP_REL = 1e-4


BF16_HALF_ULP_REL = 2.0 ** -8

# Every bf16 comparison of the session: (what, literal max |gpu - ref|, the
# part beyond the output's own rounding, relative Frobenius error, max |ref|).
# The test session prints them at its end (tests/conftest.py), marking each
# comparison whose literal max-abs error exceeds 2e-2.
RECORD = []


def errors(gpu, ref):
    g = gpu.detach().to("cpu", torch.float64)
    r = ref.detach().to("cpu", torch.float64)
    diff = g - r
    max_abs = float(diff.abs().max()) if diff.numel() else 0.0
    den = float(r.norm())
    rel = float(diff.norm()) / den if den > 0 else float(diff.norm())
    return max_abs, rel, float(r.abs().max()) if r.numel() else 0.0


def bf16_excess(gpu, ref):
    """max over elements of |gpu - ref| - 2^-8 |ref| (the part not explained
    by rounding the stored output to bf16)."""
    g = gpu.detach().to("cpu", torch.float64)
    r = ref.detach().to("cpu", torch.float64)
    if not r.numel():
        return 0.0
    return float(((g - r).abs() - BF16_HALF_ULP_REL * r.abs()).max())


def assert_bf16_close(gpu, ref, what, atol=ATOL_BF16, rel_fro=REL_FRO):
    max_abs, rel, ref_max = errors(gpu, ref)
    excess = bf16_excess(gpu, ref)
    msg = (f"{what}: max_abs={max_abs:.3e} beyond_rounding={excess:.3e} rel_fro={rel:.3e} "
           f"max|ref|={ref_max:.3e}")
    print(msg, flush=True)
    RECORD.append((what, max_abs, excess, rel, ref_max))
    assert excess <= atol and rel <= rel_fro, msg
    return max_abs, rel


def assert_rel_close(gpu, ref, what, rel=LOGP_REL, floor=1e-6):
    g = gpu.detach().to("cpu", torch.float64)
    r = ref.detach().to("cpu", torch.float64)
    err = float(((g - r).abs() / r.abs().clamp(min=floor)).max()) if r.numel() else 0.0
    msg = f"{what}: max_rel={err:.3e}"
    print(msg, flush=True)
    assert err <= rel, msg
    return err
