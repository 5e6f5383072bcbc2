"""GPU parity of the view-masked attention (C ABI -> HIP kernels) against the
oracle: full comparisons at sizes the oracle finishes quickly (several tiles
and ragged tails), sampled rows and keys at the long workloads' full sizes,
bit-exact mask bits, determinism, and negative controls."""
import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import views as V
from paper_2609_00865_amd import mv, synth
from tests.parity import ATOL_BF16, REL_FRO, assert_bf16_close, errors

pytestmark = pytest.mark.gpu

F64, F32 = torch.float64, torch.float32


def _run(trajs, q, k, v, do, repeat_bwd=False):
    print(f"[gpu] attention T={q.shape[0]} Hq={q.shape[1]} Hkv={k.shape[1]} d={q.shape[2]}",
          flush=True)
    m = mv.ViewMask(trajs).upload()
    qd, kd, vd, dd = (x.cuda().contiguous() for x in (q, k, v, do))
    o, lse = mv.attn_fwd(m, qd, kd, vd)
    dq, dk, dv = mv.attn_bwd(m, qd, kd, vd, o, dd, lse)
    out = {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}
    if repeat_bwd:
        out["again"] = mv.attn_bwd(m, qd, kd, vd, o, dd, lse)
    torch.cuda.synchronize()
    return m, out


def _check_full(trajs, q, k, v, do, what):
    m, g = _run(trajs, q, k, v, do, repeat_bwd=True)
    O, L, dQ, dK, dV = OA.logittree(trajs, q.to(F64), k.to(F64), v.to(F64), dout=do.to(F64),
                                    row_chunk=1024)
    assert_bf16_close(g["o"], O, f"{what} O")
    lse_err = errors(g["lse"], L)[0]
    print(f"{what} LSE max_abs={lse_err:.3e}", flush=True)
    assert lse_err < 1e-3
    assert_bf16_close(g["dq"], dQ, f"{what} dQ")
    assert_bf16_close(g["dk"], dK, f"{what} dK")
    assert_bf16_close(g["dv"], dV, f"{what} dV")
    # deterministic: a second backward gives the same bits
    for a, b in zip((g["dq"], g["dk"], g["dv"]), g["again"]):
        assert torch.equal(a, b)
    return g, (O, L, dQ, dK, dV)


@pytest.mark.parametrize("seed", [0, 1])
def test_tiny(seed):
    trajs = synth.make_trajectories("tiny", seed)
    q, k, v, do = synth.make_attn_tensors("tiny", seed)      # fp32 draws rounded to bf16
    _check_full(trajs, q, k, v, do, f"tiny/{seed}")


@pytest.mark.parametrize("seed", [0, 1])
def test_tiny_negative_controls(seed):
    """The Naive-Full and Naive-Compressed masks fail the same gates by >= 10x,
    for the output and for every gradient."""
    trajs = synth.make_trajectories("tiny", seed)
    t = trajs[0]
    q, k, v, do = synth.make_attn_tensors("tiny", seed)
    _, g = _run(trajs, q, k, v, do)
    for kind in ("full", "compressed"):
        M = torch.zeros(512, 512, dtype=torch.bool)
        for r, s in enumerate(V.naive_views(t, kind)):
            M[r, list(s)] = True
        On, _, dQn, dKn, dVn = OA.dense(trajs, q.to(F64), k.to(F64), v.to(F64),
                                        dout=do.to(F64), mask=M)
        for name, ref in (("o", On), ("dq", dQn), ("dk", dKn), ("dv", dVn)):
            max_abs, rel, _ = errors(g[name], ref)
            print(f"negative control {kind} {name}: max_abs={max_abs:.3e} rel_fro={rel:.3e}",
                  flush=True)
            assert max_abs >= 10 * ATOL_BF16 and rel >= 10 * REL_FRO


@pytest.mark.parametrize("d,hq,hkv,lens,seed", [
    (128, 4, 2, [300, 477, 223], 3),
    (64, 6, 3, [129, 64, 700], 4),
    (128, 2, 1, [1], 5),
    (128, 3, 1, [65], 6),
    (128, 2, 2, [129], 7),
    (64, 4, 2, [200, 57], 8),
])
def test_ragged_packed(d, hq, hkv, lens, seed):
    """Several trajectories, lengths off the tile grid, GQA, both head sizes."""
    rng = np.random.default_rng(seed)
    trajs = synth.random_trajectories(rng, lens, max_edits=6, max_span=80, summary_max=30)
    T = trajs[-1].end
    gen = torch.Generator().manual_seed(seed)
    q, do = (torch.randn(T, hq, d, generator=gen).to(torch.bfloat16) for _ in range(2))
    k, v = (torch.randn(T, hkv, d, generator=gen).to(torch.bfloat16) for _ in range(2))
    _check_full(trajs, q, k, v, do, f"ragged{lens}/d{d}")


@pytest.mark.parametrize("d,lens,seed", [(128, [700, 450, 301], 31), (64, [1200, 257], 32)])
def test_keys_that_re_enter(d, lens, seed):
    """Offload / retrieve records: evicted keys restored by later edits have
    several live intervals; every row must still attend exactly its view.
    The device mask bits are checked too (kernels share the predicate)."""
    rng = np.random.default_rng(seed)
    trajs = synth.random_trajectories(rng, lens, max_edits=10, max_span=80, summary_max=20,
                                      restore_max=60)
    assert any(e.restore for t in trajs for e in t.edits)
    T = trajs[-1].end
    gen = torch.Generator().manual_seed(seed)
    q, do = (torch.randn(T, 4, d, generator=gen).to(torch.bfloat16) for _ in range(2))
    k, v = (torch.randn(T, 2, d, generator=gen).to(torch.bfloat16) for _ in range(2))
    _check_full(trajs, q, k, v, do, f"restores{lens}/d{d}")
    m = mv.ViewMask(trajs).upload()
    dev = mv.unpack_bits(m.materialize(0, T).cpu(), T)
    assert torch.equal(dev, OA.visibility(trajs))


@pytest.mark.parametrize("d", [128, 64])
@pytest.mark.parametrize("jump", [False, True])
def test_scores_far_above_earlier_tiles(jump, d):
    """One key every 64 positions scores 20 base-2 units above the previous
    such key, so that most tiles exceed every score their rows have seen by
    more than 16 and take the forward's slow path (exact maximum, rescale);
    with jump, one of those keys scores another 200 units higher, so its
    probability overflows fp32 unless the slow path recomputes it from the
    score.  (A steady ramp of all keys would make dQ ill-conditioned: a
    large key component common to the few keys of each softmax, under dS
    rows that sum to zero.)"""
    hq, hkv, lens, seed = 2, 1, [700, 300], 41
    rng = np.random.default_rng(seed)
    trajs = synth.random_trajectories(rng, lens, max_edits=5, max_span=60, summary_max=20)
    T = trajs[-1].end
    gen = torch.Generator().manual_seed(seed)
    u = torch.randn(d, generator=gen)
    u = u / u.norm()
    q = (torch.randn(T, hq, d, generator=gen) * 0.25 + 8.0 * u).to(torch.bfloat16)
    k = torch.randn(T, hkv, d, generator=gen)
    c = d ** -0.5 * 1.4426950408889634   # base-2 units per unit of q.k
    for t in trajs:
        for m, p in enumerate(range(t.begin + 17, t.end, 64)):
            x = 20.0 * (m + 1) + (200.0 if jump and m == 4 else 0.0)   # target base-2 score
            k[p] = k[p] * 0.25 + (x / (8.0 * c)) * u
    k = k.to(torch.bfloat16)
    v, do = torch.randn(T, hkv, d, generator=gen), torch.randn(T, hq, d, generator=gen)
    _check_full(trajs, q, k, v.to(torch.bfloat16), do.to(torch.bfloat16),
                f"growing scores (jump={jump}, d={d})")


def test_no_compression_is_causal():
    T, hq, hkv, d = 700, 4, 1, 128
    gen = torch.Generator().manual_seed(11)
    q, do = (torch.randn(T, hq, d, generator=gen).to(torch.bfloat16) for _ in range(2))
    k, v = (torch.randn(T, hkv, d, generator=gen).to(torch.bfloat16) for _ in range(2))
    _check_full([synth.Trajectory(0, T, ())], q, k, v, do, "causal")


@pytest.mark.parametrize("seed", [0, 1])
def test_medium(seed):
    trajs = synth.make_trajectories("medium", seed)
    q, k, v, do = synth.make_attn_tensors("medium", seed)
    _check_full(trajs, q, k, v, do, f"medium/{seed}")


@pytest.mark.parametrize("workload", ["tiny", "medium"])
def test_materialized_bits(workload):
    trajs = synth.make_trajectories(workload, 0)
    m = mv.ViewMask(trajs).upload()
    T = m.total_tokens
    dev = m.materialize(0, T).cpu()
    host = m.materialize_host(0, T)
    assert torch.equal(dev, host)
    bits = mv.unpack_bits(dev, T)
    assert torch.equal(bits, OA.visibility(trajs))


def _sample_rows(trajs, rng, n_random=24):
    rows = set()
    for t in trajs:
        rows.update([t.begin, t.begin + 1, t.end - 1])
        for e in t.edits[:: max(1, len(t.edits) // 4)]:
            rows.update([e.junction - 1, e.junction, e.junction + 127])
    T = trajs[-1].end
    rows.update(int(x) for x in rng.integers(0, T, size=n_random))
    return sorted(r for r in rows if 0 <= r < T)


def _sampled_keys(trajs, death, rng, max_range, with_prompt_key):
    """Keys of the last trajectory whose dK/dV the oracle recomputes: evicted
    span ends, summary starts, the last rows and random keys with at most
    max_range rows seeing them; optionally a prompt key (seen by every later
    row of its trajectory) and always one key seen by more than 32 query
    blocks of 64 rows, so that split key tiles (partials summed by the reduce
    pass) are compared too."""
    keys = []
    t = trajs[-1]
    if with_prompt_key:
        keys.append(t.begin + 5)
    split = [j for j in range(t.begin, t.end) if 32 * 64 < death[j] - j <= max_range]
    if split:
        keys.append(int(split[int(rng.integers(0, len(split)))]))
    keys += [p for e in t.edits[:3] for (b, x) in e.evict for p in (b, x - 1)]
    keys += [e.summary[0] for e in t.edits[:2]]
    keys.append(t.end - 3)
    keys += [int(x) for x in rng.integers(t.begin, t.end, size=40)]
    out = []
    for j in keys:
        if (death[j] - j <= max_range or (with_prompt_key and j == t.begin + 5)) and j not in out:
            out.append(j)
    return out[:8]


@pytest.mark.slow
@pytest.mark.timeout(600)
@pytest.mark.parametrize("workload,seed,kv_heads,prompt_key", [("b4x32k", 0, [0, 3], True),
                                                               ("b4x32k", 1, [1, 2], True),
                                                               ("long128k", 0, [5], True)])
def test_full_size_sampled(workload, seed, kv_heads, prompt_key):
    """At the benchmark's size: sampled rows (O, LSE, dQ) and sampled keys
    (dK, dV, over every row that sees them) against the oracle.  The prompt
    key of the 128K trajectory is seen by all its 131072 rows: its key tile
    is cut into 64 items whose fp32 partials the reduce pass sums."""
    trajs = synth.make_trajectories(workload, seed)
    wl = synth.ATTN_WORKLOADS[workload]
    G = wl.n_heads_q // wl.n_heads_kv
    q, k, v, do = synth.make_attn_tensors(workload, seed, device="cuda")
    print(f"[gpu] {workload} seed {seed} full size", flush=True)
    m = mv.ViewMask(trajs).upload()
    o, lse = mv.attn_fwd(m, q, k, v)
    dq, dk, dv = mv.attn_bwd(m, q, k, v, o, do, lse)
    torch.cuda.synchronize()
    qc, kc, vc, dc = (x.cpu() for x in (q, k, v, do))
    oc, lc, dqc, dkc, dvc = (x.cpu() for x in (o, lse, dq, dk, dv))
    del q, k, v, do, o, lse, dq, dk, dv
    rng = np.random.default_rng(7 + seed)
    rows = _sample_rows(trajs, rng)
    heads = [hk * G + i for hk in kv_heads for i in (0, G - 1)]
    O, L = OA.rows(trajs, qc, kc, vc, rows, heads=heads)
    assert_bf16_close(oc[rows][:, heads], O, f"{workload} sampled O")
    assert errors(lc[heads][:, rows], L)[0] < 1e-3
    dQ = OA.row_grads(trajs, qc, kc, vc, dc, rows, heads=heads)
    assert_bf16_close(dqc[rows][:, heads], dQ, f"{workload} sampled dQ")
    death = [x for t in trajs for x in V.death_rows(t)]
    keys = _sampled_keys(trajs, death, rng, max_range=6000, with_prompt_key=prompt_key)
    hk = kv_heads[0]
    grp = list(range(hk * G, (hk + 1) * G))
    print(f"[gpu] {workload} sampled keys {[(j, death[j] - j) for j in keys]}", flush=True)
    for j in keys:
        _, _, _, dK, dV = OA.logittree(trajs, qc, kc, vc, dout=dc, heads=grp, dtype=F32,
                                       row_range=(j, death[j]), row_chunk=2048)
        assert_bf16_close(dkc[j, hk], dK[j, hk], f"{workload} dK key {j} (rows {death[j] - j})")
        assert_bf16_close(dvc[j, hk], dV[j, hk], f"{workload} dV key {j}")
