"""Benchmark of the view-masked scoring hot path on one MI355X.

One step = the whole path over one batch of synthetic input:
  * view-masked attention forward + backward over 4 packed trajectories of
    32768 tokens (28 query / 4 KV heads, head_dim 128, bf16; 16 compression
    events per trajectory, 2048-token protected prompt), and
  * the fused LM-head token log-prob / ratio / clip forward + backward over
    32768 tokens (hidden 3584, vocab 152064, bf16).
The eviction records are turned into the mask on the host before the timed
region (the mask is an input, like the tensors); its build time is reported.

Printed JSON (one line).  `value` is the metric itself: useful TFLOP/s of the
view-masked attention forward + backward of the 32K-token trajectories
(14 d P Hq FLOPs, P the visible (row, key) pairs), timed with events around
the attention part of every step; `tokens_per_s` is trajectory tokens over the
same attention time.  `ms_per_step` covers the whole step (attention and LM
head); the LM head and the step blend are sub-objects.  After the step, the
attention alone is timed on the other trajectory shapes (the second seed of the
4 x 32K batch, the 131072-token trajectory with 64/8 heads for both seeds, the
8192-token trajectory), and the SDCC pass, the LM-head weight gradient and the
branch-replicated layer on their own.  The roofline object covers the step's
longest kernel; `roofline_attention` the attention's longest kernel, with its
useful FLOPs.  The CPU oracle is timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "view-masked attn fwd+bwd useful TFLOP/s + % MFMA peak; trajectory tokens/s"
PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA (256 CU x 2.4 GHz x 4096 flop/clk)
PEAK_HBM_GBS = 8000.0
ATTN_WORKLOAD = "b4x32k"
LM_WORKLOAD = "lmhead"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one plain 1 GiB device copy (PMC byte-counter calibration)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-sdcc", action="store_true",
                    help="skip the separately timed SDCC junction-KL pass")
    ap.add_argument("--no-packed", action="store_true",
                    help="skip the separately timed branch-replicated attention layer")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the attention timings on the other trajectory shapes")
    return ap.parse_args()


def attn_kernel_flops(st, d, hq):
    """Useful and executed FLOPs of one launch of each attention kernel.

    Useful: the backward's five products over the visible pairs P (S
    recomputed once, dP, dV, dK, dQ) split as the kernels split them: dK/dV
    holds S, dP, dV and dK (8 d P Hq), dQ only its own product (2 d P Hq; its
    S and dP are recomputations beyond the five).  Executed: every product a
    kernel runs over the (row, key) pairs of the tiles it visits."""
    P = st["visible_pairs"]
    fp, bp = st["fwd_tile_pairs"], st["bwd_tile_pairs"]
    return {
        "attn_fwd": {"useful": 4.0 * d * P * hq, "executed": 4.0 * d * fp * hq},
        "attn_bwd_dkdv": {"useful": 8.0 * d * P * hq, "executed": 8.0 * d * bp * hq},
        "attn_bwd_dq": {"useful": 2.0 * d * P * hq, "executed": 6.0 * d * fp * hq},
    }


def lm_kernel_flops(T_lm, H, V):
    """Algorithmic FLOPs of one launch of each LM-head product."""
    return {n: 2.0 * T_lm * H * V for n in ("lm_logits", "lm_grad", "lm_dh")}


def measured_traffic(kernel):
    """HBM bytes per launch recorded by the counter runs under profiles/, or None
    when the kernel's sources have changed since (or were never measured)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "roofline_traffic.txt")
    if not os.path.exists(path):
        return None
    for line in open(path):
        if line.startswith("#") or not line.strip():
            continue
        kv = dict(x.split("=", 1) for x in line.split())
        if kv.get("kernel") != kernel:
            continue
        m = hashlib.sha256()
        for n in kv["sources"].split(","):
            src = os.path.join(ROOT, "paper_2609_00865_amd", "csrc", n)
            if not os.path.exists(src):
                return None
            with open(src, "rb") as f:
                m.update(f.read())
        if m.hexdigest()[:16] != kv["sha256_16"]:
            return None
        return float(kv["fetch_bytes"]) + float(kv["write_bytes"])
    return None


def cpu_baseline(trajs, wl, lmw, attn_flops_step, lm_flops_step):
    """The oracle, untouched, on a bounded sample of the same workload."""
    import torch
    from oracle import attention as OA
    from oracle import logprob as OL
    from oracle import views as V
    from paper_2609_00865_amd import synth

    cores = torch.get_num_threads()
    # attention: first trajectory, KV groups 0 and 1, rows [0, R), fp32 forward + backward
    R = 24576
    G = wl.n_heads_q // wl.n_heads_kv
    heads = list(range(2 * G))
    t0 = trajs[0]
    sub = [synth.Trajectory(t0.begin, t0.begin + R,
                            tuple(e for e in t0.edits if e.junction < t0.begin + R))]
    gen = torch.Generator().manual_seed(99)
    q = torch.randn(R, wl.n_heads_q, wl.head_dim, generator=gen).to(torch.bfloat16)
    k = torch.randn(R, wl.n_heads_kv, wl.head_dim, generator=gen).to(torch.bfloat16)
    v = torch.randn(R, wl.n_heads_kv, wl.head_dim, generator=gen).to(torch.bfloat16)
    do = torch.randn(R, wl.n_heads_q, wl.head_dim, generator=gen).to(torch.bfloat16)
    pairs = sum(V.view_sizes(sub[0]))
    a0 = time.perf_counter()
    OA.logittree(sub, q, k, v, dout=do, heads=heads, dtype=torch.float32, row_chunk=2048)
    a_s = time.perf_counter() - a0
    attn_rate = 14.0 * wl.head_dim * pairs * len(heads) / a_s
    log(f"cpu oracle attention sample: {a_s:.2f}s, {attn_rate / 1e9:.1f} GFLOP/s")
    # LM head: 2048 tokens, fp32 forward + backward
    n = 2048
    h, w, y, old, g = synth.make_logprob_inputs(n, lmw.hidden, lmw.vocab, 0)
    l0 = time.perf_counter()
    OL.token_logprob(h, w, y, old, dtype=torch.float32)
    OL.token_logprob_bwd(h, w, y, g, dtype=torch.float32)
    l_s = time.perf_counter() - l0
    lm_rate = 6.0 * n * lmw.hidden * lmw.vocab / l_s
    log(f"cpu oracle lm-head sample: {l_s:.2f}s, {lm_rate / 1e9:.1f} GFLOP/s")
    step_s = attn_flops_step / attn_rate + lm_flops_step / lm_rate
    return {
        "value": attn_rate / 1e12,
        "unit": "TFLOP/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"attention (the metric): trajectory 0 rows [0,{R}) x KV groups 0-1 "
                   f"({len(heads)} heads), fp32 LogitTree fwd+bwd, {a_s:.2f}s, rate in useful "
                   f"FLOPs 14 d P Hq; lm-head: {n} tokens x full vocab, fp32 fwd+bwd, {l_s:.2f}s "
                   f"({lm_rate / 1e12:.3f} TFLOP/s); whole step scaled by useful FLOPs "
                   f"= {step_s:.0f}s"),
        "lm_head_tflops": lm_rate / 1e12,
        "step_s": step_s,
    }


def time_sdcc(args, mv, synth, mask, wl, lmw, dev):
    """The SDCC junction KL (forward + student gradient) over the diverging
    leaves of the same packed batch, timed on its own after the step: teacher
    rows of a live-view pass, student rows of a final-walk pass (hidden states
    drawn like the LM head's), the LM head's vocabulary and width."""
    import torch
    _, rows_t, rows_s = mask.leaves()
    n = rows_t.numel()
    T, H, V = wl.total_tokens, lmw.hidden, lmw.vocab
    hT, w, _, _, _ = synth.make_logprob_inputs(T, H, V, args.seed, device="cuda")
    hS, _, _, _, _ = synth.make_logprob_inputs(T, H, V, args.seed + 1, device="cuda")
    rt, rs = rows_t.to(dev), rows_s.to(dev)
    dkl = torch.full((n,), 0.1, dtype=torch.float32, device=dev)   # lambda at the ramp's end
    s = mv.KLShape(n, H, V, T, T)
    import ctypes
    ws_f = torch.empty(int(mv.mv_sdcc_kl_workspace_bytes(ctypes.byref(s))), dtype=torch.uint8,
                       device=dev)
    ws_b = torch.empty(int(mv.mv_sdcc_kl_bwd_workspace_bytes(ctypes.byref(s))),
                       dtype=torch.uint8, device=dev)

    def kl_step():
        kl, lt, ls = mv.sdcc_kl(hT, rt, hS, rs, w, workspace=ws_f)
        mv.sdcc_kl_bwd(hT, rt, hS, rs, w, lt, ls, dkl, workspace=ws_b)
        return kl

    for _ in range(args.warmup):
        kl_step()
    torch.cuda.synchronize()
    mv.profile_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    stream = torch.cuda.current_stream()
    e0.record(stream)
    for _ in range(args.steps):
        kl = kl_step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    kt = {}
    for name in ("kl_logits", "kl_combine", "kl_grad", "kl_dh"):
        tot, cnt = mv.profile_read(name)
        if cnt:
            kt[name] = round(tot / cnt, 3)
    mv.profile_enable(False)
    flops = 10.0 * n * H * V
    tflops = flops / (ms * 1e-3) / 1e12
    log(f"sdcc: {n} leaves, {ms:.2f} ms fwd+bwd, {tflops:.0f} TFLOP/s")
    return {
        "leaves": n,
        "ms": round(ms, 3),
        "tflop": round(flops / 1e12, 3),
        "tflops": round(tflops, 2),
        "frac_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "leaves_per_s": round(n / (ms * 1e-3), 1),
        "kl_mean": round(float(kl.mean()), 5),
        "kernels_ms": kt,
        "flop_convention": "forward 4nHV (teacher + student logits), backward 6nHV "
                           "(both recomputed, then the student dH)",
    }


def time_dweight(args, mv, h, w, ws):
    """The LM-head weight gradient dW = G^T H over the step's tokens (G left in
    the backward workspace by the step), timed on its own: 2 T H V FLOPs."""
    import torch
    for _ in range(args.warmup):
        dw = mv.token_logprob_dweight(h, w, ws)
    torch.cuda.synchronize()
    mv.profile_enable(True)
    for _ in range(args.steps):
        dw = mv.token_logprob_dweight(h, w, ws)
    torch.cuda.synchronize()
    tot, cnt = mv.profile_read("lm_dw")
    mv.profile_enable(False)
    del dw
    ms = tot / cnt
    tflops = 2.0 * h.shape[0] * h.shape[1] * w.shape[0] / (ms * 1e-3) / 1e12
    log(f"lm-head dW: {ms:.2f} ms, {tflops:.0f} TFLOP/s")
    return {"ms": round(ms, 3), "tflops": round(tflops, 2),
            "frac_peak": round(tflops / PEAK_BF16_TFLOPS, 4)}


def time_grpo(args, mv, synth, h, w, y, old):
    """The forward with the GRPO loss and drift statistics fused into the
    log-prob's combine pass, against the log-prob forward followed by the
    stand-alone GRPO pass, on the step's LM-head inputs laid out as the
    recipe's groups (64 trajectories of 512 tokens, groups of 16)."""
    import torch
    T = h.shape[0]
    lengths = [512] * (T // 512)
    ptr, r, _, _, _, mask = synth.make_grpo_inputs(lengths, args.seed)
    gen = torch.Generator(device="cuda").manual_seed(synth.tensor_seed("grpo", args.seed))
    ref = old + 0.05 * torch.randn(T, generator=gen, device="cuda")
    pd, rd, md = ptr.cuda(), r.cuda(), mask.cuda()
    ws = mv.token_logprob_grpo_workspace(h, w, len(lengths), 16)
    lp_ws = mv.token_logprob_workspace(h, w)
    gr_ws = None

    def fused():
        return mv.token_logprob_grpo(h, w, y, old, pd, rd, ref, md, group_size=16, beta=0.001,
                                     workspace=ws)

    def two_calls():
        logp, ratio, clipped, lse = mv.token_logprob(h, w, y, old, 0.2, 0.28, workspace=lp_ws)
        return mv.grpo_loss(pd, rd, logp, old, ref, md, group_size=16, beta=0.001,
                            workspace=gr_ws)

    def run(fn, tail):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        mv.profile_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        kt = {}
        for name in ("lm_logits", "lm_combine") + tail:
            tot, cnt = mv.profile_read(name)
            if cnt:
                kt[name] = round(tot / args.steps, 4)
        mv.profile_enable(False)
        return e0.elapsed_time(e1) / args.steps, kt

    ms_f, kt_f = run(fused, ("grpo_prep", "grpo_finish"))
    ms_2, kt_2 = run(two_calls, ("grpo",))
    post_f = sum(v for n, v in kt_f.items() if n != "lm_logits")
    post_2 = sum(v for n, v in kt_2.items() if n != "lm_logits")
    del ws, lp_ws
    log(f"log-prob + GRPO forward: fused {ms_f:.3f} ms, two calls {ms_2:.3f} ms "
        f"(after the logits GEMM: {post_f:.3f} vs {post_2:.3f} ms)")
    return {"fused_ms": round(ms_f, 3), "two_calls_ms": round(ms_2, 3),
            "fused_kernels_ms": kt_f, "two_calls_kernels_ms": kt_2,
            "after_gemm_ms": {"fused": round(post_f, 4), "two_calls": round(post_2, 4)}}


def time_packed(args, mv, synth, trajs, wl, dev, shared):
    """One exact attention layer on a packed stream of the same batch's branch
    layers (the forms that stay exact through a stack of layers), from the
    physical tokens' Q, K, V to their gradients: Q and K gathered into the
    stream and rotated by per-branch positions in one pass each, V gathered,
    attention forward and backward under the stream's mask, dQ and dK rotated
    back and summed over their copies in one pass each, dV summed.  The same
    layer with separate rotary passes (gather, rotate; rotate back, sum) is
    timed beside it.  shared = False: every branch replicates its trunk
    (LogitTree's branch forwards); True: each branch stores only what it does
    not share with the branch before it and reads the shared trunk's keys in
    place.  Timed on its own after the step; useful FLOPs 14 d P Hq with P
    the stream's visible pairs."""
    import torch
    pk = mv.BranchPack(trajs, shared_trunk=shared).upload(dev)
    st = pk.stats()
    N = st["n_packed"]
    q, k, v, _ = synth.make_attn_tensors(ATTN_WORKLOAD, args.seed, device="cuda")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(synth.tensor_seed("packed", args.seed))
    do = torch.randn((N, wl.n_heads_q, wl.head_dim), generator=gen, device="cuda").to(torch.bfloat16)
    ws = mv.attn_bwd_workspace(pk.mask, do, torch.empty((N, wl.n_heads_kv, wl.head_dim),
                                                        dtype=torch.bfloat16, device="cuda"))
    theta = 1e6

    def layer_fused():
        qr, kr = mv.pack_rows_rope(pk, q, theta), mv.pack_rows_rope(pk, k, theta)
        vp = mv.pack_rows(pk, v)
        o, lse = mv.attn_fwd(pk.mask, qr, kr, vp)
        dq, dk, dv = mv.attn_bwd(pk.mask, qr, kr, vp, o, do, lse, workspace=ws)
        return (mv.unpack_rows_sum_rope(pk, dq, theta), mv.unpack_rows_sum_rope(pk, dk, theta),
                mv.unpack_rows_sum(pk, dv))

    def layer_separate():
        qr = mv.rope(pk, mv.pack_rows(pk, q), theta)
        kr = mv.rope(pk, mv.pack_rows(pk, k), theta)
        vp = mv.pack_rows(pk, v)
        o, lse = mv.attn_fwd(pk.mask, qr, kr, vp)
        dq, dk, dv = mv.attn_bwd(pk.mask, qr, kr, vp, o, do, lse, workspace=ws)
        mv.rope(pk, dq, theta, inverse=True, out=dq)
        mv.rope(pk, dk, theta, inverse=True, out=dk)
        return (mv.unpack_rows_sum(pk, dq), mv.unpack_rows_sum(pk, dk),
                mv.unpack_rows_sum(pk, dv))

    names = ("pack", "pack_rope", "rope", "attn_fwd", "attn_bwd_dkdv",
             "attn_bwd_reduce", "attn_bwd_dq", "unpack", "unpack_rope")

    def run(layer):
        for _ in range(args.warmup):
            layer()
        torch.cuda.synchronize()
        mv.profile_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        stream = torch.cuda.current_stream()
        e0.record(stream)
        for _ in range(args.steps):
            layer()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        kt = {}
        for name in names:
            tot, cnt = mv.profile_read(name)
            if cnt:
                kt[name] = round(tot / args.steps, 3)   # per layer (some run 2-3 times)
        mv.profile_enable(False)
        return ms, kt

    ms, kt = run(layer_fused)
    ms_sep, kt_sep = run(layer_separate)
    attn_ms = sum(x for n, x in kt.items() if n.startswith("attn"))
    useful = 14.0 * wl.head_dim * st["causal_pairs"] * wl.n_heads_q
    tflops = useful / (ms * 1e-3) / 1e12
    del q, k, v, do, ws
    torch.cuda.empty_cache()
    log(f"{'shared-trunk' if shared else 'replicated'} stream: N={N}, {ms:.2f} ms per exact layer "
        f"fwd+bwd incl. gathers ({attn_ms:.2f} ms attention kernels; {ms_sep:.2f} ms with "
        f"separate rotary passes), {tflops:.0f} TFLOP/s")
    return {
        "form": "shared trunk" if shared else "replicated trunk",
        "n_packed": N,
        "segments": st["n_segments"],
        "visible_pairs": st["causal_pairs"],
        "ms": round(ms, 3),
        "attn_ms": round(attn_ms, 3),
        "useful_tflops": round(tflops, 2),
        "frac_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "kernels_ms_per_layer": kt,
        "separate_rope": {"ms": round(ms_sep, 3), "kernels_ms_per_layer": kt_sep},
    }


def time_naive_compressed(args, mv, synth, trajs, wl, dev):
    """The Naive-Compressed baseline's attention (Section 3.3): each trajectory
    scored once over its final compressed walk (the C tokens no edit removes),
    plain causal, same heads; forward + backward."""
    import torch
    from paper_2609_00865_amd.synth import Trajectory
    lens = []
    for tr in trajs:
        gone = set()
        for e in tr.edits:
            for b, x in e.evict:
                gone.update(range(b, x))
            for b, x in getattr(e, "restore", ()):
                gone.difference_update(range(b, x))
        lens.append(tr.end - tr.begin - len(gone))
    comp, off = [], 0
    for n in lens:
        comp.append(Trajectory(off, off + n, ()))
        off += n
    m = mv.ViewMask(comp).upload(dev)
    P = m.stats()["visible_pairs"]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(synth.tensor_seed("compressed", args.seed))
    mk = lambda h: torch.randn((off, h, wl.head_dim), generator=gen, device="cuda").to(torch.bfloat16)
    q, k, v, do = mk(wl.n_heads_q), mk(wl.n_heads_kv), mk(wl.n_heads_kv), mk(wl.n_heads_q)
    ws = mv.attn_bwd_workspace(m, q, k)

    def f():
        o, lse = mv.attn_fwd(m, q, k, v)
        mv.attn_bwd(m, q, k, v, o, do, lse, workspace=ws)

    for _ in range(args.warmup):
        f()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        f()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    del q, k, v, do, ws
    torch.cuda.empty_cache()
    log(f"naive-compressed: {off} tokens, {ms:.2f} ms attention fwd+bwd")
    return {"tokens": off, "visible_pairs": P, "ms": round(ms, 3)}


def time_attention(args, mv, synth, workload, seed, dev):
    """View-masked attention forward + backward alone on one workload, timed
    with events on the launch stream (per-kernel durations from the library's
    own launch events)."""
    import torch
    wl = synth.ATTN_WORKLOADS[workload]
    trajs = synth.make_trajectories(workload, seed)
    b0 = time.perf_counter()
    mask = mv.ViewMask(trajs)
    build_ms = (time.perf_counter() - b0) * 1e3
    mask.upload(dev)
    st = mask.stats()
    q, k, v, do = synth.make_attn_tensors(workload, seed, device="cuda")
    ws = mv.attn_bwd_workspace(mask, q, k)

    def attn():
        o, lse = mv.attn_fwd(mask, q, k, v)
        mv.attn_bwd(mask, q, k, v, o, do, lse, workspace=ws)

    for _ in range(args.warmup):
        attn()
    torch.cuda.synchronize()
    mv.profile_enable(True)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        attn()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    kt = {}
    for name in ("attn_fwd", "attn_bwd_dkdv", "attn_bwd_reduce", "attn_bwd_dq"):
        tot, cnt = mv.profile_read(name)
        if cnt:
            kt[name] = round(tot / cnt, 3)
    mv.profile_enable(False)
    d, hq = wl.head_dim, wl.n_heads_q
    P = st["visible_pairs"]
    useful = 14.0 * d * P * hq
    tflops = useful / (ms * 1e-3) / 1e12
    fwd_ms = kt.get("attn_fwd", float("nan"))
    bwd_ms = sum(x for n, x in kt.items() if n != "attn_fwd")
    del q, k, v, do, ws
    torch.cuda.empty_cache()
    log(f"attention {workload} seed {seed}: {ms:.2f} ms fwd+bwd, {tflops:.0f} TFLOP/s "
        f"({tflops / PEAK_BF16_TFLOPS:.1%} of peak)")
    return {
        "workload": workload,
        "seed": seed,
        "shape": (f"{wl.n_traj} x {wl.traj_len} tokens, {wl.n_heads_q}/{wl.n_heads_kv} heads, "
                  f"d={d}"),
        "visible_pairs": P,
        "ms": round(ms, 3),
        "fwd_ms": round(fwd_ms, 3),
        "bwd_ms": round(bwd_ms, 3),
        "useful_tflop": round(useful / 1e12, 3),
        "useful_tflops": round(tflops, 2),
        "frac_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "trajectory_tokens_per_s": round(wl.total_tokens / (ms * 1e-3), 1),
        "fwd_frac_peak": round(4.0 * d * P * hq / (fwd_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "bwd_frac_peak": round(10.0 * d * P * hq / (bwd_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        # forward 4 and dQ 6 products over the forward tiles, dK/dV 8 over its own
        "executed_vs_useful": round((10.0 * st["fwd_tile_pairs"] + 8.0 * st["bwd_tile_pairs"])
                                    / (14.0 * P), 4),
        "kernels_ms": kt,
        "mask_build_ms": round(build_ms, 2),
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(each trajectory's attention and LM-head work runs on a single GPU).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_00865_amd import mv, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = synth.ATTN_WORKLOADS[ATTN_WORKLOAD]
    lmw = synth.LOGPROB_WORKLOADS[LM_WORKLOAD]

    # ---- inputs (resident in HBM before timing) ----
    trajs = synth.make_trajectories(ATTN_WORKLOAD, args.seed)
    b0 = time.perf_counter()
    mask = mv.ViewMask(trajs)
    build_ms = (time.perf_counter() - b0) * 1e3
    mask.upload(dev)
    st = mask.stats()
    P = st["visible_pairs"]
    log(f"mask built in {build_ms:.1f} ms: {st}")
    q, k, v, do = synth.make_attn_tensors(ATTN_WORKLOAD, args.seed, device="cuda")
    h, w, y, old, g = synth.make_logprob_inputs(lmw.n_tokens, lmw.hidden, lmw.vocab, args.seed,
                                                device="cuda")
    attn_ws = mv.attn_bwd_workspace(mask, q, k)
    lp_ws = mv.token_logprob_workspace(h, w)
    lpb_ws = mv.token_logprob_bwd_workspace(h, w)
    torch.cuda.synchronize()
    log("inputs resident")
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        o, lse = mv.attn_fwd(mask, q, k, v)
        mv.attn_bwd(mask, q, k, v, o, do, lse, workspace=attn_ws)
        if ev is not None:
            ev[1].record(stream)
        logp, ratio, clipped, lse_lm = mv.token_logprob(h, w, y, old, lmw.eps_low, lmw.eps_high,
                                                        workspace=lp_ws)
        mv.token_logprob_bwd(h, w, y, lse_lm, g, workspace=lpb_ws)

    for i in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    if args.calib_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("calibration copy of 1 GiB done")

    mv.profile_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    attn_ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(args.steps):
        step(attn_ev[i])
    e1.record(stream)
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ms_per_step = e0.elapsed_time(e1) / args.steps
    attn_ms = sum(a.elapsed_time(b) for a, b in attn_ev) / args.steps
    kt = {}
    for name in mv.KERNELS:
        tot, n = mv.profile_read(name)
        if n:
            kt[name] = {"ms_per_launch": tot / n, "launches": n}
    mv.profile_enable(False)
    bad = mv.token_logprob_bad_targets(lp_ws) + mv.token_logprob_bad_targets(lpb_ws)
    assert bad == 0, f"{bad} target ids outside the vocabulary"
    log(f"timed {args.steps} steps: {ms_per_step:.2f} ms/step (host wall {wall_ms:.2f}), "
        f"attention {attn_ms:.2f} ms")
    dweight = time_dweight(args, mv, h, w, lpb_ws)
    grpo = time_grpo(args, mv, synth, h, w, y, old)
    sdcc = None if args.no_sdcc else time_sdcc(args, mv, synth, mask, wl, lmw, dev)
    del h, w, y, old, g, lp_ws, lpb_ws
    torch.cuda.empty_cache()
    packed = shared = naive = None
    if not args.no_packed:
        packed = time_packed(args, mv, synth, trajs, wl, dev, shared=False)
        shared = time_packed(args, mv, synth, trajs, wl, dev, shared=True)
        naive = time_naive_compressed(args, mv, synth, trajs, wl, dev)
    others = []
    if not args.no_configs:
        del q, k, v, do, attn_ws
        torch.cuda.empty_cache()
        for wname, sd in ((ATTN_WORKLOAD, 1 - args.seed), ("long128k", 0), ("long128k", 1),
                          ("medium", 0)):
            others.append(time_attention(args, mv, synth, wname, sd, dev))

    d, hq = wl.head_dim, wl.n_heads_q
    T_lm, H, V = lmw.n_tokens, lmw.hidden, lmw.vocab
    attn_useful = 14.0 * d * P * hq
    lm_useful = 6.0 * T_lm * H * V
    step_flops = attn_useful + lm_useful
    af = attn_kernel_flops(st, d, hq)
    lf = lm_kernel_flops(T_lm, H, V)
    lm_ms = sum(kt[n]["ms_per_launch"] for n in kt if n.startswith("lm"))
    attn_kernels_ms = sum(kt[n]["ms_per_launch"] for n in kt if n.startswith("attn"))
    value = attn_useful / (attn_ms * 1e-3) / 1e12
    tokens = wl.total_tokens

    per_kernel = {}
    for n, x in kt.items():
        e = {"ms": round(x["ms_per_launch"], 3)}
        if n in af:
            for kind in ("useful", "executed"):
                r = af[n][kind] / (x["ms_per_launch"] * 1e-3) / 1e12
                e[f"{kind}_tflop"] = round(af[n][kind] / 1e12, 3)
                e[f"{kind}_tflops"] = round(r, 2)
                e[f"{kind}_frac_peak"] = round(r / PEAK_BF16_TFLOPS, 4)
        elif n in lf:
            r = lf[n] / (x["ms_per_launch"] * 1e-3) / 1e12
            e["tflops"] = round(r, 2)
            e["frac_peak"] = round(r / PEAK_BF16_TFLOPS, 4)
        per_kernel[n] = e

    def roofline(names, flops_of, label):
        dom = max((n for n in kt if n in names), key=lambda n: kt[n]["ms_per_launch"])
        ach = flops_of(dom) / (kt[dom]["ms_per_launch"] * 1e-3) / 1e12
        return {
            "bound": "mfma",
            "kernel": dom,
            "achieved": round(ach, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(ach / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic(dom),
            "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated)",
            "flops": label,
        }

    all_flops = {**{n: af[n]["useful"] for n in af}, **lf}
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": (f"{ATTN_WORKLOAD}: {wl.n_traj} x {wl.traj_len}-token packed trajectories, "
                         f"{wl.n_heads_q}/{wl.n_heads_kv} heads, d={d}, 16 edits/trajectory, "
                         f"view-masked attention fwd+bwd (value); the step also runs "
                         f"{LM_WORKLOAD}: {T_lm} tokens x {H} hidden x {V} vocab log-prob/"
                         f"ratio/clip fwd+bwd"),
            "global_batch": wl.n_traj,
            "seq_len": wl.traj_len,
            "parallelism": "single GPU",
            "seed": args.seed,
            "visible_pairs": P,
            "attention_useful_tflop_per_step": round(attn_useful / 1e12, 3),
        },
        "frac_peak": round(value / PEAK_BF16_TFLOPS, 4),
        "tokens_per_s": round(tokens / (attn_ms * 1e-3), 1),
        "attn": {
            "ms": round(attn_ms, 3),
            "kernels_ms_sum": round(attn_kernels_ms, 3),
            "useful_tflop": round(attn_useful / 1e12, 3),
            "useful_tflops": round(value, 2),
            "frac_peak": round(value / PEAK_BF16_TFLOPS, 4),
            "trajectory_tokens_per_s": round(tokens / (attn_ms * 1e-3), 1),
            "executed_vs_useful": round(sum(af[n]["executed"] for n in af) / attn_useful, 4),
        },
        "lmhead": {
            "ms": round(lm_ms, 3),
            "useful_tflops": round(lm_useful / (lm_ms * 1e-3) / 1e12, 2),
            "frac_peak": round(lm_useful / (lm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "tokens_per_s": round(T_lm / (lm_ms * 1e-3), 1),
            "dweight": dweight,
            "grpo_fused_forward": grpo,
        },
        "step": {
            "ms": round(ms_per_step, 3),
            "useful_tflop": round(step_flops / 1e12, 3),
            "useful_tflops": round(step_flops / (ms_per_step * 1e-3) / 1e12, 2),
            "frac_peak": round(step_flops / (ms_per_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
            "host_wall_ms": round(wall_ms, 3),
        },
        "kernels": per_kernel,
        "mask_build_ms": round(build_ms, 2),
        "roofline": roofline(all_flops, lambda n: all_flops[n],
                             "algorithmic FLOPs per launch (attention kernels: useful)"),
        "roofline_attention": roofline(af, lambda n: af[n]["useful"],
                                       "useful FLOPs per launch (visible pairs only)"),
    }
    if others:
        out["attention_configs"] = others
    if sdcc is not None:
        out["sdcc"] = sdcc
    if packed is not None:
        for pk in (packed, shared):
            pk["pairs_vs_union"] = round(pk["visible_pairs"] / P, 4)
            pk["attn_ms_vs_union"] = round(pk["attn_ms"] / attn_ms, 4)
        out["branch_packed"] = packed
        out["shared_trunk_packed"] = shared
        nc = naive["ms"]
        out["cost_ratios"] = {
            "what": ("attention fwd+bwd of one layer over the 4 x 32K batch, each relative to "
                     "the Naive-Compressed form (final compressed walk, plain causal)"),
            "naive_compressed_ms": nc,
            "naive_compressed_tokens": naive["tokens"],
            "union_4d_mask": round(attn_ms / nc, 3),
            "logittree_shared_trunk": round(shared["attn_ms"] / nc, 3),
            "logittree_replicated_trunk": round(packed["attn_ms"] / nc, 3),
            "paper_table_main_context": {"4D mask": 1.35, "LogitTree": 4.20,
                                         "note": "whole training step multipliers over "
                                                 "Naive-Compressed, Qwen3-4B, A100/H800-class; "
                                                 "context, not this measurement"},
        }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(trajs, wl, lmw, attn_useful, lm_useful)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
