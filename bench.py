#!/usr/bin/env python3
"""Benchmark of the packed pair-state hot path on one MI355X.

One step = one pass of the whole workload over its batch, every op one launch
over all samples.  Default workload: the four-block Pairformer-style stack
(B=16, lognormal lengths around 192 clipped to [16, 768], C_s=384, C_z=128,
4 heads x 32, transition 128->512->128, bf16 with fp32 accumulation); each
block is pair broadcast, outgoing and incoming triangle updates, row and
column attention with pair bias, the SwiGLU transition and the column mean
back to the single track.  value = blocks x sum N^2 / step time (valid pair
positions per second per pair block).

The same JSON line nests the near-uniform (B=8, 208..224) and high-variation
(B=8, 32..512) single pair blocks, the packed-token encoder layer (tokens per
second) and the training step (forward, joint diagnostic loss, backward) of
the single-pair-single program on square and rectangular pairs, each timed
the same way.  Step times are reported warm (steps
back to back) and cold (a 512 MB write flushes the memory-side cache before
each step), as median, p10 and p90.

--gpus N > 1 is rejected: the path runs on one GPU.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "valid pair positions/sec per pair block (1 MI355X) + % HBM / MFMA roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 matrix cores, TFLOP/s
F32_PEAK_TFLOPS = 157.3        # fp32 vector


# Measured HBM traffic per launch of each op's kernels: rocprofv3 --pmc
# FETCH_SIZE and --pmc WRITE_SIZE passes (KiB per dispatch, summed over the
# op's kernels), per workload, tagged with a hash of the kernel's source file
# (plus the shared device header) at the time the counters were taken.  A
# plain 256 MiB device copy reads 131,087 KiB on FETCH_SIZE and 262,144 KiB on
# WRITE_SIZE, so bytes = 2.0 x FETCH_SIZE + 1.0 x WRITE_SIZE.  When the source
# hash no longer matches, the kernel has changed since the counters and
# traffic is null.
FETCH_SCALE, WRITE_SCALE = 2.0, 1.0
COUNTERS = {  # workload: {op: (kernel source, source hash, FETCH_SIZE KiB, WRITE_SIZE KiB)}
    "pairformer4_b16_lognormal192_bf16": {
        "attention_row": ("k_attention.hip", "87a973263a55fff9", 321637 + 8058, 174371 + 6472),
        "attention_col": ("k_attention.hip", "87a973263a55fff9", 321637 + 8058, 174371 + 6472),
        "triangle_out": ("k_triangle.hip", "78ed89d0163e3191", 637979, 175997),
        "triangle_in": ("k_triangle.hip", "78ed89d0163e3191", 637979, 175997),
        "transition": ("k_transition.hip", "fc86ddcdca398fdb", 102020 + 268, 174369 + 384),
        "attn_proj": ("k_linear.hip", "8c9d00dd2754951b", 87689, 528988),
        "tri_proj": ("k_linear.hip", "8c9d00dd2754951b", 87748, 386304),
        "attn_out_residual": ("k_linear.hip", "8c9d00dd2754951b", 174601, 174370),
        "pair_broadcast": ("k_segment.hip", "28f1c83801f4cc17", 68891, 174369),
        "segment_mean": ("k_segment.hip", "28f1c83801f4cc17", 87298, 1492),
        "single_proj": ("k_linear.hip", "8c9d00dd2754951b", 5282, 1492),
        "single_update": ("k_linear.hip", "8c9d00dd2754951b", 6023, 2237),
    },
    "pair_b8_n208_224_bf16": {
        "transition": ("k_transition.hip", "e2f701d5925d7f6e", 53091, 91003),
        "segment_mean": ("k_segment.hip", "c95eabc6d4c62896", 45570, 853),
    },
}


def source_hash(fname: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in (fname, "nt_device.h"):
        with open(os.path.join(ROOT, "paper_2609_30379_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(op: str, workload: str):
    """HBM bytes per launch from the committed counters, or None when they do
    not apply (no counters for this workload and op, or the kernel source
    changed since they were taken)."""
    entry = COUNTERS.get(workload, {}).get(op)
    if entry is None:
        return None
    src, tag, fetch_kib, write_kib = entry
    if source_hash(src) != tag:
        return None
    return int((FETCH_SCALE * fetch_kib + WRITE_SCALE * write_kib) * 1024)


def op_costs(w, L):
    """Algorithmic HBM bytes and flops per launch of every op of one block
    (bf16 storage = 2 bytes; every tensor read or written once)."""
    R = sum(n * n for n in L)
    S = sum(L)
    N3 = sum(n ** 3 for n in L)
    C, Cs, H, d, F = w.c_z, w.c_s, w.heads, w.head_dim, w.hidden
    e = 2 if w.dtype == "bf16" else 4
    c = {
        "single_proj": (S * (Cs + 2 * C) * e, 2 * S * Cs * 2 * C),
        # the stacks' broadcast accumulates into the pair state (z read and
        # written) in every block but the first, so the median launch is an
        # accumulating one
        "pair_broadcast": (2 * R * C * e + 2 * S * C * e, R * C),
        "ln_linear": (R * 2 * C * e, 2 * R * C * C),
        "bcast_ln_linear": (2 * S * C * e + R * C * e, R * C + 2 * R * C * C),
        "attn_proj": (R * (C + 3 * C + H) * e, 2 * R * C * (3 * C + H)),
        "attention_row": (R * (4 * H * d + H) * e, 4 * H * d * N3),
        "attention_col": (R * (4 * H * d + H) * e, 4 * H * d * N3),
        "attn_out_residual": (R * 3 * C * e, 2 * R * C * C),
        "tri_proj": (R * 3 * C * e, 2 * R * C * 2 * C),
        "triangle_out": (R * 4 * C * e, 2 * C * N3),
        "triangle_in": (R * 4 * C * e, 2 * C * N3),
        "transition": (R * 2 * C * e, 2 * R * (C * 2 * F + F * C)),
        "segment_mean": (R * C * e + S * C * 4, R * C),
        "single_update": (S * (C * 4 + 2 * Cs * e), 2 * S * C * Cs),
        # gated (AlphaFold 3 form) steps: [q|k|v|g] + bias projection; gated
        # attention (q, k, v, g, bias read, o written); [a_p|a_g|b_p|b_g] and
        # g projections (z read twice); the contraction on gated operands
        # (a_p, a_g, b_p, b_g read, t written); LN(t) W_o gated residual (t,
        # g, z read, z written)
        "attn_proj_g": (R * (C + 4 * C + H) * e, 2 * R * C * (4 * C + H)),
        "attention_row_g": (R * (5 * H * d + H) * e, 4 * H * d * N3),
        "attention_col_g": (R * (5 * H * d + H) * e, 4 * H * d * N3),
        "tri_proj_g": (R * (2 * C + 5 * C) * e, 2 * R * C * 5 * C),
        "triangle_out_g": (R * 5 * C * e, 2 * C * N3),
        "triangle_in_g": (R * 5 * C * e, 2 * C * N3),
        "tri_out_gated_residual": (R * 4 * C * e, 2 * R * C * C),
    }
    return c


def token_op_costs(w, L):
    """Algorithmic HBM bytes and flops per launch of the token-path ops (one
    pre-LN encoder layer on packed tokens and the per-sample mean pool)."""
    T = sum(L)
    S2 = sum(n * n for n in L)
    c, F = w.c_s, w.hidden
    e = 2 if w.dtype == "bf16" else 4
    return {
        "qkv_proj": (T * (c + 3 * c) * e, 2 * T * c * 3 * c),
        "attention_1d": (T * 4 * c * e, 4 * c * S2),
        "out_proj_residual": (T * 3 * c * e, 2 * T * c * c),
        "ffn_up_gelu": (T * (c + F) * e, 2 * T * c * F),
        "ffn_down_residual": (T * (F + 2 * c) * e, 2 * T * F * c),
        "sample_mean": (T * c * e + len(L) * c * 4, T * c),
    }


def mechanism_op_costs(w, L, M):
    """Algorithmic HBM bytes and flops per launch of the ops of one training
    step of the single-pair-single program (forward, loss, backward); M is
    None for square pairs.  bf16 tensors 2 bytes, fp32 4."""
    # non-leading layout: every packed position holds s_axis feature vectors,
    # so each count of positions below is s_axis times larger
    Sx = w.s_axis
    S = sum(L) * Sx
    Mc = S if M is None else sum(M)
    cells = (sum(n * n for n in L) if M is None else sum(n * m for n, m in zip(L, M))) * Sx
    C, Cp, F = w.c_s, w.c_z, w.hidden
    xin = (S + (0 if M is None else Mc)) * C * 2
    return {
        "mech_proj": (xin + (S + Mc) * Cp * 2, 2 * (S + Mc) * C * Cp),
        "mech_broadcast": (cells * Cp * 2 + (S + Mc) * Cp * 2, cells * Cp),
        "mech_transition": (cells * Cp * 2 * 2, 2 * cells * (Cp * 2 * F + F * Cp)),
        "mech_column_mean": (cells * Cp * 2 + S * Cp * 4, cells * Cp),
        "mech_single_update": (S * (Cp * 4 + 2 * C * 2), 2 * S * Cp * C),
        "mech_loss": (2 * S * C * 2 + cells * Cp * 2 + S * C * (2 + 4) + cells * Cp * 2, 3 * (2 * S * C) + 3 * cells * Cp),
        "mech_single_update_bwd": (S * Cp * 4 * 2 + S * C * 2, 2 * 2 * S * C * Cp),
        "mech_column_mean_bwd": (S * Cp * 4 + cells * Cp * 2 * 2, cells * Cp),
        "mech_transition_bwd": (cells * Cp * 2 * 3, 2 * cells * Cp * 8 * F),
        "mech_broadcast_bwd": (cells * Cp * 2 * 2 + (S + Mc) * Cp * 2, 2 * cells * Cp),
        "mech_proj_bwd": (xin + (S + Mc) * Cp * 2 + S * C * 4 * 2 + (0 if M is None else Mc * C * 4),
                          2 * 2 * (S + Mc) * C * Cp),
    }


def roofline_for(name, bytes_, flops, us, dtype):
    """Bound = whichever of HBM time and matrix-core time is longer."""
    peak_f = BF16_PEAK_TFLOPS if dtype == "bf16" else F32_PEAK_TFLOPS
    t_hbm = bytes_ / (HBM_PEAK_GBS * 1e9)
    t_mma = flops / (peak_f * 1e12)
    if t_mma > t_hbm:
        ach = flops / (us * 1e-6) / 1e12
        return {"kernel": name, "bound": "mfma", "achieved": round(ach, 2), "peak": peak_f, "unit": "TFLOP/s",
                "frac": round(ach / peak_f, 4), "traffic": None}
    ach = bytes_ / (us * 1e-6) / 1e9
    return {"kernel": name, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": None}


def cpu_baseline_tokens(w, run, min_s: float = 10.0):
    """The CPU oracle on the token path: one encoder layer over samples taken
    smallest first until at least min_s seconds of work; tokens per second."""
    import numpy as np
    from oracle import blocks as OB
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    eta = np.concatenate([[0], np.cumsum(run.lengths)])
    done, tokens, dt = [], 0, 0.0
    for i in np.argsort(run.lengths, kind="stable"):
        n = int(run.lengths[i])
        t0 = time.perf_counter()
        OB.encoder_layer(run.x_init[eta[i]:eta[i] + n], [n], run.params, w.heads, w.head_dim, dtype=w.dtype)
        dt += time.perf_counter() - t0
        done.append(f"{int(i)} (N={n})")
        tokens += n
        if dt >= min_s:
            break
    return {"value": round(tokens / dt, 1), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"samples {', '.join(done[:8])}{' ...' if len(done) > 8 else ''} of the batch ({tokens} tokens), "
                      f"one encoder layer each in float64 NumPy, {dt:.1f} s; host has {os.cpu_count()} CPUs"}


def cpu_baseline(w, run, min_s: float = 10.0):
    """The CPU oracle timed on this host: the whole workload (every block) on
    samples of the batch taken smallest first, one at a time, until at least
    min_s seconds of work.  The oracle's time is dominated by the per-sample
    N^3 contractions, so the time of the whole batch is estimated as the
    measured time scaled by the batch's sum N^3 over the timed samples'."""
    import numpy as np
    from oracle import blocks as OB
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    dims = dict(c_z=w.c_z, heads=w.heads, head_dim=w.head_dim)
    eta = np.concatenate([[0], np.cumsum(run.lengths)])
    done, n3, dt = [], 0, 0.0
    for i in np.argsort(run.lengths, kind="stable"):
        n = int(run.lengths[i])
        s = run.s_init[eta[i]:eta[i] + n]
        t0 = time.perf_counter()
        z = None
        for b in range(w.blocks):
            steps = w.steps if b == 0 else tuple(t for t in w.steps if t != "lin")
            s, z, _ = OB.pair_block(s, [n], run.params[b], dims, steps, z=z, dtype=w.dtype)
        dt += time.perf_counter() - t0
        done.append(f"{int(i)} (N={n})")
        n3 += n ** 3
        if dt >= min_s:
            break
    total_n3 = sum(int(n) ** 3 for n in run.lengths)
    est = dt * total_n3 / n3
    positions = w.blocks * sum(int(n) ** 2 for n in run.lengths)
    return {"value": round(positions / est, 1), "unit": "pair positions/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"samples {', '.join(done)} of the batch, every block in float64 NumPy, {dt:.1f} s; "
                      f"they hold {n3 / total_n3:.1%} of the batch's sum N^3, so the whole batch is estimated at "
                      f"{est:.1f} s ({positions} pair positions over {w.blocks} block(s)); "
                      f"host has {os.cpu_count()} CPUs"}


def bench_single_attention(args, w):
    """Single attention with pair bias (axis 3) alone, on the workload's
    lengths with C_s / 32 heads of 32: q, k, v, o token-major, the bias from
    the pair state.  value = query-key scores per second (H * sum N^2 / t)."""
    import torch
    from paper_2609_30379_amd import binding, synth
    L = [int(n) for n in synth.lengths_for(w)]
    H, d = w.c_s // 32, 32
    T, R = sum(L), sum(n * n for n in L)
    lay = binding.NestedLayout(L)
    qkv = torch.from_numpy(synth.normal(w.seed, "single_attn_qkv", (T, 3 * H * d), dtype="bf16")).to("cuda", torch.bfloat16)
    bias = torch.from_numpy(synth.normal(w.seed, "single_attn_bias", (H, R), dtype="bf16")).to("cuda", torch.bfloat16)
    o = torch.empty((T, H * d), dtype=torch.bfloat16, device="cuda")
    c = H * d
    ws = binding.workspace_tensor(binding.attention_workspace_bytes(lay, 3, H, d, "bf16", True))
    call = lambda: binding.nt_pair_row_attention(lay, 3, H, d, qkv[:, :c], qkv[:, c:2 * c], qkv[:, 2 * c:], o,  # noqa: E731
                                                 bias=bias, bias_layout="heads", workspace=ws)
    for _ in range(max(1, args.warmup)):
        call()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        call()
    ev1.record(stream)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    us = ev0.elapsed_time(ev1) * 1e3 / args.steps
    nbytes = (4 * T * c + H * R) * 2
    flops = 4 * H * d * R
    line = {"metric": "query-key scores/sec, single attention with pair bias (1 MI355X)",
            "value": round(H * R / (ms * 1e-3), 1), "unit": "scores/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": w.name + "_single_attention", "lengths": L, "heads": H, "head_dim": d},
            "roofline": {"bound": "hbm", "achieved": round(nbytes / (us * 1e-6) / 1e9, 2), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                         "traffic": None, "algorithmic_bytes": nbytes, "us_per_launch": round(us, 2),
                         "mfma_frac": round(flops / (us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4)}}
    if not args.no_cpu_baseline:
        # the oracle on the smallest sample, scaled to scores per second
        from oracle import ops as oracle_ops
        n = min(L)
        q1 = qkv[:n].float().cpu().numpy()
        b1 = bias[:, :n * n].float().cpu().numpy().T
        t0, reps = time.perf_counter(), 0
        while time.perf_counter() - t0 < 1.0:
            oracle_ops.single_attention_pair_bias(q1[:, :c], q1[:, c:2 * c], q1[:, 2 * c:], b1, [n], H, d)
            reps += 1
        dt = (time.perf_counter() - t0) / reps
        line["cpu_baseline"] = {"value": round(H * n * n / dt, 1), "unit": "scores/s", "cores": torch.get_num_threads(),
                                "kind": "oracle", "sample": f"one sample of N={n}, {reps} runs"}
    print(json.dumps(line), flush=True)


def bench_cross_attention(args, w):
    """Cross-attention alone (queries and keys ragged differently): queries on
    the packed-token workload's lengths, keys and values on lengths from the
    same distribution drawn with the next seed, hidden 768 as 12 heads of 64.
    value = query-key scores per second (H * sum N_i M_i / t)."""
    import numpy as np
    import torch
    from paper_2609_30379_amd import binding, synth
    wt = synth.WORKLOADS["tokens_b64_lognormal230_bf16"]
    Lq = [int(n) for n in synth.lengths_for(wt)]
    Lk = [int(n) for n in synth.lengths_for(wt, seed=wt.seed + 1)]
    H, d = wt.heads, wt.head_dim
    c = H * d
    Tq, Tk, NM = sum(Lq), sum(Lk), sum(n * m for n, m in zip(Lq, Lk))
    lq, lk = binding.NestedLayout(Lq), binding.NestedLayout(Lk)
    q = torch.from_numpy(synth.normal(wt.seed, "cross_q", (Tq, c), dtype="bf16")).to("cuda", torch.bfloat16)
    kv = torch.from_numpy(synth.normal(wt.seed, "cross_kv", (Tk, 2 * c), dtype="bf16")).to("cuda", torch.bfloat16)
    o = torch.empty((Tq, c), dtype=torch.bfloat16, device="cuda")
    call = lambda: binding.nt_cross_attention(lq, lk, H, d, q, kv[:, :c], kv[:, c:], o)  # noqa: E731
    ms, us = _time_call(call, args)
    nbytes = (2 * Tq * c + 2 * Tk * c) * 2
    flops = 4 * H * d * NM
    line = {"metric": "query-key scores/sec, cross-attention with different query and key lengths (1 MI355X)",
            "value": round(H * NM / (ms * 1e-3), 1), "unit": "scores/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "cross_attention_b64_lognormal230_bf16", "q_lengths": Lq, "kv_lengths": Lk,
                       "heads": H, "head_dim": d},
            "roofline": {"bound": "hbm", "achieved": round(nbytes / (us * 1e-6) / 1e9, 2), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                         "traffic": None, "algorithmic_bytes": nbytes, "us_per_launch": round(us, 2),
                         "mfma_frac": round(flops / (us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4)}}
    if not args.no_cpu_baseline:
        from oracle import ops as oracle_ops
        i = int(np.argmin([n * m for n, m in zip(Lq, Lk)]))
        q1 = q[sum(Lq[:i]):sum(Lq[:i + 1])].float().cpu().numpy()
        kv1 = kv[sum(Lk[:i]):sum(Lk[:i + 1])].float().cpu().numpy()
        t0, reps = time.perf_counter(), 0
        while time.perf_counter() - t0 < 1.0:
            oracle_ops.attention_1d(q1, kv1[:, :c], kv1[:, c:], [Lq[i]], H, d, kv_lengths=[Lk[i]])
            reps += 1
        dt = (time.perf_counter() - t0) / reps
        line["cpu_baseline"] = {"value": round(H * Lq[i] * Lk[i] / dt, 1), "unit": "scores/s",
                                "cores": torch.get_num_threads(), "kind": "oracle",
                                "sample": f"sample {i} alone (N={Lq[i]} queries, M={Lk[i]} keys), {reps} runs"}
    print(json.dumps(line), flush=True)


def _time_call(call, args):
    """(host ms, device us) per call over args.steps calls after args.warmup,
    HIP events on the launch stream."""
    import torch
    for _ in range(max(1, args.warmup)):
        call()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        call()
    ev1.record(stream)
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / args.steps, ev0.elapsed_time(ev1) * 1e3 / args.steps


def _pct(xs, q):
    import numpy as np
    return round(float(np.percentile(np.asarray(xs), q)), 4)


def measure(w, steps: int, warmup: int, graph: bool = False, cpu: bool = False):
    """Times `steps` steps of workload w; returns the result dict."""
    import torch
    from paper_2609_30379_amd import blocks
    tokens = w.kind == "tokens"
    mech = w.kind == "mechanism"
    run = blocks.TokenRun(w) if tokens else (blocks.MechanismRun(w) if mech else blocks.PairRun(w))
    L = run.lengths
    R, S = sum(n * n for n in L), sum(L)
    if mech and run.rect:
        R = sum(n * m for n, m in zip(L, run.cols))
    if mech:                                      # non-leading: s_axis pair positions per packed cell
        R, S = R * w.s_axis, S * w.s_axis
    stream = torch.cuda.current_stream()          # the stream every nt_* call launches on

    for _ in range(max(1, warmup)):
        ref = [t.clone() for t in run.step() if t is not None]
    torch.cuda.synchronize()

    # With graph=True the step is captured once into a HIP graph and replayed
    # in the timed region, after checking that a replay reproduces the eager
    # step bit for bit (otherwise, and by default, eager steps are timed).
    g = None
    if graph:
        try:
            gg = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gg):
                outs = [t for t in run.step() if t is not None]
            gg.replay()
            torch.cuda.synchronize()
            if all(torch.equal(a, b) for a, b in zip(ref, outs)):
                g = gg
            else:
                print("bench.py: graph replay differs from the eager step; timing eager steps", file=sys.stderr)
        except Exception as e:                       # capture unsupported: time eager steps
            print(f"bench.py: graph capture failed ({e}); timing eager steps", file=sys.stderr)
        torch.cuda.synchronize()
    step = g.replay if g is not None else run.step

    # timed region: events at every step boundary on the launch stream (one
    # event between steps adds no gap inside a step), wall clock around it
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    evs[0].record(stream)
    for k in range(steps):
        step()
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / steps
    warm = [evs[k].elapsed_time(evs[k + 1]) for k in range(steps)]

    # cold steps: a 512 MB write evicts the 256 MB memory-side cache before
    # each step, outside the step's events
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    cold = []
    for _ in range(max(3, min(steps, 20))):
        flush.fill_(1)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        step()
        b.record(stream)
        torch.cuda.synchronize()
        cold.append(a.elapsed_time(b))
    del flush

    # per-op attribution: eager steps with an event pair around every op on
    # the launch stream (a captured graph cannot carry timing events)
    tm = blocks.OpTimer()
    blocks.timer = tm
    torch.cuda.synchronize()
    for _ in range(steps):
        run.step()
    torch.cuda.synchronize()
    blocks.timer = None
    per_op = tm.summary()                            # {op: (launches, median us per launch)}

    costs = token_op_costs(w, L) if tokens else (mechanism_op_costs(w, L, run.cols) if mech else op_costs(w, L))
    total_us = {k: n * us / steps for k, (n, us) in per_op.items()}
    dominant = max(total_us, key=total_us.get)
    n_launch, us_launch = per_op[dominant]
    rl = roofline_for(dominant, costs[dominant][0], costs[dominant][1], us_launch, w.dtype)
    rl["traffic"] = measured_traffic(dominant, w.name)
    rl["algorithmic_bytes"] = costs[dominant][0]
    rl["algorithmic_flops"] = costs[dominant][1]
    rl["us_per_launch"] = round(us_launch, 2)
    rl["launches_per_step"] = n_launch // steps
    kernels = {}
    for k, (n, us) in per_op.items():
        r = roofline_for(k, costs[k][0], costs[k][1], us, w.dtype)
        kernels[k] = {"us": round(us, 2), "launches_per_step": n // steps, "bound": r["bound"],
                      "frac": r["frac"], "algorithmic_bytes": costs[k][0],
                      "traffic": measured_traffic(k, w.name)}
    timing = {"warm_ms": {"median": _pct(warm, 50), "p10": _pct(warm, 10), "p90": _pct(warm, 90)},
              "cold_ms": {"median": _pct(cold, 50), "p10": _pct(cold, 10), "p90": _pct(cold, 90),
                          "reps": len(cold)},
              "op_sum_ms": round(sum(total_us.values()) / 1e3, 4)}
    if mech:
        out = {"metric": "valid pair positions/sec per training step (forward + loss + backward) of the "
                         "single-pair-single program (1 MI355X)",
               "value": round(R / (ms * 1e-3), 1), "unit": "pair positions/s",
               "tokens_per_s": round(S / (ms * 1e-3), 1),
               "config": {"workload": w.name, "batch": w.batch, "lengths": L, "cols": run.cols, "sum_n": S,
                          "pair_cells": R, "s_axis": w.s_axis, "c": w.c_s, "c_p": w.c_z, "hidden": w.hidden,
                          "step": "forward, joint diagnostic loss, backward of every parameter and input"}}
    elif tokens:
        out = {"metric": "packed tokens/sec per encoder layer (1 MI355X)", "value": round(S / (ms * 1e-3), 1),
               "unit": "tokens/s",
               "config": {"workload": w.name, "batch": w.batch, "lengths": L, "sum_n": S, "sum_n2": R,
                          "c": w.c_s, "heads": w.heads, "head_dim": w.head_dim, "hidden": w.hidden}}
    else:
        out = {"metric": METRIC, "value": round(w.blocks * R / (ms * 1e-3), 1), "unit": "pair positions/s",
               "tokens_per_s": round(w.blocks * S / (ms * 1e-3), 1),
               "config": {"workload": w.name, "batch": w.batch, "lengths": L, "sum_n": S, "sum_n2": R,
                          "c_s": w.c_s, "c_z": w.c_z, "heads": w.heads, "head_dim": w.head_dim,
                          "hidden": w.hidden, "blocks": w.blocks, "steps_per_block": list(w.steps)}}
    out.update({"ms_per_step": round(ms, 4), "graph": g is not None, "timing": timing, "roofline": rl,
                "kernels": kernels})
    if cpu:
        out["cpu_baseline"] = cpu_baseline_tokens(w, run) if tokens else cpu_baseline(w, run)
    return out


NESTED = ("pair_b8_n208_224_bf16", "pair_b8_n32_512_bf16", "pairformer4_gated_b16_lognormal192_bf16",
          "tokens_b64_lognormal230_bf16", "mechanism_square_b8_n66_317_bf16",
          "mechanism_rect_b8_n66_307_m66_309_bf16", "mechanism_nonleading_s3_b8_n40_182_bf16")


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="pairformer4_b16_lognormal192_bf16",
                    help="headline workload (default: the four-block stack, the largest single-GPU workload)")
    ap.add_argument("--no-nested", action="store_true", help="time only the headline workload")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true", help="time replays of the step captured into a HIP graph")
    ap.add_argument("--kernels", action="store_true", help="also print the per-op breakdown to stderr")
    ap.add_argument("--op", choices=["single_attention", "cross_attention"], default=None,
                    help="time one widened op alone instead of the pair block (its own JSON line)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 256 MiB device-to-device copy (scale reference for HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this path runs on one GPU; --gpus {args.gpus} is not supported "
              "(samples are independent, see the sharding notes in the design document)", file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        import torch
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_per_launch": src.numel() * 4, "launches": args.steps}), flush=True)
        return

    import torch
    from paper_2609_30379_amd import binding, synth
    binding.load()
    w = synth.WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    if args.op == "single_attention":
        bench_single_attention(args, w)
        return
    if args.op == "cross_attention":
        bench_cross_attention(args, w)
        return
    head = measure(w, args.steps, args.warmup, args.graph, cpu=not args.no_cpu_baseline)
    out = {"metric": head.pop("metric"), "value": head.pop("value"), "unit": head.pop("unit"),
           "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": head.pop("ms_per_step"),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
           "config": head.pop("config")}
    out.update(head)
    if not args.no_nested:
        nested = {}
        for name in NESTED:
            if name == w.name:
                continue
            r = measure(synth.WORKLOADS[name], args.steps, args.warmup, args.graph, cpu=False)
            if synth.WORKLOADS[name].kind != "mechanism" and "gated" not in name:
                r.pop("kernels")
            nested[name] = r
        out["other_workloads"] = nested
    if args.kernels:
        for k, v in sorted(out["kernels"].items(), key=lambda kv: -kv[1]["us"] * kv[1]["launches_per_step"]):
            tr = v["traffic"]
            ratio = f"  traffic/alg {tr / v['algorithmic_bytes']:.2f}" if tr else ""
            print(f"{k:20s} {v['us']:9.2f} us x{v['launches_per_step']}  {v['bound']} frac {v['frac']:.3f}{ratio}",
                  file=sys.stderr)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
