#!/usr/bin/env python3
"""Benchmark: block-diffusion masked attention, forward + backward, on one MI355X.

One step = bd_attn_fwd + bd_attn_bwd over one batch of the 8B-shaped training
workload (B=2, Hq=32, Hkv=8, D=128, L=2048 so 4096 packed tokens, S=4, bf16
N(0,1)*0.5 inputs, dO ~ N(0,1)), inputs resident in HBM (warm caches: the
working set fits the 256 MB Infinity Cache).  First a clock-settle phase of
untimed steps for a fixed wall time (250 ms by default, reported as
`settle_ms`: the GPU's clocks settle only after tens of milliseconds under
load), then W untimed warm-up steps (10), then K timed steps (50) bracketed
by device synchronisation and HIP events on the stream the library runs on;
the per-step median is reported beside the mean.

value  = effective TFLOP/s counting only visible (query, key) pairs:
         (4 + 10) * D * N_visible * B * Hq per step (forward 4D, backward 10D per
         visible pair, the FlashAttention convention).
roofline: the dominant kernel's algorithmic FLOPs per launch over its average
         duration, from events that its dispatches record as they begin and
         end (no packets of their own between the kernels) in every fourth
         timed step, against the bf16 dense MFMA peak.
kernels: per kernel the event-timed duration and algorithmic rate, and, from
         the committed rocprofv3 counter record of the same kernel sources
         (profiles/bd_attn_8b_counters.md), the executed MFMA rate over this
         run's duration, the MFMA and LDS busy fractions the counters showed and
         the HBM bytes per launch and GB/s.
cpu_baseline: the fp64 oracle (test infrastructure) timed on the host cores on
         a bounded sample of the same workload (whole GQA groups).
packed:  the same step over packed sequences of mixed lengths (the same heads,
         4096 tokens per copy in all) through the varlen calls, reported
         beside the headline (not part of `value`).
lce:     token log-probabilities through the 8B LM head (4096 scored positions,
         151,936 vocabulary rows, hidden 4096): forward (GEMM with fused
         softmax statistics), the Eq. 7 objective, backward (recomputed
         logits -> g, dH = g W, dW = g^T H); GEMM FLOPs over the event-timed
         duration against the bf16 dense peak (not part of `value`).
decode:  one block-decoding call over a KV cache (64 rollouts of the 8B
         shape, caches of 512..8192 tokens, blocks of 4): HBM bytes the call
         must move (cached K/V rows up to each length, the block's K/V, Q, O,
         LSE) over its duration, against the 8 TB/s HBM peak (not part of
         `value`).

Prints exactly one JSON line on stdout; details go to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 bf16 FLOP/clk x 2.4 GHz (dense)
METRIC = "effective TFLOP/s (unmasked FLOPs) bd_attn fwd+bwd, 8B shape, % of bf16 peak"


def visible_pairs(L: int, S: int) -> int:
    """Visible (query, key) pairs per (batch, head): sum over blocks of
    2 s_j (P_j + s_j), s_j the block size and P_j the tokens before it."""
    S = min(S, L)
    total, prefix = 0, 0
    for a in range(0, L, S):
        s = min(S, L - a)
        total += 2 * s * (prefix + s)
        prefix += s
    return total


def log(msg: str):
    print(msg, file=sys.stderr, flush=True)


HERE = os.path.dirname(os.path.abspath(__file__))
MARK_EVERY = 4  # timed steps per step that records the per-kernel dispatch events
COUNTERS_FILE = os.path.join(HERE, "profiles", "bd_attn_8b_counters.md")


def kernel_source_hash() -> str:
    """sha256 over the library's kernel sources (file names and contents)."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(HERE, "paper_2512_22234_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".hpp", ".h")):
            h.update(name.encode())
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(f.read())
    return h.hexdigest()


def counter_record(kernel: str, workload: str):
    """The committed rocprofv3 counter figures of `kernel` (per launch), or None
    when there are none for this workload or the kernel sources changed since
    the counters were taken (the summary records the source hash)."""
    try:
        text = open(COUNTERS_FILE).read()
    except OSError:
        return None
    start = text.find("```json")
    if start < 0:
        return None
    rec = json.loads(text[start + 7:text.index("```", start + 7)])
    if rec.get("source_sha256") != kernel_source_hash() or rec.get("workload") != workload:
        return None
    return rec.get("kernels", {}).get(kernel)


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter summary, or None."""
    k = counter_record(kernel, workload)
    return None if k is None else int(k["hbm_bytes_per_launch"])


def copy_calibration(nbytes: int = 256 << 20, reps: int = 5):
    """A plain device-to-device copy of known size, the reference the HBM
    byte counters are scaled by (run under rocprofv3 --pmc)."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"[copy] {reps} copies of {nbytes} bytes (each reads {nbytes} and writes {nbytes} bytes)")


def cpu_baseline(w, budget_s: float, max_groups: int):
    import numpy as np
    import oracle
    from paper_2512_22234_amd.workloads import make_inputs
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
                      or [1])
        blas = ",".join(sorted({i.get("internal_api", "?") for i in threadpool_info()
                                if i.get("user_api") == "blas"}))
    except Exception:  # pragma: no cover
        threads, blas = len(os.sched_getaffinity(0)), "unknown"
    q, k, v, do = make_inputs(w)
    G = w.Hq // w.Hkv
    groups = [(b, g) for b in range(w.B) for g in range(w.Hkv)]
    done, t_fwd, t_bwd = 0, 0.0, 0.0
    for b, g in groups[:max_groups]:
        sl = slice(g * G, (g + 1) * G)
        Q = q[b:b + 1, sl].double().numpy()
        K = k[b:b + 1, g:g + 1].double().numpy()
        V = v[b:b + 1, g:g + 1].double().numpy()
        dO = do[b:b + 1, sl].double().numpy()
        t0 = time.perf_counter()
        oracle.forward(Q, K, V, w.L, w.S)
        t1 = time.perf_counter()
        oracle.backward(dO, Q, K, V, w.L, w.S)
        t2 = time.perf_counter()
        t_fwd += t1 - t0
        t_bwd += t2 - t1
        done += 1
        log(f"[cpu] oracle group {done}: fwd {t_fwd:.1f}s bwd {t_bwd:.1f}s cumulative")
        if t_fwd + t_bwd >= budget_s:
            break
    t_total = t_fwd + t_bwd
    npairs = visible_pairs(w.L, w.S) * G * done
    flops = 14 * w.D * npairs
    # the oracle materialises the mask and multiplies dense 2L x 2L matrices:
    # forward Z = Q K^T and O = P V, backward dP, dQ, dK and dV, per query head
    N = 2 * w.L
    dense_fwd, dense_bwd = 4 * N * N * w.D * G * done, 8 * N * N * w.D * G * done
    n_groups = w.B * w.Hkv
    return {"value": round(flops / t_total / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{done} of {n_groups} GQA groups ({G} query heads + 1 KV head each) of the {w.name} "
                      f"workload, fwd+bwd in fp64 numpy ({blas} BLAS), {t_total:.1f} s; value counts the same "
                      f"visible-pair FLOPs as the GPU line; the full workload is extrapolated from this sample",
            "fwd_s": round(t_fwd, 3), "bwd_s": round(t_bwd, 3),
            "groups_timed": done, "groups_total": n_groups,
            "full_workload_s_extrapolated": round(t_total * n_groups / done, 2),
            "effective_gflop_sample": round(flops / 1e9, 3),
            "dense_fp64_gflop_executed": {"fwd": round(dense_fwd / 1e9, 3), "bwd": round(dense_bwd / 1e9, 3)},
            "dense_fp64_gflops_rate": round((dense_fwd + dense_bwd) / t_total / 1e9, 2)}


def packed_step(steps: int, warmup: int, settle_ms: float, name: str = "8b_packed"):
    """fwd+bwd over packed sequences (varlen calls): effective TFLOP/s with the
    same visible-pair FLOP count as the headline, summed over the sequences.
    It runs after the other measurements, so it has its own clock-settle phase."""
    import torch
    import paper_2512_22234_amd as bd
    from paper_2512_22234_amd.workloads import VARLEN_WORKLOADS, make_varlen_inputs, varlen_lengths
    c = VARLEN_WORKLOADS[name]
    lengths = varlen_lengths(c["total"], c["seed"], c["lo"], c["hi"])
    dev = torch.device("cuda:0")
    q, k, v, do, cu = (t.to(dev) for t in make_varlen_inputs(lengths, c["Hq"], c["Hkv"], c["D"], c["seed"]))
    max_L, S, T = max(lengths), c["S"], sum(lengths)
    code = bd.BD_ATTN_BF16
    o, lse = torch.empty_like(q), torch.empty((c["Hq"], 2 * T), dtype=torch.float32, device=dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    wsb = torch.empty(bd.bd_attn_varlen_workspace_bytes(len(lengths), T, max_L, S, c["Hq"], c["Hkv"], c["D"],
                                                        code, 1), dtype=torch.uint8, device=dev)

    def step():
        bd.bd_attn_varlen_fwd(q, k, v, cu, max_L, S, out=o, lse=lse)
        bd.bd_attn_varlen_bwd(do, q, k, v, o, lse, cu, max_L, S, dq=dq, dk=dk, dv=dv, workspace=wsb)

    t_settle = time.perf_counter()
    while (time.perf_counter() - t_settle) * 1e3 < settle_ms:
        for _ in range(10):
            step()
        torch.cuda.synchronize()
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    npairs = sum(visible_pairs(Li, S) for Li in lengths) * c["Hq"]
    tflops = 14 * c["D"] * npairs / (ms * 1e-3) / 1e12
    log(f"[bench] packed {name}: {len(lengths)} sequences {lengths}, {ms:.4f} ms/step, {tflops:.1f} TFLOP/s eff")
    return {"workload": f"{name}: {len(lengths)} packed sequences of {lengths} tokens per copy "
                        f"(T={T}), Hq={c['Hq']} Hkv={c['Hkv']} D={c['D']} S={S}, bf16, fwd+bwd",
            "ms_per_step": round(ms, 5), "tflops_eff": round(tflops, 2),
            "pct_of_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 3), "settle_ms": settle_ms}


PEAK_HBM_GBS = 8000.0        # MI355X HBM3E


def decode_step(steps: int, warmup: int, name: str = "8b_decode"):
    """bd_attn_decode_fwd over a rollout batch: algorithmic HBM GB/s."""
    import torch
    import paper_2512_22234_amd as bd
    from paper_2512_22234_amd.workloads import DECODE_WORKLOADS, decode_cache_lens, make_decode_inputs
    c = DECODE_WORKLOADS[name]
    lens = decode_cache_lens(c["B"], c["seed"], c["lo"], c["hi"])
    B, Hq, Hkv, D, S, C = c["B"], c["Hq"], c["Hkv"], c["D"], c["S"], c["capacity"]
    q, kc, vc, kn, vn, cl = make_decode_inputs(B, Hq, Hkv, D, S, C, lens, seed=c["seed"], device="cuda")
    o, lse = torch.empty_like(q), torch.empty((B, Hq, S), dtype=torch.float32, device=q.device)
    ws = torch.empty(bd.bd_attn_decode_workspace_bytes(B, S, Hq, Hkv, D, C), dtype=torch.uint8, device=q.device)

    def call():
        bd.bd_attn_decode_fwd(q, kc, vc, kn, vn, cl, out=o, lse=lse, workspace=ws)

    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        call()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    nbytes = (sum(lens) * Hkv * D * 2 * 2          # cached K and V rows, bf16
              + B * Hkv * S * D * 2 * 2            # the block's K and V
              + 2 * B * Hq * S * D * 2             # Q in, O out
              + B * Hq * S * 4)                    # LSE out
    gbs = nbytes / (ms * 1e-3) / 1e9
    log(f"[bench] decode {name}: cache lengths {min(lens)}..{max(lens)} (mean {sum(lens) / B:.0f}), "
        f"{ms * 1e3:.1f} us/call, {nbytes / 1e6:.1f} MB, {gbs:.0f} GB/s")
    return {"workload": f"{name}: B={B} Hq={Hq} Hkv={Hkv} D={D} S={S}, capacity {C}, cache lengths "
                        f"log-uniform {c['lo']}..{c['hi']} (sum {sum(lens)}), bf16",
            "us_per_call": round(ms * 1e3, 2), "algorithmic_bytes": nbytes, "gbs": round(gbs, 1),
            "bound": "hbm", "peak_gbs": PEAK_HBM_GBS, "frac": round(gbs / PEAK_HBM_GBS, 4),
            "traffic": measured_traffic("decode", "8b"), "traffic_unit": "HBM bytes per launch of the decode kernel"}


def lce_step(steps: int, warmup: int, name: str = "8b_lm_head"):
    """bd_lce_fwd + bd_lce_objective + bd_lce_bwd over the 8B LM head."""
    import torch
    import paper_2512_22234_amd as bd
    from paper_2512_22234_amd.workloads import LCE_WORKLOADS, make_lce_inputs
    c = LCE_WORKLOADS[name]
    N, V, Dm = c["N"], c["V"], c["Dm"]
    h, w, t = make_lce_inputs(N, V, Dm, seed=c["seed"], device="cuda")
    dev = h.device
    lse, logp = torch.empty(N, device=dev), torch.empty(N, device=dev)
    adv = torch.randn(N, device=dev, generator=torch.Generator(device=dev).manual_seed(1))
    wgt = torch.full((N,), 1.0 / N, device=dev)
    loss, dlogp = torch.empty(N, device=dev), torch.empty(N, device=dev)
    dh, dw = torch.empty_like(h), torch.empty_like(w)
    wsf = torch.empty(bd.bd_lce_workspace_bytes(N, V, Dm, 0), dtype=torch.uint8, device=dev)
    wsb = torch.empty(bd.bd_lce_workspace_bytes(N, V, Dm, 1), dtype=torch.uint8, device=dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    keep = None

    def step(timed=False):
        if timed:
            ev[0].record()
        bd.bd_lce_fwd(h, w, t, lse=lse, logp=logp, workspace=wsf, logits=keep)
        if timed:
            ev[1].record()
        # Eq. 7: online update, the behaviour policy is the detached current one
        bd.bd_lce_objective(logp, wgt, bd.BD_LCE_DIPO, logp_old=logp, adv=adv, eps=0.2, beta=0.0, loss=loss,
                            dlogp=dlogp)
        if timed:
            ev[2].record()
        bd.bd_lce_bwd(h, w, t, lse, dlogp, dh=dh, dw=dw, workspace=wsb, logits=keep)
        if timed:
            ev[3].record()

    def measure():
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        tf = to = tb = 0.0
        for _ in range(steps):
            step(True)
            torch.cuda.synchronize()
            tf += ev[0].elapsed_time(ev[1])
            to += ev[1].elapsed_time(ev[2])
            tb += ev[2].elapsed_time(ev[3])
        return tf / steps, to / steps, tb / steps

    tf, to, tb = measure()
    # the same step keeping the forward's logits (float32 [N][V rounded up]) for the backward
    keep = torch.empty(bd.bd_lce_logits_bytes(N, V, Dm) // 4, dtype=torch.float32, device=dev)
    kf, ko, kb = measure()
    keep = None
    gemm = 2.0 * N * V * Dm
    fwd_tf = gemm / (tf * 1e-3) / 1e12
    bwd_tf = 3 * gemm / (tb * 1e-3) / 1e12   # executed: recomputed logits, dH, dW
    step_tf = 3 * gemm / ((tf + to + tb) * 1e-3) / 1e12  # useful: logits, dH, dW
    log(f"[bench] lce {name}: fwd {tf:.3f} ms ({fwd_tf:.0f} TFLOP/s), objective {to * 1e3:.1f} us, "
        f"bwd {tb:.3f} ms ({bwd_tf:.0f} TFLOP/s executed); keeping the logits: fwd {kf:.3f} ms, bwd {kb:.3f} ms, "
        f"step {kf + ko + kb:.3f} ms ({3 * gemm / ((kf + ko + kb) * 1e-3) / 1e12:.0f} TFLOP/s)")
    return {"workload": f"{name}: N={N} scored positions, V={V}, Dm={Dm}, bf16 H ~ N(0,1), W ~ N(0, 9/Dm), "
                        f"DiPO objective with online ratio",
            "fwd_ms": round(tf, 4), "objective_ms": round(to, 4), "bwd_ms": round(tb, 4),
            "step_ms": round(tf + to + tb, 4),
            "tflops_useful": round(step_tf, 1), "fwd_tflops": round(fwd_tf, 1), "bwd_tflops_executed": round(bwd_tf, 1),
            "bound": "mfma", "peak_tflops": PEAK_BF16_TFLOPS, "frac_fwd": round(fwd_tf / PEAK_BF16_TFLOPS, 4),
            "frac_bwd_executed": round(bwd_tf / PEAK_BF16_TFLOPS, 4),
            "kept_logits": {"fwd_ms": round(kf, 4), "bwd_ms": round(kb, 4), "step_ms": round(kf + ko + kb, 4),
                            "tflops_useful": round(3 * gemm / ((kf + ko + kb) * 1e-3) / 1e12, 1),
                            "logits_bytes": bd.bd_lce_logits_bytes(N, V, Dm)}}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--settle-ms", type=float, default=250.0,
                    help="wall time of untimed steps before the warm-up, for the clocks to settle (0: none)")
    ap.add_argument("--workload", default="8b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-packed", action="store_true", help="skip the packed-sequence measurement")
    ap.add_argument("--no-decode", action="store_true", help="skip the KV-cache decode measurement")
    ap.add_argument("--no-lce", action="store_true", help="skip the LM-head log-probability measurement")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle time to spend")
    ap.add_argument("--cpu-max-groups", type=int, default=4)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the plain 256 MiB copy used to scale the HBM byte counters")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus} GPUs, WORLD_SIZE={world}); "
              "the block-diffusion attention path here has no multi-GPU mode.", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration()
        return

    import torch
    import paper_2512_22234_amd as bd
    from paper_2512_22234_amd.workloads import WORKLOADS, make_inputs

    w = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    q, k, v, do = (t.to(dev) for t in make_inputs(w))
    L, S = w.L, w.S
    o = torch.empty_like(q)
    lse = torch.empty((w.B, w.Hq, 2 * L), dtype=torch.float32, device=dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    code = bd.BD_ATTN_BF16
    wsf = torch.empty(bd.bd_attn_workspace_bytes(w.B, L, S, w.Hq, w.Hkv, w.D, code, 0), dtype=torch.uint8,
                      device=dev)
    wsb = torch.empty(bd.bd_attn_workspace_bytes(w.B, L, S, w.Hq, w.Hkv, w.D, code, 1), dtype=torch.uint8,
                      device=dev)
    fwd_names = bd.bd_attn_stage_names(False, code)
    bwd_names = bd.bd_attn_stage_names(True, code)
    nf, nb = 2 * len(fwd_names), 2 * len(bwd_names)  # each kernel's start and end, from its dispatch
    K = args.steps
    # Every MARK_EVERY-th timed step carries the dispatch events the per-kernel
    # durations come from; the others run the same calls unmarked (the events
    # cost ~15 us per marked 8B step, which the step time then includes).
    marked = [i for i in range(K) if i % MARK_EVERY == 0]
    fwd_marks = [[torch.cuda.Event(enable_timing=True) for _ in range(nf)] for _ in marked]
    bwd_marks = [[torch.cuda.Event(enable_timing=True) for _ in range(nb)] for _ in marked]
    for evs in fwd_marks + bwd_marks:   # create the events before the timed region
        for e in evs:
            e.record()
    torch.cuda.synchronize()

    def step(i=None):
        if i is None or i % MARK_EVERY:
            bd.bd_attn_fwd(q, k, v, L, S, out=o, lse=lse, workspace=wsf)
            bd.bd_attn_bwd(do, q, k, v, o, lse, L, S, dq=dq, dk=dk, dv=dv, workspace=wsb)
        else:
            u = i // MARK_EVERY
            bd.bd_attn_fwd_marked(q, k, v, L, S, fwd_marks[u], out=o, lse=lse, workspace=wsf)
            bd.bd_attn_bwd_marked(do, q, k, v, o, lse, L, S, bwd_marks[u], dq=dq, dk=dk, dv=dv, workspace=wsb)

    # Clock settle: the GPU's clocks settle only after tens of milliseconds of
    # sustained load, so before the W warm-up steps the step runs for a fixed
    # wall time (reported as its own field; 0 disables it).
    settle_steps, t_settle = 0, time.perf_counter()
    while args.settle_ms > 0 and (time.perf_counter() - t_settle) * 1e3 < args.settle_ms:
        for _ in range(10):
            step()
        settle_steps += 10
        torch.cuda.synchronize()
    settle_ms = (time.perf_counter() - t_settle) * 1e3 if settle_steps else 0.0
    log(f"[bench] {w.describe()}: clock settle {settle_ms:.0f} ms ({settle_steps} steps), warmup {args.warmup}, "
        f"timed {K} steps")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for i in range(K):
        step(i)
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end) / K
    log(f"[bench] timed region: {ms:.4f} ms/step (events), {wall * 1e3 / K:.4f} ms/step (host clock)")

    # per-kernel durations from the marks (mean over the marked timed steps),
    # and the per-step fwd / bwd durations, first kernel's start to last
    # kernel's end (median over the marked timed steps)
    per = {}
    for names, marks in ((fwd_names, fwd_marks), (bwd_names, bwd_marks)):
        for j, name in enumerate(names):
            per[name] = sum(m[2 * j].elapsed_time(m[2 * j + 1]) for m in marks) / len(marks)
    t_fwd = sum(per[n] for n in fwd_names)
    t_bwd = sum(per[n] for n in bwd_names)
    step_ms = sorted(f[0].elapsed_time(f[-1]) + b[0].elapsed_time(b[-1]) for f, b in zip(fwd_marks, bwd_marks))
    med_step = step_ms[len(step_ms) // 2]

    npairs = visible_pairs(L, S) * w.B * w.Hq
    f_fwd, f_bwd, f_bwd8 = 4 * w.D * npairs, 10 * w.D * npairs, 8 * w.D * npairs
    tflops = (f_fwd + f_bwd) / (ms * 1e-3) / 1e12
    # algorithmic FLOPs of each kernel (useful work only; recomputation not counted)
    alg = {"fwd": 4 * w.D * npairs, "bwd_dkdv": 8 * w.D * npairs, "bwd_dq": 2 * w.D * npairs}
    alg = {n: f for n, f in alg.items() if n in per}
    kernels = {}
    for name, t in per.items():
        entry = {"ms": round(t, 5)}
        if name in alg:
            entry["tflops"] = round(alg[name] / (t * 1e-3) / 1e12, 2)
            entry["frac_of_peak"] = round(entry["tflops"] / PEAK_BF16_TFLOPS, 4)
        # counter-derived figures (committed rocprofv3 record of these sources), over this run's timing
        rec = counter_record(name, w.name)
        if rec is not None:
            entry["executed_mfma_tflops"] = round(rec["sq_insts_mfma"] * 32768 / (t * 1e-3) / 1e12, 1)
            entry["mfma_busy_frac"] = rec["mfma_busy_frac"]
            entry["lds_busy_frac"] = rec["lds_busy_frac"]
            entry["hbm_bytes"] = rec["hbm_bytes_per_launch"]
            entry["hbm_gbs"] = round(rec["hbm_bytes_per_launch"] / (t * 1e-3) / 1e9, 1)
        kernels[name] = entry
    dom = max(alg, key=lambda n: per[n])
    ach = alg[dom] / (per[dom] * 1e-3) / 1e12
    log(f"[bench] kernels: {json.dumps(kernels)}")
    log(f"[bench] fwd {t_fwd:.4f} ms ({f_fwd / t_fwd / 1e9:.1f} TFLOP/s eff), bwd {t_bwd:.4f} ms "
        f"({f_bwd / t_bwd / 1e9:.1f} TFLOP/s eff at 10D, {f_bwd8 / t_bwd / 1e9:.1f} at 8D)")

    packed = None if args.no_packed else packed_step(args.steps, args.warmup, args.settle_ms)
    decode = None if args.no_decode else decode_step(args.steps, args.warmup)
    lce = None if args.no_lce else lce_step(min(args.steps, 10), min(args.warmup, 3))

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args.cpu_budget, args.cpu_max_groups)

    out = {
        "metric": METRIC,
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "pct_of_bf16_peak": round(100 * tflops / PEAK_BF16_TFLOPS, 3),
        "settle_ms": round(settle_ms, 1), "settle_steps": settle_steps,
        "config": {"workload": f"{w.name}: B={w.B} Hq={w.Hq} Hkv={w.Hkv} D={w.D} L={L} (packed {2 * L}) "
                               f"S={S}, bf16 N(0,1)*0.5, fwd+bwd",
                   "global_batch": w.B, "seq_len": 2 * L, "parallelism": "single GPU",
                   "visible_pairs_per_head": visible_pairs(L, S),
                   "flops_per_step": f_fwd + f_bwd, "fwd_ms": round(t_fwd, 5), "bwd_ms": round(t_bwd, 5),
                   "median_step_ms": round(med_step, 5),
                   "fwd_tflops_eff": round(f_fwd / t_fwd / 1e9, 2), "bwd_tflops_eff": round(f_bwd / t_bwd / 1e9, 2)},
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(ach / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(dom, w.name), "traffic_unit": "HBM bytes per launch",
                     "algorithmic_flops_per_launch": alg[dom]},
        "kernels": kernels,
        "packed": packed,
        "decode": decode,
        "lce": lce,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
