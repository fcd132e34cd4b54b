#!/usr/bin/env python3
"""Benchmark of the guarded decode step on one MI355X.

Workload: the 7B-shaped batch (32 sequences, 28 layers, 28 query / 4 KV heads, head_dim 128,
bf16, KV budget 2048, context 8192; half the sequences carry a planted loop), synthetic inputs
from the seeded generator, resident in HBM before timing. One step = every layer's
lg_decode_attend + lg_detect_and_prune (the detector and the keep set in one launch, then the
compaction) for the whole batch.

Prints one JSON line: steps/s (value), KV tokens read/s, algorithmic GB/s (also as a fraction of
peak and of the copy bandwidth measured on the device), the interventions and budget-overflow
compactions of the timed steps, the roofline object of the attention kernels (algorithmic bytes
per launch / average launch time, from HIP events on the launch stream around each step's
back-to-back launches) and the CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

PEAK_HBM_GBPS = 8000.0
POLICIES = {"loopguard": 0, "h2o": 1, "streaming": 2}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=120)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--config", type=int, default=2, help="workload index (2 = 7B-shaped batch 32)")
    ap.add_argument("--form", type=int, default=0,
                    help="attention kernel form of the test hook (0 = what lg_decode_attend runs, "
                         "1 portable, 2 merge launch, 3 one-launch)")
    ap.add_argument("--max-split", type=int, default=0,
                    help="split length of the test hook (0 = default)")
    ap.add_argument("--attend-flags", type=int, default=0,
                    help="flags of the test hook (lg_testing.h)")
    ap.add_argument("--policy", choices=sorted(POLICIES), default="loopguard",
                    help="keep policy of the prune step (the paper's method or a Sec. 6.1 baseline)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--copy-only", action="store_true",
                    help="run only the 1 GiB copy kernel (calibrates the HBM byte counters)")
    ap.add_argument("--prune-event", action="store_true",
                    help="time one lg_prune_compact call with every sequence of the workload at "
                         "its budget (all layers), for each keep policy")
    return ap.parse_args()


TRAFFIC_PROFILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                               "attend_mfma_7b_b32_traffic.md")
ATTEND_SOURCE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2604_10044_amd",
                             "csrc", "lg_attend.hip")


def measured_traffic(workload: str):
    """HBM bytes per lg_decode_attend launch from the committed counter profile, or None when the
    profile was taken on another workload or the attention source has changed since."""
    import hashlib
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    fields = {}
    for line in open(TRAFFIC_PROFILE):
        if ":" in line and line.startswith("- "):
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    src = hashlib.sha256(open(ATTEND_SOURCE, "rb").read()).hexdigest()
    if fields.get("lg_attend.hip sha256") != src or fields.get("workload") != workload:
        return None
    try:
        return float(fields["HBM bytes per lg_decode_attend launch"])
    except (KeyError, ValueError):
        return None


def _value_or_range(a):
    """A per-sequence setting as one number, or [min, max] when the batch is ragged."""
    a = np.asarray(a)
    return int(a[0]) if np.all(a == a[0]) else [int(a.min()), int(a.max())]


def attend_bytes(lens_live, Hkv, Hq, D, e, B):
    """Algorithmic bytes of one lg_decode_attend launch: K and V rows of every live slot, the
    acc read-modify-write, q in, out/lse/suffix mass out."""
    slots = float(np.sum(lens_live))
    return slots * (2 * Hkv * D * e + 8 * Hkv) + B * Hq * (2 * D * e + 8)


def cpu_baseline(wl, budget_s, policy):
    """The oracle as it stands, single-threaded, on one sequence of the workload: as many whole
    steps (all layers, detector, prune) as fit in ~budget_s seconds."""
    import oracle
    from oracle.trajectory import SequenceOracle
    so = SequenceOracle(wl, 0, params=oracle.paper_params(policy=policy), threads=1)
    t0 = time.perf_counter()
    k = 0
    while k < wl.steps:
        so.step(k)
        k += 1
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    per_seq_step = dt / k
    return {"value": 1.0 / (per_seq_step * wl.batch), "unit": "steps/s", "cores": 1,
            "nproc": len(os.sched_getaffinity(0)), "kind": "oracle",
            "layer_step_ms": per_seq_step / wl.n_layers * 1e3,
            "sequence_step_ms": per_seq_step * 1e3,
            "sample": "sequence 0 of the batch, %d whole guarded steps (all %d layers, detector, "
                      "keep set) in %.1f s, one thread of the host's %d; batch rate extrapolated "
                      "as the per-sequence rate / %d (sequences are independent); "
                      "layer_step_ms = one sequence's time per step / %d layers"
                      % (k, wl.n_layers, dt, len(os.sched_getaffinity(0)), wl.batch, wl.n_layers)}


def prune_event(args):
    """Median time of a prune event that hits every sequence at once: live slots = budget - 1 at
    even positions, plus the step's append; the cache contents are random (compaction moves rows
    regardless of their values)."""
    import torch
    from paper_2604_10044_amd import lg
    from paper_2604_10044_amd import synth
    wl = synth.config(args.config, steps=1)
    B, L, Hq, Hkv, D, cap = wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.cap
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    K = [torch.randn(B, Hkv, cap, D, device="cuda").to(dt) for _ in range(L)]
    V = [torch.randn(B, Hkv, cap, D, device="cuda").to(dt) for _ in range(L)]
    A = [torch.rand(B, Hkv, cap, device="cuda") for _ in range(L)]
    layers = [lg.layer_cache(K[l], V[l], A[l], Hq) for l in range(L)]
    budget = torch.as_tensor(np.asarray(wl.budget, np.int32), device="cuda")
    pos0 = (torch.arange(cap, dtype=torch.int32, device="cuda") * 2).repeat(B, 1).contiguous()
    len0 = (budget - 1).to(torch.int32)
    tap = torch.full((B,), 2 * cap + 5, dtype=torch.int32, device="cuda")
    pos, ln = pos0.clone(), len0.clone()
    kidx = torch.zeros(B, cap, dtype=torch.int32, device="cuda")
    nlen = torch.zeros(B, dtype=torch.int32, device="cuda")
    res = {}
    for name, code in sorted(POLICIES.items(), key=lambda x: x[1]):
        p = lg.lg_guard_params_default()
        p.policy = code
        ts = []
        for it in range(args.warmup + args.steps):
            pos.copy_(pos0)
            ln.copy_(len0)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            lg.lg_prune_compact(p, B, cap, layers, pos, ln, budget, tap, None, kidx, nlen)
            e1.record()
            torch.cuda.synchronize()
            if it >= args.warmup:
                ts.append(e0.elapsed_time(e1) * 1e3)
        res[name] = {"us_median": float(np.median(ts)), "kept_slots_seq0": int(nlen[0])}
    print(json.dumps({"prune_event": res, "workload": wl.name, "batch": B, "layers": L,
                      "events_timed": args.steps}))


FORM_NAMES = {1: "attend_valu + attend_combine (portable pair)",
              2: "attend_mfma sweep + attend_combine_mfma (merge form)",
              3: "attend_mfma (one-launch form)"}


def attend_kernel_name(header: dict) -> str:
    """The attention launch that ran, from the form the workspace was initialised for."""
    return "lg_decode_attend: %s, splits of <= %d slots" % (
        FORM_NAMES.get(header["form"], "form %d" % header["form"]), header["split"])


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this path has no multi-GPU mode (sequences shard "
              "across GPUs with no exchange; see the design notes)", file=sys.stderr)
        sys.exit(2)
    if args.prune_event:
        prune_event(args)
        return
    import torch
    from paper_2604_10044_amd import lg
    from paper_2604_10044_amd import synth
    from paper_2604_10044_amd.decoder import GuardedDecoder
    if args.copy_only:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(4):
            lg.lg_copy_bandwidth(src, dst, 1 << 30)
        torch.cuda.synchronize()
        print(json.dumps({"copy_only": True, "bytes_per_launch_each_way": 1 << 30, "launches": 4}))
        return

    total = args.warmup + args.steps
    wl = synth.config(args.config, steps=total)
    policy = POLICIES[args.policy]
    dec = GuardedDecoder(wl, params={"policy": policy}, form=args.form, max_split=args.max_split,
                         attend_flags=args.attend_flags)
    dec.prefill()
    dec.load_steps(total)
    B, L, Hq, Hkv, D = wl.batch, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim
    e = wl.elem_bytes
    stream = torch.cuda.current_stream()

    for s in range(args.warmup):
        dec.step(s)
    torch.cuda.synchronize()

    # copy ceiling on this device (same memory system, 1 GiB each way)
    nbytes = 1 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        lg.lg_copy_bandwidth(src, dst, nbytes)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(10):
        lg.lg_copy_bandwidth(src, dst, nbytes)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_gbps = 2 * nbytes * 10 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del src, dst

    # Snapshot the state after warmup: the timed graph pass and the per-launch timing pass both
    # start from it.
    snap = dec.snapshot()

    # Pass 1 (throughput): one HIP graph per step (every layer's attention, detector, prune),
    # captured up front and replayed back to back.
    graphs = []
    cap_stream = torch.cuda.Stream()
    for i in range(args.steps):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap_stream):
            dec.step(args.warmup + i)
        graphs.append(g)
    torch.cuda.synchronize()
    # One untimed replay of every graph (a graph's first launch carries one-time set-up), undone
    # by restoring the snapshot, so the timed replays hold only the steps' own work.
    dec.restore(snap)
    for g in graphs:
        g.replay()
    torch.cuda.synchronize()
    dec.restore(snap)
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for g in graphs:
        g.replay()
    end.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    ms_per_step = total_ms / args.steps
    n_int_col = lg.STATE_FIELDS.index("n_int")
    n_int = int(dec.state[:, n_int_col].sum().item() - snap["state"][:, n_int_col].sum().item())
    del graphs

    # Pass 2 (launch timing of the attention kernels): the same steps again from the snapshot,
    # launched eagerly, with HIP events on the launch stream around each step's L back-to-back
    # lg_decode_attend calls (every layer of a step sees the same live lengths, hence the same
    # bytes); the average launch is that interval / L. Events around every single call would add
    # a marker between launches that the graph replay does not have. Each step starts behind
    # three 1 GiB copies (~1.3 ms of GPU time, several times what the host needs to enqueue a
    # step's launches through the binding) so its launches are all queued before the GPU reaches
    # them.
    dec.restore(snap)
    pad_src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    pad_dst = torch.empty_like(pad_src)
    len_hist = torch.zeros(args.steps + 1, B, dtype=torch.int32, device="cuda")
    trig_hist = torch.zeros(args.steps, B, dtype=torch.int32, device="cuda")
    trig_col = lg.DECISION_FIELDS.index("trigger")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        s = args.warmup + i
        for _ in range(3):
            lg.lg_copy_bandwidth(pad_src, pad_dst, 1 << 30)
        len_hist[i].copy_(dec.len, non_blocking=True)
        a, b = ev[i]
        a.record(stream)
        for l in range(L):
            dec.attend_layer(s, l)
        b.record(stream)
        dec.detect_prune(s)
        trig_hist[i].copy_(dec.decision[:, trig_col], non_blocking=True)
    len_hist[args.steps].copy_(dec.len)
    torch.cuda.synchronize()
    del pad_src, pad_dst
    lh = len_hist.cpu().numpy().astype(np.int64)
    # A compaction at step i leaves fewer live slots than the step's append gave; the ones without
    # a trigger are budget overflows.
    compacted = lh[1:] < lh[:-1] + 1
    n_overflow = int((compacted & (trig_hist.cpu().numpy() == 0)).sum())
    lens = lh[:-1] + 1                                             # live slots incl. the append
    att_ms = np.array([ev[i][0].elapsed_time(ev[i][1]) / L for i in range(args.steps)])
    bytes_per_launch = np.array([attend_bytes(lens[i], Hkv, Hq, D, e, B) for i in range(args.steps)])
    achieved_gbps = float(bytes_per_launch.sum() / (att_ms.sum() * 1e-3) / 1e9)
    step_bytes = float(bytes_per_launch.sum() * L)
    kv_tokens = float(lens.sum() * L)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(synth.config(args.config, steps=total), args.cpu_seconds, policy)

    res = {
        "metric": "guarded decode steps/sec (KV tokens read/s) and % of MI355X peak HBM GB/s",
        "value": 1000.0 / ms_per_step,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded generator; no datasets or checkpoints)",
        "config": {"workload": wl.name, "batch": B, "layers": L, "q_heads": Hq, "kv_heads": Hkv,
                   "head_dim": D, "budget": _value_or_range(wl.budget),
                   "context": _value_or_range(wl.ctx),
                   "decode_steps": total, "keep_policy": args.policy,
                   "parallelism": "none (1 GPU)"},
        "kv_tokens_per_s": kv_tokens / (total_ms * 1e-3),
        "step_gbps": step_bytes / (total_ms * 1e-3) / 1e9,
        "step_hbm_frac": step_bytes / (total_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS,
        "copy_gbps": copy_gbps,
        "step_frac_of_copy": step_bytes / (total_ms * 1e-3) / 1e9 / copy_gbps,
        "interventions": n_int,
        "overflow_compactions": n_overflow,
        "roofline": {"bound": "hbm", "achieved": achieved_gbps, "peak": PEAK_HBM_GBPS,
                     "unit": "GB/s", "frac": achieved_gbps / PEAK_HBM_GBPS,
                     "traffic": measured_traffic(wl.name),
                     "kernel": attend_kernel_name(lg.workspace_header(dec.workspace)),
                     "avg_launch_us": float(att_ms.mean() * 1e3),
                     "bytes_per_launch": float(bytes_per_launch.mean())},
        "cpu_baseline": cpu,
    }
    print(json.dumps(res))


if __name__ == "__main__":
    main()
