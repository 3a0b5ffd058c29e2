#!/usr/bin/env python3
"""Per-step mask + apply benchmark on one MI355X.

A step is one pass of the whole hot path over one batch: psc_compute_masks
(classifier walk + mask-row gather) followed by psc_apply_mask (in-place
-inf on the logits), both on one stream, inputs already resident in HBM.
Prints ONE JSON line (see the field list at the bottom).
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

METRIC = "per-step mask+apply latency (µs) at B=64,V=151,936; masks/s; achieved HBM GB/s"
HBM_PEAK_GBS = 8000.0
MALL_BYTES = 256 << 20


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="schema")
    ap.add_argument("--distinct-steps", type=int, default=None,
                    help="distinct prefix batches generated (default: the workload's step count)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--warm-cache", action="store_true", help="single logits buffer (cache-resident; labelled)")
    ap.add_argument("--calibration-copy-mb", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration under rocprofv3 --pmc)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build measures one GPU only; --gpus must be 1 "
                                   "(the mask path shards by batch or vocabulary with no exchange)"}))
        sys.exit(2)

    import numpy as np
    import torch

    from inputs import configs
    from paper_2608_03065_amd.psc import Classifier, apply_mask, pack_states

    dev = torch.device("cuda:0")
    wl = configs.get(args.workload)
    B, V = wl.B, wl.V
    W = (V + 31) // 32
    s_logit = 2 if wl.logits_dtype == "bf16" else 4
    log(f"workload {wl.name}: B={B} V={V} dtype={wl.logits_dtype}")

    t0 = time.time()
    clf = Classifier(wl.grammar, wl.vocab)
    info = clf.info()
    log(f"psc_build {info['build_seconds']:.2f}s states={info['dfa_states']} classes={info['n_classes']}"
        f" (total setup {time.time() - t0:.1f}s)")
    stream = torch.cuda.Stream(device=dev)     # default priority
    clf.bind(dev, stream=stream)

    n_distinct = args.distinct_steps or wl.steps
    n_distinct = max(1, min(n_distinct, wl.steps))
    t0 = time.time()
    step_inputs, step_states = [], []
    depth_hist = []
    for s in range(n_distinct):
        st = wl.states(s)
        step_states.append(st)
        depth_hist += [len(x[1]) for x in st]
        step_inputs.append(pack_states(st, dev))
        if (s + 1) % 200 == 0:
            log(f"inputs {s + 1}/{n_distinct} ({time.time() - t0:.1f}s)")
    torch.cuda.synchronize()
    log(f"generated {n_distinct} distinct steps in {time.time() - t0:.1f}s; "
        f"stack depth mean {np.mean(depth_hist):.1f} max {max(depth_hist)}")

    # logits pool larger than 2x the 256 MiB Infinity Cache, unless --warm-cache
    per_buf = B * V * s_logit
    n_pool = 1 if args.warm_cache else max(2, math.ceil(2.2 * MALL_BYTES / per_buf))
    tdt = torch.bfloat16 if wl.logits_dtype == "bf16" else torch.float32
    gen = torch.Generator(device=dev).manual_seed(0x50534300 + wl.index)
    pool = [(torch.randn(B, V, generator=gen, device=dev) * wl.logits_std).to(tdt) for _ in range(n_pool)]
    n_bm = 4
    bms = [torch.empty((B, W), dtype=torch.int32, device=dev) for _ in range(n_bm)]
    log(f"logits pool {n_pool} x {per_buf / 1e6:.1f} MB")

    if args.calibration_copy_mb:
        # a plain copy of known size: its FETCH_SIZE / WRITE_SIZE readings
        # give the counters' bytes-per-KiB scale on this GPU
        n = args.calibration_copy_mb << 20
        src_t = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst_t = torch.empty(n, dtype=torch.uint8, device=dev)
        for _ in range(3):
            dst_t.copy_(src_t)
        torch.cuda.synchronize()
        del src_t, dst_t
        log(f"calibration copy: 3 x {args.calibration_copy_mb} MiB device-to-device")

    def step(i):
        stacks, lens, qs = step_inputs[i % n_distinct]
        bm = bms[i % n_bm]
        clf.compute_masks(stacks, lens, qs, out=bm, stream=stream)
        apply_mask(pool[i % n_pool], bm, stream=stream)

    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()

        # (1) clean timed loop: whole-step latency
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for i in range(args.steps):
            step(i)
        end.record(stream)
        torch.cuda.synchronize()
        total_ms = start.elapsed_time(end)
        ms_per_step = total_ms / args.steps

        # (2) per-kernel durations with events around each launch
        K = min(args.steps, 1000)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(K)]
        torch.cuda.synchronize()
        for i in range(K):
            stacks, lens, qs = step_inputs[i % n_distinct]
            bm = bms[i % n_bm]
            ev[i][0].record(stream)
            clf.compute_masks(stacks, lens, qs, out=bm, stream=stream)
            ev[i][1].record(stream)
            apply_mask(pool[i % n_pool], bm, stream=stream)
            ev[i][2].record(stream)
        torch.cuda.synchronize()
        t_compute_ev = float(np.mean([e[0].elapsed_time(e[1]) for e in ev])) * 1e3   # us
        t_apply_ev = float(np.mean([e[1].elapsed_time(e[2]) for e in ev])) * 1e3

        # (3) each kernel alone, back to back on the stream: the average launch
        # duration (events over the whole loop, no per-launch markers)
        def solo(fn, n=1000):
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            for i in range(20):
                fn(i)
            torch.cuda.synchronize()
            a.record(stream)
            for i in range(n):
                fn(i)
            z.record(stream)
            torch.cuda.synchronize()
            return a.elapsed_time(z) / n * 1e3

        def only_compute(i):
            stacks, lens, qs = step_inputs[i % n_distinct]
            clf.compute_masks(stacks, lens, qs, out=bms[i % n_bm], stream=stream)

        # masks of the first n_bm steps stay in bms for the apply-only loop
        for i in range(n_bm):
            only_compute(i)

        def only_apply(i):
            apply_mask(pool[i % n_pool], bms[i % n_bm], stream=stream)

        t_apply = solo(only_apply)          # masks of steps 0..n_bm-1, as counted below
        t_compute = solo(only_compute)

    # Algorithmic bytes of the in-place apply, from the actual masks: the
    # bitmask is read once; a 16-byte vector of logits whose entries are all
    # masked is written once (16 B); one that keeps some entries and masks
    # others must be read to be written (32 B); one that keeps all entries is
    # not touched.  (V % 32 == 0 here, so vectors never straddle rows.)
    per_vec = 16 // s_logit
    apply_bytes, stack_total = [], 0
    for s in range(n_distinct):
        stacks, lens, qs = step_inputs[s]
        clf.compute_masks(stacks, lens, qs, out=bms[0], stream=stream)
        torch.cuda.synchronize()
        m = bms[0].cpu().numpy().view(np.uint32)
        if per_vec == 8:
            groups = m.view(np.uint8).reshape(-1)
            full = 0xFF
        else:
            b8 = m.view(np.uint8).reshape(-1)
            groups = np.stack([b8 & 0xF, b8 >> 4], axis=1).reshape(-1)
            full = 0xF
        n_masked = int((groups == 0).sum())
        n_mixed = int(((groups != 0) & (groups != full)).sum())
        apply_bytes.append(4 * W * B + 16 * n_masked + 32 * n_mixed)
        stack_total += int(lens.sum().item())
    stack_words = stack_total / n_distinct
    bytes_compute = 4 * stack_words + 8 * B + 2 * 4 * W * B         # stacks, lens+states, row read + write
    bytes_apply = float(np.mean(apply_bytes))
    bytes_step = bytes_compute + bytes_apply
    one_pass_model = B * (2 * V * s_logit + 3 * 4 * W) + 4 * (stack_words + 2 * B)

    lat_us = ms_per_step * 1e3
    masks_per_s = B / (ms_per_step * 1e-3)
    bytes_apply_solo = float(np.mean(apply_bytes[:n_bm]))
    achieved_apply = bytes_apply_solo / (t_apply * 1e-6) / 1e9
    roofline = {
        "bound": "hbm", "kernel": "apply_fast_kernel" if V % 32 == 0 else "apply_generic_kernel",
        "achieved": round(achieved_apply, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(achieved_apply / HBM_PEAK_GBS, 4),
        "traffic": measured_traffic(wl.name, "apply_fast_kernel") if V % 32 == 0 else None,
        "algorithmic_bytes_per_launch": round(bytes_apply_solo),
        "avg_launch_us": round(t_apply, 3),
        "timing": "HIP events around 1000 back-to-back launches of the kernel alone on the bench stream",
    }

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, step_states, args.cpu_seconds, B)

    out = {
        "metric": METRIC,
        "value": round(masks_per_s, 1),
        "unit": "masks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "latency_us": round(lat_us, 3),
        "hbm_gbs_step": round(bytes_step / (ms_per_step * 1e-3) / 1e9, 1),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {wl.description}",
            "B": B, "V": V, "logits": wl.logits_dtype, "distinct_steps": n_distinct,
            "logits_pool_buffers": n_pool, "warm_cache": bool(args.warm_cache),
        },
        "kernels_us": {"compute_masks_solo": round(t_compute, 3), "apply_mask_solo": round(t_apply, 3),
                       "compute_masks_in_step_events": round(t_compute_ev, 3),
                       "apply_mask_in_step_events": round(t_apply_ev, 3)},
        "bytes_per_step": {"algorithmic": round(bytes_step), "one_pass_read_write_model": round(one_pass_model)},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "build": {k: info[k] for k in ("dfa_states", "n_classes", "table_bytes", "mask_table_bytes",
                                        "build_seconds", "dfa_rows", "dense_rows")},
    }
    print(json.dumps(out), flush=True)


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, or
    None when there is none for this workload or the kernel source changed
    since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"{workload}_c3_pmc_traffic.md" if workload == "schema" else
                        f"{workload}_pmc_traffic.md")
    if not os.path.exists(path):
        return None
    meta = None
    for line in open(path):
        if line.startswith("traffic_json: "):
            meta = json.loads(line[len("traffic_json: "):])
    src = os.path.join(ROOT, "paper_2608_03065_amd", "csrc", "psc_device.hip")
    h = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    if not meta or meta.get("source_sha256_16") != h or kernel not in meta.get("kernels", {}):
        return None
    return meta["kernels"][kernel]["hbm_bytes"]


def cpu_baseline(wl, step_states, seconds, B):
    """The oracle as it stands, on this host's cores, over a bounded sample."""
    import numpy as np

    from oracle import Oracle
    orc = Oracle(wl.grammar, wl.vocab)
    flat = [st for s in step_states for st in s]
    t0 = time.time()
    orc.masks(flat[:1])
    one = time.time() - t0
    n = int(max(1, min(len(flat), seconds / max(one, 1e-4))))
    log(f"cpu baseline: oracle on {n} sequences (~{n * one:.1f}s)")
    t0 = time.time()
    orc.masks(flat[:n])
    dt = time.time() - t0
    return {
        "value": round(n / dt, 3), "unit": "masks/s", "cores": int(orc.threads_used), "kind": "oracle",
        "sample": f"first {n} sequences (of {len(flat)}) of the benchmark's prefix batches, "
                  f"all {wl.V} tokens each; {dt:.1f}s wall",
        "per_step_latency_us": round(dt / n * B * 1e6, 1),
    }


if __name__ == "__main__":
    main()
