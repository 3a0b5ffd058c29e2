#!/usr/bin/env python3
"""Per-step mask + apply benchmark on one MI355X.

A step is one pass of the whole hot path over one batch, inputs already
resident in HBM: the classifier walk, the gather of each class's mask row
into the bitmask, and the in-place -inf on the logits.  By default it is one
psc_compute_and_apply launch; --mode two-launch times psc_compute_masks
followed by psc_apply_mask on the same stream instead.
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
    ap.add_argument("--mode", choices=["fused", "two-launch"], default="fused",
                    help="fused: psc_compute_and_apply (one launch); two-launch: psc_compute_masks + "
                         "psc_apply_mask")
    ap.add_argument("--distinct-steps", type=int, default=None,
                    help="distinct prefix batches generated (default: the workload's step count)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--warm-cache", action="store_true", help="single logits buffer (cache-resident; labelled)")
    ap.add_argument("--decode-steps", type=int, default=256,
                    help="tokens per sequence in the on-device decoding loop (advance + masks)")
    ap.add_argument("--calibration-copy-mb", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration under rocprofv3 --pmc)")
    ap.add_argument("--masks", choices=["flat", "sliced"], default="flat",
                    help="layout of the mask table on the device (psc_bind_device_ex)")
    ap.add_argument("--predictor-batches", type=int, default=200,
                    help="held-out prefix batches walked once before the warmup to fill the class predictor "
                         "(0: start empty)")
    ap.add_argument("--timeline", type=int, default=0,
                    help="also run this many steps of the timeline variant and report per-workgroup times")
    ap.add_argument("--speculate", action="store_true",
                    help="PSC_OPT_SPECULATE: the fused step loads the predicted class's data during the walk")
    ap.add_argument("--no-prequeue", action="store_true",
                    help="time loops without first queueing them behind a device-side delay")
    ap.add_argument("--latency-probe", action="store_true",
                    help="instead of the step: ns per dependent load (the walk's load kinds) against the table's "
                         "size, in this workload's launch shape (libpsc_probe.so); prints one JSON line")
    ap.add_argument("--batch", type=int, default=None,
                    help="sequences per step instead of the workload's own B (a sweep over batch sizes; the "
                         "prefixes of sequences past B are drawn the same way; labelled in config)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1 "
                                   "(the mask path shards by batch or vocabulary with no exchange)"}))
        sys.exit(2)

    import numpy as np
    import torch

    from inputs import configs
    from paper_2608_03065_amd.psc import Classifier, apply_mask, pack_states

    dev = torch.device("cuda:0")
    wl = configs.get(args.workload)
    if args.batch is not None:
        import dataclasses
        if not 1 <= args.batch <= 65535:
            print(json.dumps({"error": "--batch must be in 1..65535"}))
            sys.exit(2)
        wl = dataclasses.replace(wl, B=args.batch)
    B, V = wl.B, wl.V
    W = (V + 31) // 32
    s_logit = 2 if wl.logits_dtype == "bf16" else 4
    log(f"workload {wl.name}: B={B} V={V} dtype={wl.logits_dtype}")

    if args.latency_probe:
        from paper_2608_03065_amd.probe import chase_latency
        stream = torch.cuda.Stream(device=dev)     # default priority
        grid = ((W + 255) // 256, B)              # the fused step's grid for bf16 logits
        res = chase_latency(dev, stream, grid)
        print(json.dumps({"latency_probe": res, "config": {"workload": wl.name, "grid": list(grid),
                                                           "dependent_loads": 8, "launches": 500},
                          "note": "per extra dependent load: (t(8) - t(0)) / 8 over back-to-back launches, each "
                                  "starting its chains at other rows of a table of random 1 KiB rows; wave_1KiB is "
                                  "a sparse row's or chain's load, scalar_8B a dense row's entry; with_stores adds "
                                  "the step's 16 KiB per workgroup of nontemporal stores"}), flush=True)
        return

    t0 = time.time()
    clf = Classifier(wl.grammar, wl.vocab)
    info = clf.info()
    log(f"psc_build {info['build_seconds']:.2f}s states={info['dfa_states']} classes={info['n_classes']}"
        f" (total setup {time.time() - t0:.1f}s)")
    stream = torch.cuda.Stream(device=dev)     # default priority
    clf.bind(dev, stream=stream, layout=args.masks)
    clf.set_options(speculate=args.speculate)

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

    # the class predictor, filled from prefix batches the timed steps do not
    # use (the workload's generator at step indices past its own), as a
    # decoding loop fills it from its first steps or a prompt set
    t0 = time.time()
    n_calib = 0
    with torch.cuda.stream(stream):
        for s_ in range(args.predictor_batches):
            st_, ln_, q_ = pack_states(wl.states(wl.steps + s_), dev)
            clf.compute_classes(st_, ln_, q_, stream=stream)
            n_calib += B
    torch.cuda.synchronize()
    calib_updates = clf.predictor_updates(reset=True, stream=stream)
    log(f"class predictor: {args.predictor_batches} held-out batches walked ({time.time() - t0:.1f}s), "
        f"{calib_updates} entries set")

    # a device-side delay in front of a timed loop lets the host queue the
    # whole loop before the first event fires, so that the host's launch
    # latency stays out of the timed region (the GPU time of the steps)
    sleep_cycles_per_us = None

    def prequeue(n_calls, us_per_call=12.0):
        nonlocal sleep_cycles_per_us
        if args.no_prequeue:
            return
        if sleep_cycles_per_us is None:
            a_, z_ = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda._sleep(1000)
            a_.record(stream)
            torch.cuda._sleep(1 << 20)
            z_.record(stream)
            torch.cuda.synchronize()
            sleep_cycles_per_us = (1 << 20) / max(a_.elapsed_time(z_) * 1e3, 1.0)
        want_us = min(100.0 + n_calls * us_per_call, 60000.0)
        torch.cuda._sleep(int(want_us * sleep_cycles_per_us))

    def fused_step(i):
        stacks, lens, qs = step_inputs[i % n_distinct]
        clf.compute_and_apply(stacks, lens, qs, pool[i % n_pool], out=bms[i % n_bm], stream=stream)

    def two_launch_step(i):
        stacks, lens, qs = step_inputs[i % n_distinct]
        bm = bms[i % n_bm]
        clf.compute_masks(stacks, lens, qs, out=bm, stream=stream)
        apply_mask(pool[i % n_pool], bm, stream=stream)

    step = fused_step if args.mode == "fused" else two_launch_step
    other = two_launch_step if args.mode == "fused" else fused_step

    def loop(fn, n, warm=20):
        """HIP events on the bench stream around n back-to-back calls."""
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for i in range(warm):
            fn(i)
        torch.cuda.synchronize()
        prequeue(n)
        a.record(stream)
        for i in range(n):
            fn(i)
        z.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(z) / n * 1e3     # us per call

    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            step(i)
        torch.cuda.synchronize()

        # (1) the timed loop: exactly --steps steps, whole-step latency
        torch.cuda.synchronize()
        clf.predictor_updates(reset=True, stream=stream)
        ms_per_step = loop(step, args.steps, warm=0) * 1e-3
        timed_misses = clf.predictor_updates(reset=True, stream=stream)
        # (2) the other formulation of the same step, for comparison
        t_other = loop(other, min(args.steps, 1000))
        # (2b) the spread: the same back-to-back loop cut by events into
        # chunks of 20 steps (an event after every step would itself cost
        # more than a step's launch overlap), per-step time of each chunk
        chunk, n_chunks = 20, max(1, min(args.steps, 2000) // 20)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n_chunks + 1)]
        torch.cuda.synchronize()
        prequeue(n_chunks * chunk)
        evs[0].record(stream)
        for c in range(n_chunks):
            for i in range(c * chunk, (c + 1) * chunk):
                step(i)
            evs[c + 1].record(stream)
        torch.cuda.synchronize()
        per_step = np.array([evs[c].elapsed_time(evs[c + 1]) * 1e3 / chunk for c in range(n_chunks)])

        # (3) each kernel of the two-launch step alone, back to back
        def only_compute(i):
            stacks, lens, qs = step_inputs[i % n_distinct]
            clf.compute_masks(stacks, lens, qs, out=bms[i % n_bm], stream=stream)

        # masks of the first n_bm steps stay in bms for the apply-only loop
        for i in range(n_bm):
            only_compute(i)

        def only_apply(i):
            apply_mask(pool[i % n_pool], bms[i % n_bm], stream=stream)

        t_apply = loop(only_apply, 1000)     # masks of steps 0..n_bm-1, as counted below
        t_compute = loop(only_compute, 1000)

        # greedy decoding folded into the mask step (reads the logits only)
        tok_out = torch.empty(B, dtype=torch.int32, device=dev)

        def argmax_step(i):
            stacks, lens, qs = step_inputs[i % n_distinct]
            clf.compute_and_argmax(stacks, lens, qs, pool[i % n_pool], out=tok_out, stream=stream)

        t_argmax = loop(argmax_step, 1000)

        # the classification step alone (psc_compute_classes: the walk, one
        # wavefront per sequence, class ids out)
        cls_out = torch.empty(B, dtype=torch.int32, device=dev)

        def classes_step(i):
            stacks, lens, qs = step_inputs[i % n_distinct]
            clf.compute_classes(stacks, lens, qs, out=cls_out, stream=stream)

        # a call this short is bound by the host when launched eagerly, so
        # 100 of them are captured in a HIP graph and replayed
        t_walk_eager = loop(classes_step, 1000)
        g_walk = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_walk, stream=stream):
            for i in range(100):
                classes_step(i)
        g_walk.replay()
        torch.cuda.synchronize()
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(10):
            g_walk.replay()
        z.record(stream)
        torch.cuda.synchronize()
        t_walk = a.elapsed_time(z) / 1000 * 1e3
        del g_walk

        # inputs handed over from pinned host memory: the copies alone, and
        # copies + the step (PCIe-inclusive; never the headline)
        host_in = []
        for s_ in range(min(n_distinct, 8)):
            host_in.append(tuple(t.cpu().pin_memory() for t in step_inputs[s_]))
        dev_in = [tuple(torch.empty(h.shape, dtype=h.dtype, device=dev) for h in hs) for hs in host_in]

        def upload(i):
            for d, h in zip(dev_in[i % len(host_in)], host_in[i % len(host_in)]):
                d.copy_(h, non_blocking=True)

        def upload_step(i):
            upload(i)
            stacks, lens, qs = dev_in[i % len(host_in)]
            clf.compute_and_apply(stacks, lens, qs, pool[i % n_pool], out=bms[i % n_bm], stream=stream)

        t_upload = loop(upload, 1000)
        t_upload_step = loop(upload_step, 1000)

        def graph_loop(fn, G=100, reps=10):
            """G calls captured in a HIP graph (rotating inputs and logits as
            above), replayed back to back: the GPU-side time per call, free
            of the host's per-call cost."""
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=stream):
                for i in range(G):
                    fn(i)
            graph.replay()
            torch.cuda.synchronize()
            a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for _ in range(reps):
                graph.replay()
            z.record(stream)
            torch.cuda.synchronize()
            del graph
            return a.elapsed_time(z) / (reps * G) * 1e3

        t_graph = graph_loop(step, reps=max(1, min(args.steps, 2000) // 100))
        t_other_graph = graph_loop(other)
        t_compute_graph = graph_loop(only_compute)
        for i in range(n_bm):
            only_compute(i)
        t_apply_graph = graph_loop(only_apply)
        t_argmax_graph = graph_loop(argmax_step)

        # what plain streaming kernels of the same size achieve on this GPU
        # (torch's own fill and copy of one logits tensor, graph-replayed):
        # the practical ceiling for a launch that touches this many bytes
        def fill(i):
            pool[i % n_pool].fill_(float("-inf"))

        # (a single-buffer pool copies from a spare tensor: a copy onto itself
        # launches nothing)
        spare = torch.empty_like(pool[0]) if n_pool == 1 else None

        def copy(i):
            pool[i % n_pool].copy_(pool[(i + 7) % n_pool] if spare is None else spare)

        # (after every timing of the mask kernels: the logits values do not
        # affect the kernels' work, but the pool is overwritten from here on)
        t_fill = graph_loop(fill)
        t_copy = graph_loop(copy)

        # the apply kernel's floors at this shape: an all-zero bitmask (every
        # vector one store of -inf, no logits read) and an all-one bitmask
        # (no logits touched: the launch and the bitmask read); beside
        # apply_mask_solo they show what reading the mixed vectors costs
        bm_const = {"all_masked": torch.zeros((B, W), dtype=torch.int32, device=dev),
                    "all_allowed": torch.full((B, W), -1, dtype=torch.int32, device=dev)}
        t_apply_floor = {}
        for name_, bm_c in bm_const.items():
            t_apply_floor[name_] = round(loop(lambda i: apply_mask(pool[i % n_pool], bm_c, stream=stream), 1000), 3)

        tl = None
        if args.timeline > 0 and V % 32 != 0:
            tl = {"skipped": "the timeline records come from the fast path of the fused step (V % 32 == 0)"}
        elif args.timeline > 0:
            tl = timeline(clf, wl, step_inputs, pool, bms, stream, dev, args.timeline, prequeue)

        # (4) Algorithm 2 entirely on the GPU: device-resident prefix states
        # advanced by one token each (psc_advance), then the single-launch
        # step on them (psc_compute_and_apply_dense)
        decode = decode_steps(wl, clf, B, pool, bms, stream, dev, args.decode_steps)

    # Algorithmic bytes, from the actual masks.  The apply touches logits per
    # 16-byte vector: one whose entries are all masked is written once
    # (16 B); one that keeps some entries and masks others must be read to be
    # written (32 B); one that keeps all entries is not touched.  (V % 32 == 0
    # here, so vectors never straddle rows.)  The walk reads the stacks, lens
    # and states; the gather reads the class's mask row and writes the
    # bitmask (4 W B each); the two-launch apply reads the bitmask back.
    per_vec = 16 // s_logit
    logit_bytes, stack_total = [], 0
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
        logit_bytes.append(16 * n_masked + 32 * n_mixed)
        stack_total += int(lens.sum().item())
    stack_words = stack_total / n_distinct
    bytes_walk_gather = 4 * stack_words + 8 * B + 2 * 4 * W * B
    bytes_fused = bytes_walk_gather + float(np.mean(logit_bytes))
    bytes_two_launch = bytes_fused + 4 * W * B
    bytes_step = bytes_fused if args.mode == "fused" else bytes_two_launch
    one_pass_model = B * (2 * V * s_logit + 3 * 4 * W) + 4 * (stack_words + 2 * B)

    lat_us = ms_per_step * 1e3
    masks_per_s = B / (ms_per_step * 1e-3)
    bytes_apply_solo = 4 * W * B + float(np.mean(logit_bytes[:n_bm]))
    achieved_apply = bytes_apply_solo / (t_apply * 1e-6) / 1e9
    fast = V % 32 == 0
    if args.mode == "fused":
        kname = ("fused_spec_kernel" if args.speculate else "fused_fast_kernel") if fast else "fused_generic_kernel"
        achieved = bytes_fused / (lat_us * 1e-6) / 1e9
        roofline = {
            "bound": "hbm", "kernel": kname,
            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(wl, kname) if fast else None,
            "algorithmic_bytes_per_launch": round(bytes_fused),
            "avg_launch_us": round(lat_us, 3),
            "timing": "HIP events on the bench stream around the timed loop; one launch per step",
            # the read-every-logit-and-write-it-back byte model, for comparison
            # only: the kernel does not move these bytes (fully masked vectors
            # are only written, kept ones not touched)
            "one_pass_model": {"bytes": round(one_pass_model),
                               "gbs": round(one_pass_model / (lat_us * 1e-6) / 1e9, 1),
                               "frac": round(one_pass_model / (lat_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)},
        }
    else:
        kname = "apply_fast_kernel" if fast else "apply_generic_kernel"
        roofline = {
            "bound": "hbm", "kernel": kname,
            "achieved": round(achieved_apply, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved_apply / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(wl, kname) if fast else None,
            "algorithmic_bytes_per_launch": round(bytes_apply_solo),
            "avg_launch_us": round(t_apply, 3),
            "timing": "HIP events around 1000 back-to-back launches of the kernel alone on the bench stream",
        }

    # the two-call step of the boundary (psc_compute_masks, then
    # psc_apply_mask on the same stream), measured as the other mode above
    t_two = t_other if args.mode == "fused" else lat_us
    ach_two = bytes_two_launch / (t_two * 1e-6) / 1e9
    roofline_two = {
        "calls": "psc_compute_masks + psc_apply_mask (two launches, one stream)",
        "bound": "hbm", "kernels": ["walk_gather_kernel", "apply_fast_kernel" if fast else "apply_generic_kernel"],
        "achieved": round(ach_two, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(ach_two / HBM_PEAK_GBS, 4), "algorithmic_bytes_per_step": round(bytes_two_launch),
        "step_us": round(t_two, 3),
        "per_kernel_us": {"compute_masks": round(t_compute, 3), "apply_mask": round(t_apply, 3),
                          "compute_masks_graph": round(t_compute_graph, 3),
                          "apply_mask_graph": round(t_apply_graph, 3)},
    }
    if args.mode == "fused":
        roofline["calls"] = "psc_compute_and_apply (one launch)"

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, step_states, args.cpu_seconds, B, clf)

    out = {
        "metric": METRIC,
        "value": round(masks_per_s, 1),
        "unit": "masks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "latency_us": round(lat_us, 3),
        "latency_us_dist": {"p10": round(float(np.percentile(per_step, 10)), 3),
                            "p50": round(float(np.percentile(per_step, 50)), 3),
                            "p90": round(float(np.percentile(per_step, 90)), 3),
                            "max": round(float(per_step.max()), 3), "chunks": int(n_chunks),
                            "note": f"per-step time of each run of {chunk} consecutive steps of a back-to-back "
                                    "loop (HIP events on the bench stream between the runs)"},
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
            "batch_override": args.batch is not None,
        },
        "step_mode": args.mode,
        "other_mode_step_us": {("two_launch" if args.mode == "fused" else "fused"): round(t_other, 3),
                               ("two_launch" if args.mode == "fused" else "fused") + "_graph":
                                   round(t_other_graph, 3)},
        "decode_step_us": decode,
        "argmax_step_us": round(t_argmax, 3),
        "argmax_step_graph_us": round(t_argmax_graph, 3),
        "walk_us": {"graph_replayed": round(t_walk, 3), "eager": round(t_walk_eager, 3),
                    "call": "psc_compute_classes (the walk alone, class ids out)"},
        "stack_depth": {"mean": round(float(np.mean(depth_hist)), 2),
                        "p50": int(np.percentile(depth_hist, 50)), "p90": int(np.percentile(depth_hist, 90)),
                        "p99": int(np.percentile(depth_hist, 99)), "max": int(max(depth_hist)),
                        "hist": depth_histogram(depth_hist)},
        "host_inputs": {"upload_us": round(t_upload, 3), "upload_and_step_us": round(t_upload_step, 3),
                        "note": "stacks, lengths and lexer states copied from pinned host memory on the "
                                "bench stream before the step; PCIe-inclusive, not the headline"},
        "graph_step_us": round(t_graph, 3),
        "kernels_us": {"compute_masks_solo": round(t_compute, 3), "apply_mask_solo": round(t_apply, 3),
                       "apply_mask_all_masked": t_apply_floor["all_masked"],
                       "apply_mask_all_allowed": t_apply_floor["all_allowed"],
                       "apply_mask_solo_gbs": round(achieved_apply, 1),
                       "compute_masks_solo_graph": round(t_compute_graph, 3),
                       "apply_mask_solo_graph": round(t_apply_graph, 3)},
        "bytes_per_step": {"algorithmic": round(bytes_step), "fused": round(bytes_fused),
                           "two_launch": round(bytes_two_launch),
                           "one_pass_read_write_model": round(one_pass_model)},
        "roofline": roofline,
        "roofline_two_launch": roofline_two,
        "predictor": {"held_out_batches": args.predictor_batches, "entries_set": calib_updates,
                      "misses_in_timed_loop": timed_misses,
                      "miss_rate_in_timed_loop": round(timed_misses / max(1, args.steps * B), 4),
                      "note": "class predictor filled by psc_compute_classes over prefix batches the timed "
                              "steps do not use; a miss is a walk whose class differed from the prediction "
                              "(results never depend on it)"},
        "mask_layout": args.masks,
        "speculate": bool(args.speculate),
        "timing_method": ("each timed loop is queued behind a device-side delay (torch.cuda._sleep) so that "
                          "the host's launch latency is not in the timed region" if not args.no_prequeue else
                          "loops launched eagerly from the host"),
        "timeline": tl,
        "reference_kernels_us": {
            "torch_fill_logits": round(t_fill, 3), "torch_copy_logits": round(t_copy, 3),
            "fill_gbs": round(B * V * s_logit / (t_fill * 1e-6) / 1e9, 1),
            "copy_gbs": round(2 * B * V * s_logit / (t_copy * 1e-6) / 1e9, 1),
            "note": "torch's fill_ and copy_ of one [B, V] logits tensor, 100 per HIP graph, replayed"},
        "cpu_baseline": cpu,
        "build": {k: info[k] for k in ("dfa_states_built", "dfa_states", "n_classes", "table_bytes",
                                        "mask_table_bytes", "sliced_mask_bytes", "mask_slices_unique",
                                        "build_seconds", "dfa_rows", "dense_rows", "chain_states", "chains")},
    }
    print(json.dumps(out), flush=True)


def timeline(clf, wl, step_inputs, pool, bms, stream, dev, n_steps, prequeue):
    """n_steps back-to-back launches of the fused step's timeline variant
    (psc_compute_and_apply_timeline): per wavefront the GPU's 100 MHz clock
    at its start, after the walk's first step, when the class is known and
    after its last store.  Returns percentiles in microseconds, relative to
    the earliest start in each launch."""
    import numpy as np
    import torch
    B = wl.B
    tdt = pool[0].dtype
    n = clf.timeline_records(B, tdt)
    recs = torch.zeros((n_steps, n, 4), dtype=torch.int64, device=dev)
    n_distinct, n_pool, n_bm = len(step_inputs), len(pool), len(bms)
    torch.cuda.synchronize()
    prequeue(n_steps)
    for i in range(n_steps):
        st, ln, q = step_inputs[i % n_distinct]
        clf.compute_and_apply_timeline(st, ln, q, pool[i % n_pool], recs[i], out=bms[i % n_bm], stream=stream)
    torch.cuda.synchronize()
    r = recs.cpu().numpy().view(np.uint64).astype(np.int64)
    t0 = r[:, :, 0]
    tA, tB = t0 + (r[:, :, 1] & 0xFFFFFFFF), t0 + (r[:, :, 1] >> 32)
    tE, meta = t0 + (r[:, :, 2] & 0xFFFFFFFF), r[:, :, 2] >> 32
    wave, held, done = meta & 7, (meta >> 7) & 1, (meta >> 8) & 1
    start = t0.min(axis=1, keepdims=True)
    us = lambda x: x * 0.01                     # 100 MHz ticks

    def pct(x):
        return {k: round(float(v), 3) for k, v in zip(("p10", "p50", "p90", "max"),
                                                          np.percentile(x, [10, 50, 90, 100]))}
    walker, worker = wave == 0, wave > 0
    end = tE.max(axis=1)
    gaps = us(start[1:, 0] - end[:-1]) if n_steps > 1 else np.zeros(1)
    return {
        "steps": n_steps, "records_per_step": int(n),
        "wavefront_start_us": pct(us(t0 - start)[worker]),
        "prediction_known_us": pct(us(tA - start)[walker]),
        "class_known_us": pct(us(tB - start)[walker]),
        "last_store_issued_us": pct(us(tE - start)[worker]),
        "launch_span_us": pct(us(end - start[:, 0])),
        "gap_to_next_launch_us": pct(gaps),
        "walks_ended_at_first_step": round(float(done[walker].mean()), 4),
        "prediction_held": round(float(held[walker & (done == 0)].mean()) if (walker & (done == 0)).any() else 0.0,
                                 4),
        "note": "times from the earliest wavefront start of each launch; walker = wavefront 0 of a workgroup, "
                "workers = the wavefronts that move the data",
    }


def decode_steps(wl, clf, B, pool, bms, stream, dev, max_steps):
    """Per-token time of the grammar side of decoding with the prefix states
    kept on the GPU: psc_advance (one token per sequence), alone and followed
    by psc_compute_and_apply_dense.  Each sequence follows a document of the
    workload, tokenised by longest match; the final states are checked against
    the input generator's host parser."""
    import numpy as np
    import torch

    from inputs.seeds import rng_for
    from paper_2608_03065_amd.psc import DecodeStates
    toks, texts = [], []
    for b in range(B):
        best = b""
        for k in range(8):                      # a document of at least max_steps tokens if one comes
            d = wl.make_document(rng_for(wl.index, 0xDEC, b, k), wl)
            if len(d) > len(best):
                best = d
            if len(wl.vocab.tokenize(best)) >= max_steps:
                break
        texts.append(best)
        toks.append(wl.vocab.tokenize(best))
    n = max(1, min(max_steps, min(len(t) for t in toks)))
    cap = 4096
    tok_dev = torch.tensor(np.array([t[:n] for t in toks], np.int32).T.copy(), device=dev)   # [n, B]
    ds = DecodeStates(clf, B, cap, dev, stream)
    n_pool, n_bm = len(pool), len(bms)

    def run(mode):
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ds.reset(stream)
        torch.cuda.synchronize()
        a.record(stream)
        for k in range(n):
            if mode == "one_launch":
                ds.decode_step(tok_dev[k], pool[k % n_pool], out=bms[k % n_bm], stream=stream)
                continue
            ds.advance(tok_dev[k], stream)
            if mode == "two_launches":
                ds.compute_and_apply(pool[k % n_pool], out=bms[k % n_bm], stream=stream)
        z.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(z) / n * 1e3

    def check():
        # the states after n tokens equal the host parser's at the same cut
        got = ds.host_states()
        for b in range(B):
            cut = sum(len(wl.vocab.tokens[t]) for t in toks[b][:n])
            q, st = wl.host.states_at(texts[b], [cut])[0]
            if got[b][0] != q or not np.array_equal(got[b][1], st):
                raise RuntimeError("device states after the decoding loop differ from the host parser's")

    run("two_launches")
    t_both = run("two_launches")
    check()
    t_one = run("one_launch")
    check()
    t_adv = run("advance")
    check()
    return {"advance_and_fused_step": round(t_both, 3), "psc_decode_step": round(t_one, 3),
            "advance": round(t_adv, 3), "tokens_per_sequence": n, "cap": cap, "states_checked": True}


def device_code_hash() -> str:
    """sha256 (first 16 hex digits) of the device source with its comments
    and blank space removed: a change of the code, not of its comments,
    makes the stored counter readings stale."""
    import hashlib
    import re
    src = open(os.path.join(ROOT, "paper_2608_03065_amd", "csrc", "psc_device.hip")).read()
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    src = " ".join(src.split())
    return hashlib.sha256(src.encode()).hexdigest()[:16]


def workload_fingerprint(wl) -> str:
    """sha256 (first 16 hex digits) of what defines a workload's shape: its
    grammar's sizes, the vocabulary size and the batch.  Stored counter
    readings are for one such definition."""
    import hashlib
    g = wl.grammar
    key = f"{wl.name}|{g.n_terminals}|{g.n_nonterminals}|{g.n_lr_states}|{len(g.productions)}|{wl.V}|{wl.B}"
    return hashlib.sha256(key.encode()).hexdigest()[:16]


def measured_traffic(wl, kernel: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, or
    None when there is none for this workload, the workload's definition
    changed, or the kernel source changed since the counters were taken."""
    tag = {"arithmetic": "arithmetic_c1", "json": "json_c2", "schema": "schema_c3", "pylike": "pylike_c4",
           "stress": "stress_c5"}.get(wl.name, wl.name)
    path = os.path.join(ROOT, "profiles", f"mask_kernels_{tag}_pmc_traffic.md")
    if not os.path.exists(path):
        return None
    meta = None
    for line in open(path):
        if line.startswith("traffic_json: "):
            meta = json.loads(line[len("traffic_json: "):])
    h = device_code_hash()
    if not meta or meta.get("source_sha256_16") != h or kernel not in meta.get("kernels", {}):
        return None
    if meta.get("workload_sha256_16") != workload_fingerprint(wl):
        return None
    return meta["kernels"][kernel]["hbm_bytes"]


def depth_histogram(depths):
    """Counts of stack depths in power-of-two bins [2^k, 2^(k+1))."""
    import numpy as np
    d = np.asarray(depths)
    out = {}
    k = 1
    while k <= d.max():
        out[f"{k}-{2 * k - 1}"] = int(((d >= k) & (d < 2 * k)).sum())
        k *= 2
    return out


def cpu_baseline(wl, step_states, seconds, B, clf):
    """The oracle as it stands, on this host's cores, over a bounded sample;
    beside it, the oracle on one thread (ns per token check) and the paper's
    own CPU method (the host walk of the same classifier plus the copy of the
    class's mask row, one thread, per sequence)."""
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
    cores = int(orc.threads_used)
    # one thread
    t0 = time.time()
    orc.masks(flat[:1], n_threads=1)
    one1 = time.time() - t0
    n1 = int(max(1, min(len(flat), 2.0 / max(one1, 1e-4))))
    t0 = time.time()
    orc.masks(flat[:n1], n_threads=1)
    dt1 = time.time() - t0
    # the paper's method on one CPU thread: walk, then the mask row copy
    sample = flat[:min(len(flat), 4096)]
    classes = clf.classify_host(sample)
    rows = {int(c): clf.class_mask(int(c)) for c in np.unique(classes)}
    table = np.zeros((max(rows) + 1, clf.W), np.uint32)
    for c, r in rows.items():
        table[c] = r
    t0 = time.perf_counter()
    reps = 0
    while True:
        c = clf.classify_host(sample)
        out = table[c]
        reps += 1
        if time.perf_counter() - t0 > 1.0:
            break
    t_psc = (time.perf_counter() - t0) / (reps * len(sample))
    del out
    return {
        "value": round(n / dt, 3), "unit": "masks/s", "cores": cores, "kind": "oracle",
        "sample": f"first {n} sequences (of {len(flat)}) of the benchmark's prefix batches, "
                  f"all {wl.V} tokens each; {dt:.1f}s wall",
        "per_step_latency_us": round(dt / n * B * 1e6, 1),
        "single_thread_ns_per_token_check": round(dt1 / (n1 * wl.V) * 1e9, 2),
        "single_thread_sample": f"first {n1} sequences, {dt1:.1f}s",
        "paper_method_cpu_us_per_sequence": round(t_psc * 1e6, 3),
        "paper_method_note": "host walk of the same classifier (psc_classify_host) plus a copy of the "
                             "class's mask row, one thread, over the first "
                             f"{len(sample)} sequences; the paper reports 2.2-2.6 us per token on one "
                             "Xeon Gold 6348 thread (Python)",
    }


if __name__ == "__main__":
    main()
