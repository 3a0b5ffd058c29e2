"""Every step of every workload through the benchmarked step, against the oracle.

Not collected by pytest (it runs for minutes, mostly in the oracle); run it
on a machine with the GPU, from the repository root:

    python tests/parity_all_steps.py [--workloads arithmetic,json,schema,pylike,stress]

For each workload and each of its decoding steps, the step's prefix batch
goes through psc_compute_and_apply (one launch: walk, mask row, bitmask,
masked logits), and the bitmask it writes is compared bit for bit with the
oracle's masks of the same prefix states.  Prints one line per workload and
a JSON summary; exits 1 on the first mismatch, naming workload, step and
rows.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workloads", default="arithmetic,json,schema,pylike,stress")
    ap.add_argument("--steps", type=int, default=0, help="first N steps only (default: all)")
    args = ap.parse_args()
    import numpy as np
    import torch
    from inputs import configs
    from oracle import Oracle
    from paper_2608_03065_amd.psc import Classifier, pack_states

    dev = torch.device("cuda:0")
    summary = {}
    for name in args.workloads.split(","):
        wl = configs.get(name)
        t0 = time.time()
        clf = Classifier(wl.grammar, wl.vocab)
        clf.bind(dev)
        orc = Oracle(wl.grammar, wl.vocab)
        tdt = torch.bfloat16 if wl.logits_dtype == "bf16" else torch.float32
        logits = torch.zeros((wl.B, wl.V), dtype=tdt, device=dev)
        out = torch.empty((wl.B, clf.W), dtype=torch.int32, device=dev)
        n_steps = wl.steps if args.steps <= 0 else min(args.steps, wl.steps)
        rows = 0
        t_orc = 0.0
        for s in range(n_steps):
            states = wl.states(s)
            stacks, lens, qs = pack_states(states, dev)
            clf.compute_and_apply(stacks, lens, qs, logits, out=out)
            got = out.cpu().numpy().view(np.uint32)
            t = time.time()
            want = orc.masks(states)
            t_orc += time.time() - t
            bad = np.nonzero((got != want).any(axis=1))[0]
            if bad.size:
                print(json.dumps({"workload": name, "step": s, "mismatched_rows": bad[:16].tolist()}), flush=True)
                sys.exit(1)
            rows += len(states)
            if (s + 1) % 100 == 0:
                print(f"[parity] {name}: {s + 1}/{n_steps} steps identical", flush=True)
        errs = clf.error_count()
        if errs:
            print(json.dumps({"workload": name, "device_errors": errs}), flush=True)
            sys.exit(1)
        summary[name] = {"steps": n_steps, "rows": rows, "B": wl.B, "V": wl.V,
                         "token_checks": rows * wl.V, "oracle_s": round(t_orc, 1),
                         "wall_s": round(time.time() - t0, 1), "identical": True}
        print(f"[parity] {name}: all {n_steps} steps ({rows} rows x {wl.V} tokens) identical "
              f"({time.time() - t0:.0f} s)", flush=True)
    print(json.dumps({"parity_all_steps": summary}), flush=True)


if __name__ == "__main__":
    main()
