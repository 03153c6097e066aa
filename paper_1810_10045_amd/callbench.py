"""Per-entry-point times of the hot path, with cold and with warm caches.

For each workload, each stage of the step (Unique; Seg-Sum; the stage after
it: the apply, SCATTER or the merge's EXPAND) is timed on its own, with HIP
events on the launch stream around just that stage:

  cold  before every timed rep, a 1 GiB buffer is read, which leaves nothing
        of the inputs in the 256 MB Infinity Cache or the L2s (read, not
        written, so that the timed call never pays for writing back the
        evicting data); reps cycle through the resident batches.
  warm  no eviction and the same batch every rep: whatever of the inputs the
        caches hold from the previous rep stays there.

Each is 5 untimed reps, then --reps timed ones; the table gives the median,
10th and 90th percentile in microseconds, Seg-Sum's algorithmic GB/s and its
fraction of the 8 TB/s HBM peak (from the median), and tokens/s = K / the sum
of the three cold medians. Usage (one GPU):

    python -m paper_1810_10045_amd.callbench [--workloads a,b,...] [--reps 20]
"""
from __future__ import annotations

import argparse
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402  (HipEvents, Batch, Pipeline, segsum_bytes)

DEFAULT = "word_tiny_8k,word_step_64k,merge_64x32k_bf16,char_heavy_1m,vocab2m_adam_i64"
STAGES = ("unique", "segsum", "after")
EVICT_BYTES = 1 << 30


def time_stage(pipe, stage, cold, reps, nbatch, torch, scratch, stream):
    """Microseconds of one stage over reps timed reps (after 5 untimed)."""
    ev = bench.HipEvents(2 * reps)
    out = []
    for r in range(-5, reps):
        b = (r % nbatch) if cold else 0

        def mark(k, r=r):
            if k == stage and cold:
                scratch.sum()  # read the whole buffer: evicts the caches
            if r >= 0 and k == stage:
                ev.record(2 * r, stream)
            if r >= 0 and k == stage + 1:
                ev.record(2 * r + 1, stream)

        pipe.step(b, mark)
    torch.cuda.synchronize()
    out = [1e3 * ev.ms(2 * r, 2 * r + 1) for r in range(reps)]
    ev.close()
    return np.array(out)


def run(workload, reps, torch, lz, synth):
    w = synth.WORKLOADS[workload]
    dev = torch.device("cuda:0")
    gb = 2 if w.grad_dtype == "bf16" else 4
    nbatch = max(1, min(8, math.ceil((2 << 30) / (w.tokens * w.D * gb))))
    batches = [bench.Batch(w.batch(b), torch, dev) for b in range(nbatch)]
    pipe = bench.Pipeline(w, batches, torch, lz, dev)
    U = []
    for b in range(nbatch):
        pipe.step(b)
        torch.cuda.synchronize()
        U.append(int(pipe.ures.num_unique.item()))
    lz.check(pipe.dev_err)
    scratch = torch.empty(EVICT_BYTES // 4, dtype=torch.int32, device=dev).fill_(1)
    stream = torch.cuda.current_stream()
    res = {}
    for mode, cold in (("cold", True), ("warm", False)):
        for s, name in enumerate(STAGES):
            res[(mode, name)] = time_stage(pipe, s, cold, reps, nbatch, torch, scratch, stream)
    lz.check(pipe.dev_err)
    del scratch
    seg_cold = np.mean([bench.segsum_bytes(w.tokens, w.D, u, gb) for u in U])
    seg_warm = bench.segsum_bytes(w.tokens, w.D, U[0], gb)
    return w, U, res, seg_cold, seg_warm


def table(w, U, res, seg_cold, seg_warm):
    pct = lambda a: (np.median(a), np.percentile(a, 10), np.percentile(a, 90))
    lines = [f"### {w.name}: K = {w.tokens:,}, V = {w.V:,}, D = {w.D}, {w.grad_dtype} gradients, "
             f"{w.id_dtype} ids, after Seg-Sum: {w.step}; U per batch {min(U):,}..{max(U):,}",
             "", "| stage | cold median | cold p10 | cold p90 | warm median | warm p10 | warm p90 |",
             "|---|---|---|---|---|---|---|"]
    for name in STAGES:
        c, h = pct(res[("cold", name)]), pct(res[("warm", name)])
        label = w.step if name == "after" else name
        lines.append(f"| {label} | {c[0]:.1f} | {c[1]:.1f} | {c[2]:.1f} | {h[0]:.1f} | {h[1]:.1f} | "
                     f"{h[2]:.1f} |")
    sc, sw = np.median(res[("cold", "segsum")]), np.median(res[("warm", "segsum")])
    gbc, gbw = seg_cold / sc / 1e3, seg_warm / sw / 1e3
    step = sum(np.median(res[("cold", n)]) for n in STAGES)
    lines += ["", f"Seg-Sum: {seg_cold / 1e6:.1f} MB algorithmic per call; cold {gbc:,.0f} GB/s "
              f"(frac {gbc / bench.HBM_PEAK_GBPS:.3f}), warm {gbw:,.0f} GB/s "
              f"(frac {gbw / bench.HBM_PEAK_GBPS:.3f}). Cold step {step:.1f} us: "
              f"{w.tokens / step * 1e6 / 1e6:,.1f} M tokens/s.", ""]
    return "\n".join(lines)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workloads", default=DEFAULT)
    ap.add_argument("--reps", type=int, default=20)
    args = ap.parse_args()
    import torch
    from paper_1810_10045_amd import lmzipf as lz
    from paper_1810_10045_amd import synth
    for name in args.workloads.split(","):
        w, U, res, seg_cold, seg_warm = run(name, args.reps, torch, lz, synth)
        print(table(w, U, res, seg_cold, seg_warm), flush=True)
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
