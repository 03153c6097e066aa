"""Per-entry-point times of the hot path with cold and warm caches, and the
reference rates of plain memory patterns on the same shapes (one GPU).

Per entry point (default mode). For each workload, each stage of the step
(Unique; Seg-Sum; the stage after it: the apply, SCATTER or the merge's
EXPAND; where the step is a SCATTER into a dense table or an SGD update,
also lm_segsum_rows or lm_segsum_sgd, which does Seg-Sum and that update in
one call) is timed on its own, with HIP events on the launch stream around
just that stage:

  cold  before every timed rep, a 1 GiB buffer is read, which leaves nothing
        of the inputs in the 256 MB Infinity Cache or the L2s (read, not
        written, so that the timed call never pays for writing back the
        evicting data); reps cycle through the resident batches.
  warm  no eviction and the same batch every rep: whatever of the inputs the
        caches hold from the previous rep stays there.

Each is 5 untimed reps, then --reps timed ones; the table gives the median,
10th and 90th percentile in microseconds, Seg-Sum's algorithmic GB/s and its
fraction of the 8 TB/s HBM peak (from the median), and tokens/s = K / the sum
of the cold medians of the step's stages (Unique and the fused call where
the SCATTER or SGD is fused).

Ceilings (--ceilings). Plain torch operations on a workload's shapes (its K
gradient rows of D fp32, its U types), each rep on the next of several
resident sources and destinations (2 GiB or more of each), so that nothing
comes from the Infinity Cache:

  read          grad.sum(0): sequential read of K x D
  copy          dst.copy_(src), K x D fp32: sequential read and write (50/50)
  zero fill     dst.zero_(), K x D fp32: sequential write
  row gather    torch.index_select(grad, 0, perm): K rows read in the order
                of the stable sort permutation of the step's ids, written
                contiguously (the Seg-Sum's read pattern, with every row
                written back instead of one per type)
  row scatter   table.index_copy_(0, uniq, rows): U rows written at the
                ascending type ids of the V-row table (the apply's write
                pattern)

Usage:
    python bench_calls.py [--workloads a,b,...] [--reps 20]
    python bench_calls.py --ceilings [--workloads word_step_64k] [--reps 20]
"""
from __future__ import annotations

import argparse
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402  (HipEvents, Batch, Pipeline, segsum_bytes)

DEFAULT = "word_tiny_8k,word_step_64k,merge_64x32k_bf16,char_heavy_1m,vocab2m_adam_i64"
STAGES = ("unique", "segsum", "after")
EVICT_BYTES = 1 << 30


def time_stage(pipe, stage, cold, reps, nbatch, torch, scratch, stream):
    """Microseconds of one stage over reps timed reps (after 5 untimed)."""
    ev = bench.HipEvents(2 * reps)
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


def resident_batches(w):
    gb = 2 if w.grad_dtype == "bf16" else 4
    return max(1, min(8, math.ceil((2 << 30) / (w.tokens * w.D * gb))))


def run_calls(workload, reps, torch, lz, synth):
    w = synth.WORKLOADS[workload]
    dev = torch.device("cuda:0")
    gb = 2 if w.grad_dtype == "bf16" else 4
    nbatch = resident_batches(w)
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
    fused = pipe.fused
    for mode, cold in (("cold", True), ("warm", False)):
        pipe.fused = False
        for s, name in enumerate(STAGES):
            res[(mode, name)] = time_stage(pipe, s, cold, reps, nbatch, torch, scratch, stream)
        if fused:
            pipe.fused = True
            res[(mode, "rows")] = time_stage(pipe, 1, cold, reps, nbatch, torch, scratch, stream)
    pipe.fused = fused
    lz.check(pipe.dev_err)
    del scratch
    seg_cold = np.mean([bench.segsum_bytes(w.tokens, w.D, u, gb) for u in U])
    seg_warm = bench.segsum_bytes(w.tokens, w.D, U[0], gb)
    return w, U, res, seg_cold, seg_warm


def calls_table(w, U, res, seg_cold, seg_warm):
    pct = lambda a: (np.median(a), np.percentile(a, 10), np.percentile(a, 90))
    fused = ("cold", "rows") in res
    lines = [f"### {w.name}: K = {w.tokens:,}, V = {w.V:,}, D = {w.D}, {w.grad_dtype} gradients, "
             f"{w.id_dtype} ids, after Seg-Sum: {w.step}; U per batch {min(U):,}..{max(U):,}",
             "", "| stage | cold median | cold p10 | cold p90 | warm median | warm p10 | warm p90 |",
             "|---|---|---|---|---|---|---|"]
    for name in STAGES + (("rows",) if fused else ()):
        c, h = pct(res[("cold", name)]), pct(res[("warm", name)])
        label = {"after": w.step, "rows": bench.fused_stage(w)}.get(name, name)
        lines.append(f"| {label} | {c[0]:.1f} | {c[1]:.1f} | {c[2]:.1f} | {h[0]:.1f} | {h[1]:.1f} | "
                     f"{h[2]:.1f} |")
    sc, sw = np.median(res[("cold", "segsum")]), np.median(res[("warm", "segsum")])
    gbc, gbw = seg_cold / sc / 1e3, seg_warm / sw / 1e3
    step = sum(np.median(res[("cold", n)]) for n in (("unique", "rows") if fused else STAGES))
    lines += ["", f"Seg-Sum: {seg_cold / 1e6:.1f} MB algorithmic per call; cold {gbc:,.0f} GB/s "
              f"(frac {gbc / bench.HBM_PEAK_GBPS:.3f}), warm {gbw:,.0f} GB/s "
              f"(frac {gbw / bench.HBM_PEAK_GBPS:.3f}). Cold step {step:.1f} us: "
              f"{w.tokens / step * 1e6 / 1e6:,.1f} M tokens/s.", ""]
    if fused:
        ib = 8 if w.id_dtype == "i64" else 4
        # the row ids too, and with SGD the table rows read before they are written
        rb = seg_cold + np.mean([bench.fused_extra_bytes(w, w.D, u, ib) for u in U])
        rc = rb / np.median(res[("cold", "rows")]) / 1e3
        what = ("the U row ids" if w.step == "scatter" else
                "the U row ids, the U parameter rows read and the m and v rows read and written"
                if w.step == "adam" else
                "the U row ids and the U table rows read before they are written")
        lines[-1:-1] = [f"{bench.fused_stage(w).split()[0]}: {rb / 1e6:.1f} MB algorithmic per call "
                        f"(Seg-Sum's, {what}); cold {rc:,.0f} GB/s "
                        f"(frac {rc / bench.HBM_PEAK_GBPS:.3f})."]
    return "\n".join(lines)


def timed(fn, reps, stream, torch):
    """Milliseconds per rep of fn(r) over reps timed reps (after 3 untimed)."""
    ev = bench.HipEvents(2)
    for r in range(3):
        fn(r)
    torch.cuda.synchronize()
    ev.record(0, stream)
    for r in range(reps):
        fn(r)
    ev.record(1, stream)
    torch.cuda.synchronize()
    ms = ev.ms(0, 1) / reps
    ev.close()
    return ms


def run_ceilings(workload, reps, torch, synth):
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    w = synth.WORKLOADS[workload]
    K, D, V = w.tokens, w.D, w.V
    nb = max(2, resident_batches(dataclass_f32(w)))
    grads = [torch.randn((K, D), device=dev) for _ in range(nb)]
    perms, uniqs = [], []
    for b in range(nb):
        ids = w.batch(b).ids()
        perms.append(torch.from_numpy(np.argsort(ids, kind="stable")).to(dev))
        uniqs.append(torch.from_numpy(np.unique(ids).astype(np.int64)).to(dev))
    U = int(np.mean([u.numel() for u in uniqs]))
    outs = [torch.empty((K, D), device=dev) for _ in range(nb)]
    col = torch.empty(D, device=dev)
    table = torch.zeros((V, D), device=dev)
    rows = torch.randn((max(u.numel() for u in uniqs), D), device=dev)
    rb = K * D * 4
    res = []
    ms = timed(lambda r: torch.sum(grads[r % nb], 0, out=col), reps, stream, torch)
    res.append(("read", rb, ms))
    ms = timed(lambda r: outs[r % nb].copy_(grads[(r + 1) % nb]), reps, stream, torch)
    res.append(("copy", 2 * rb, ms))
    ms = timed(lambda r: outs[r % nb].zero_(), reps, stream, torch)
    res.append(("zero fill", rb, ms))
    ms = timed(lambda r: torch.index_select(grads[(r + 1) % nb], 0, perms[r % nb], out=outs[r % nb]),
               reps, stream, torch)
    res.append(("row gather", 2 * rb + K * 8, ms))
    ms = timed(lambda r: table.index_copy_(0, uniqs[r % nb], rows[:uniqs[r % nb].numel()]),
               reps, stream, torch)
    res.append(("row scatter", 2 * U * D * 4 + U * 8, ms))
    lines = [f"### {w.name} shapes: K = {K:,} rows of {D} fp32, mean U = {U:,}, V = {V:,}; "
             f"{nb} resident copies; GPU {torch.cuda.get_device_name(0)}", "",
             "| pattern | bytes per call | us | GB/s | fraction of 8 TB/s |", "|---|---|---|---|---|"]
    for name, nbytes, t in res:
        lines.append(f"| {name} | {nbytes / 1e6:.1f} MB | {t * 1e3:.1f} | {nbytes / t / 1e6:,.0f} | "
                     f"{nbytes / t / 1e6 / bench.HBM_PEAK_GBPS:.3f} |")
    del grads, outs, table, rows
    torch.cuda.empty_cache()
    return "\n".join(lines) + "\n"


def dataclass_f32(w):
    import dataclasses
    return dataclasses.replace(w, grad_dtype="f32")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--workloads", default=None)
    ap.add_argument("--reps", type=int, default=20)
    ap.add_argument("--ceilings", action="store_true",
                    help="reference rates of plain memory patterns instead of the entry points")
    args = ap.parse_args()
    import torch
    from paper_1810_10045_amd import synth
    if args.ceilings:
        for name in (args.workloads or "word_step_64k").split(","):
            print(run_ceilings(name, args.reps, torch, synth), flush=True)
        return
    from paper_1810_10045_amd import lmzipf as lz
    for name in (args.workloads or DEFAULT).split(","):
        w, U, res, seg_cold, seg_warm = run_calls(name, args.reps, torch, lz, synth)
        print(calls_table(w, U, res, seg_cold, seg_warm), flush=True)
        torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
