"""Reference rates of plain memory patterns on the GPU, for reading the
roofline fractions of the hot path against what the memory system delivers
for the same kind of traffic. Every pattern runs as one torch operation on
the word-step shapes (65,536 gradient rows of 1024 fp32, 25.7K of them
written back), timed with fence-free HIP events on the launch stream. Each
rep takes the next of 8 resident sources and destinations (2 GiB of each),
so that neither comes from the 256 MB Infinity Cache:

  copy          dst.copy_(src), K x D fp32: sequential read and write (50/50)
  zero fill     dst.zero_(), K x D fp32: sequential write
  row gather    torch.index_select(grad, 0, perm): K rows of 4 KiB read in
                the order of the stable sort permutation of the step's ids,
                written contiguously (the Seg-Sum's read pattern, with every
                row written back instead of one per type)
  row scatter   table.index_copy_(0, uniq, rows): U rows of 4 KiB written at
                the ascending type ids of a 800,000-row table (the apply's
                write pattern)

Usage (one GPU): python -m paper_1810_10045_amd.ceilings [--reps 20]
"""
from __future__ import annotations

import argparse
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import bench  # noqa: E402  (HipEvents)
from paper_1810_10045_amd import synth  # noqa: E402


def timed(fn, reps, stream, torch):
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--reps", type=int, default=20)
    args = ap.parse_args()
    import torch
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    w = synth.WORKLOADS["word_step_64k"]
    K, D, V = w.tokens, w.D, w.V
    nb = 8
    grads = [torch.randn((K, D), device=dev) for _ in range(nb)]
    perms, uniqs = [], []
    for b in range(nb):
        ids = w.batch(b).ids()
        perms.append(torch.from_numpy(np.argsort(ids, kind="stable")).to(dev))
        uniqs.append(torch.from_numpy(np.unique(ids).astype(np.int64)).to(dev))
    U = int(np.mean([u.numel() for u in uniqs]))
    outs = [torch.empty((K, D), device=dev) for _ in range(nb)]
    table = torch.zeros((V, D), device=dev)
    rows = torch.randn((max(u.numel() for u in uniqs), D), device=dev)
    rb = K * D * 4
    res = []
    ms = timed(lambda r: outs[r % nb].copy_(grads[(r + 3) % nb]), args.reps, stream, torch)
    res.append(("copy", 2 * rb, ms))
    ms = timed(lambda r: outs[r % nb].zero_(), args.reps, stream, torch)
    res.append(("zero fill", rb, ms))
    ms = timed(lambda r: torch.index_select(grads[(r + 3) % nb], 0, perms[r % nb], out=outs[r % nb]),
               args.reps, stream, torch)
    res.append(("row gather", 2 * rb + K * 8, ms))
    ms = timed(lambda r: table.index_copy_(0, uniqs[r % nb], rows[:uniqs[r % nb].numel()]),
               args.reps, stream, torch)
    res.append(("row scatter", 2 * U * D * 4 + U * 8, ms))
    print(f"GPU: {torch.cuda.get_device_name(0)}; K = {K}, D = {D}, mean U = {U}")
    print("| pattern | bytes per call | us | GB/s | fraction of 8 TB/s |")
    print("|---|---|---|---|---|")
    for name, nbytes, t in res:
        print(f"| {name} | {nbytes / 1e6:.1f} MB | {t * 1e3:.1f} | {nbytes / t / 1e6:,.0f} | "
              f"{nbytes / t / 1e6 / bench.HBM_PEAK_GBPS:.3f} |")


if __name__ == "__main__":
    main()
