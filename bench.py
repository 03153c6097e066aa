"""Throughput of the Zipf gradient-compression hot path on one MI355X.

One step = one pass of the whole path over one batch of synthetic tokens
already resident in HBM:
    Unique (lm_unique) -> Seg-Sum (lm_segsum) -> Fill-Values / update
(EXPAND into the merged type list via lm_fill_values, by workload; a
SCATTER into a dense table and an SGD or Adam update are done by Seg-Sum
itself: lm_segsum_rows writes each type's row to its table row,
lm_segsum_sgd and lm_segsum_adam apply it there). The
headline workload is the largest one with fp32 gradients: K = 1,048,576
Zipf(1.2) token ids over a 20K character vocabulary, 2048-wide fp32
gradients (8 GiB per batch), the U reduced rows written into the dense
20K x 2048 table. Steps cycle
through resident batches (at least 2 GiB of gradients in all) so that the
gradient rows are not served from the 256 MB Infinity Cache.

The headline runs the Unique calls on a second stream, ahead of Seg-Sum and
the update (Unique reads only the token ids, which a trainer has before the
gradients exist), in groups of steps so that the two streams meet once per
group (OVERLAP_GROUP); every step still does all of its work. At the char-LM workload the two streams run on disjoint CUs
(CU-masked streams, SIDE_CUS); the same schedule on shared CUs is printed
beside it (`overlapped_all_cus`). The serial schedule (one stream) is timed too and printed beside it,
and for the SCATTER, SGD and Adam workloads also the serial schedule with
that update as a call of its own after lm_segsum (`unfused_serial`).

Prints one JSON line: tokens/s, ms per step, the Seg-Sum roofline (algorithmic
bytes per lm_segsum call / its average duration from HIP events on the launch
stream, all of the call's kernels), the CPU oracle timed on whole copies of
the same batch (one thread, and every core of the process), the check of the
timed kernels' outputs against the oracle's, and the same figures for each of
the five workloads (`workloads`), measured in the same run.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

HBM_PEAK_GBPS = 8000.0
METRIC = "tokens/s through Unique+Seg-Sum+Fill-Values; achieved HBM GB/s vs peak"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "segsum_traffic_{workload}.md")
SEGSUM_SRCS = [os.path.join(ROOT, "paper_1810_10045_amd", "csrc", f)
               for f in ("segsum.hip", "common.hpp")]
COPY_BYTES = 1 << 30  # the plain copy that scales the HBM byte counters
SEGSUM_KERNELS = "lm_segsum (k_segsum: walk and fix-up workgroups in one launch)"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def segsum_source_hash() -> str:
    """Hash of the Seg-Sum sources' code: comments, blank lines and trailing
    blanks left out, so that only a change of what is compiled voids the
    recorded counters."""
    h = hashlib.sha256()
    for path in SEGSUM_SRCS:
        with open(path) as f:
            text = re.sub(r"/\*.*?\*/", "", f.read(), flags=re.S)
        for line in text.splitlines():
            line = re.sub(r"//.*$", "", line).rstrip()
            if line:
                h.update(line.encode() + b"\n")
    return h.hexdigest()[:16]


def segsum_bytes(K, D, U, grad_bytes):
    """Algorithmic bytes of one Seg-Sum: read every gradient row once, write
    every type row once, read the permutation and the offsets."""
    return K * D * grad_bytes + U * D * 4 + K * 4 + (U + 1) * 4


def unique_bytes(K, U, id_bytes):
    """Algorithmic bytes of one Unique: read the ids, write the inverse map
    and the permutation, write the type ids, counts and offsets."""
    return K * id_bytes + K * 4 + K * 4 + U * (id_bytes + 8)


# Algorithmic bytes of the stage after Seg-Sum, per type row of D fp32: the
# apply reads the reduced row and reads and writes the table row (Adam also
# m and v); SCATTER reads the reduced row and writes the table row. The
# merge's EXPAND stage also runs shard 0's own Unique and Seg-Sum, so it has
# no single byte count here.
AFTER_ROWS = {"sgd": 3, "softmax_sgd": 3, "adam": 7, "scatter": 2}

# Steps done by the Seg-Sum call itself (lm_segsum_rows, lm_segsum_sgd), and
# the name of that fused stage.
FUSED_STEPS = ("scatter", "sgd", "softmax_sgd", "adam")


def fused_stage(w):
    return ("segsum_rows (segsum + scatter)" if w.step == "scatter" else
            "segsum_adam (segsum + adam)" if w.step == "adam" else "segsum_sgd (segsum + sgd)")


def fused_extra_bytes(w, D, U, id_bytes):
    """Bytes a fused call moves beyond lm_segsum's: the U row ids; for SGD
    the table rows it reads before it writes them; for Adam the parameter
    rows read, and the m and v rows read and written."""
    rows = {"scatter": 0, "adam": 5}.get(w.step, 1)
    return U * id_bytes + rows * U * D * 4


class HipEvents:
    """Timing events created with hipEventDisableSystemFence, recorded on the
    stream the kernels run on (torch's current stream). Torch's own events
    add a system-scope cache flush per record, about 5 us of idle GPU each."""

    DISABLE_TIMING = 0x2
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, n, timing=True):
        import ctypes
        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch already loaded
        self.hip.hipEventCreateWithFlags.argtypes = [ctypes.c_void_p, ctypes.c_uint]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipStreamWaitEvent.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint]
        flags = self.DISABLE_SYSTEM_FENCE | (0 if timing else self.DISABLE_TIMING)
        self.ev = []
        for _ in range(n):
            h = ctypes.c_void_p()
            rc = self.hip.hipEventCreateWithFlags(ctypes.byref(h), flags)
            if rc != 0:
                raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")
            self.ev.append(h)

    def record(self, i, stream):
        rc = self.hip.hipEventRecord(self.ev[i], self.ct.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def wait(self, i, stream):
        """Work queued on `stream` after this waits for event i's last record."""
        rc = self.hip.hipStreamWaitEvent(self.ct.c_void_p(stream.cuda_stream), self.ev[i], 0)
        if rc != 0:
            raise RuntimeError(f"hipStreamWaitEvent failed ({rc})")

    def ms(self, i, j):
        out = self.ct.c_float()
        rc = self.hip.hipEventElapsedTime(self.ct.byref(out), self.ev[i], self.ev[j])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return out.value

    def close(self):
        for h in self.ev:
            self.hip.hipEventDestroy(h)
        self.ev = []


class Batch:
    """One resident batch: ids and gradients on the device (and, for the
    merge workload, shard 0's own ids and gradients)."""

    def __init__(self, w, torch, dev, ids=None, grads=None, words=None):
        if w.samples:
            # sampled softmax: the shards' random words (sampled on the GPU
            # into the front of ids each step), then their batches' own words
            from paper_1810_10045_amd import seeding
            if words is None:
                words = w.sampler_words(seeding.seed_of_gpus(w.shards, w.seed_rule))
            self.words = torch.from_numpy(words.view(np.int64)).to(dev)
            true = w.ids() if ids is None else ids[w.shards * w.samples:]
            self.ids = torch.empty(w.tokens, dtype=torch.int32, device=dev)
            self.ids[w.shards * w.samples:] = torch.from_numpy(true).to(dev)
        else:
            self.ids = torch.from_numpy(w.ids() if ids is None else ids).to(dev)
        # bf16 arrives as its uint16 bit patterns, the oracle's very input
        g = w.grads() if grads is None else grads
        t = torch.from_numpy(g)
        self.grad = (t.view(torch.bfloat16) if w.grad_dtype == "bf16" else t).to(dev)
        del g, t
        if w.step in ("expand", "expand_f16"):
            self.ids0 = self.ids[:w.K]
            self.grad0 = self.grad[:w.K]


class Pipeline:
    """The timed step: device buffers for one workload and the calls of one
    pass of the hot path over resident batch b. The full-size parity tests
    drive this same class, so they check the launches that are timed here."""

    def __init__(self, w, batches, torch, lz, dev, table=None):
        self.w, self.batches, self.lz, self.torch = w, batches, lz, torch
        K, D = w.tokens, w.D
        idt = torch.int64 if w.id_dtype == "i64" else torch.int32
        self.ures = lz.unique_buffers(K, w.V, idt, dev)
        self.ws = lz.Workspace(dev)
        cap = self.ures.uniq.numel()
        self.out = torch.empty((cap, D), dtype=torch.float32, device=dev)
        self.dev_err = self.ures.dev_err
        self.state = {}
        st = self.state
        if w.step in ("sgd", "adam", "softmax_sgd"):
            st["table"] = torch.from_numpy(w.table() if table is None else table).to(dev)
        elif w.step == "scatter":
            st["table"] = torch.zeros((w.V, D), dtype=torch.float32, device=dev)
        if w.step == "adam":
            st["m"] = torch.zeros_like(st["table"])
            st["v"] = torch.zeros_like(st["table"])
        if w.step in ("expand", "expand_f16"):
            st["u0"] = lz.unique_buffers(w.K, w.V, idt, dev)
            st["out0"] = torch.empty((st["u0"].uniq.numel(), D), dtype=torch.float32, device=dev)
            mdt = torch.float16 if w.step == "expand_f16" else torch.float32
            st["M"] = torch.empty((cap, D), dtype=mdt, device=dev)
        self.sets = None
        # SCATTER into the dense table and SGD: Seg-Sum writes (or applies)
        # each type's row to its table row itself (lm_segsum_rows,
        # lm_segsum_sgd), unless `fused` is cleared (then lm_segsum into
        # `out`, and lm_fill_values SCATTER or lm_sparse_apply from there).
        self.fused = w.step in FUSED_STEPS
        self.last = None

    def reduce(self, bt, ures, err, t=1):
        """Seg-Sum of batch bt from Unique outputs ures: into `out`, or with
        `fused`, straight into the table rows of the types (SCATTER, SGD or
        Adam step t done)."""
        w, lz, st = self.w, self.lz, self.state
        self.last = (bt, ures, err)
        if self.fused and w.step == "scatter":
            lz.segsum_rows(bt.grad, ures.perm, ures.inverse, ures.offsets, ures.num_unique,
                           ures.uniq, st["table"], dev_err=err, ws=self.ws)
        elif self.fused and w.step == "adam":
            b1, b2, eps = w.adam
            lz.segsum_adam(bt.grad, ures.perm, ures.inverse, ures.offsets, ures.num_unique,
                           ures.uniq, st["table"], st["m"], st["v"], lr=w.lr, beta1=b1,
                           beta2=b2, eps=eps, step=t, dev_err=err, ws=self.ws)
        elif self.fused:
            lz.segsum_sgd(bt.grad, ures.perm, ures.inverse, ures.offsets, ures.num_unique,
                          ures.uniq, st["table"], w.lr, dev_err=err, ws=self.ws)
        else:
            lz.segsum(bt.grad, ures.perm, ures.inverse, ures.offsets, ures.num_unique,
                      out=self.out, dev_err=err, ws=self.ws)

    def reduced_rows(self, U):
        """The U reduced rows of the last step, in type order: from the table
        when the SCATTER was fused into Seg-Sum; with SGD fused, from the same
        call with lr = -1 on a zero table, where each row is 0 + 1 * sum,
        the sum itself; with Adam fused, from the same call with beta1 = 0
        on zero tables, where each m row is 0 * 0 + 1 * sum."""
        if self.fused and self.w.step == "scatter":
            return self.state["table"][self.ures.uniq[:U].long()]
        if self.fused and self.w.step == "adam":
            bt, ures, err = self.last
            p, m, v = (self.torch.zeros_like(self.state["table"]) for _ in range(3))
            self.lz.segsum_adam(bt.grad, ures.perm, ures.inverse, ures.offsets, ures.num_unique,
                                ures.uniq, p, m, v, lr=0.0, beta1=0.0, step=1, dev_err=err,
                                ws=self.ws)
            rows = m[ures.uniq[:U].long()]
            del p, m, v
            return rows
        if self.fused:
            bt, ures, err = self.last
            z = self.torch.zeros_like(self.state["table"])
            self.lz.segsum_sgd(bt.grad, ures.perm, ures.inverse, ures.offsets, ures.num_unique,
                               ures.uniq, z, -1.0, dev_err=err, ws=self.ws)
            rows = z[ures.uniq[:U].long()]
            del z
            return rows
        return self.out[:U]

    def enable_overlap(self, group=None):
        """2 x group sets of Unique outputs and a Unique workspace of their
        own, so that the Unique calls of later batches can run on a second
        stream while earlier batches' Seg-Sum and update run on the first
        (Unique reads only the token ids, which exist before the gradients
        do). The steps go in groups of `group` (run_overlapped): the Unique
        calls of one group fill one half of the sets while the other half's
        steps finish."""
        w, lz = self.w, self.lz
        group = OVERLAP_GROUP.get(w.name, OVERLAP_GROUP_DEFAULT) if group is None else group
        if group < 1:
            raise ValueError(f"a group holds at least one step, not {group}")
        dev = self.ures.uniq.device
        idt = self.ures.uniq.dtype
        self.ws_u = lz.Workspace(dev)
        self.ws_u.get(max(lz.unique_workspace_bytes(w.tokens, w.V, idt),
                          lz.unique_workspace_bytes(w.K, w.V, idt)))
        u0 = self.state.get("u0")
        self.sets = [(self.ures, u0)] + [
            (lz.unique_buffers(w.tokens, w.V, idt, dev),
             lz.unique_buffers(w.K, w.V, idt, dev) if u0 is not None else None)
            for _ in range(2 * group - 1)]

    def front(self, b, j, stream):
        """The part of step b that reads only ids, into output set j."""
        w, lz = self.w, self.lz
        bt = self.batches[b % len(self.batches)]
        ures, u0 = self.sets[j]
        if w.samples:
            lz.sample_ids(bt.words, w.V, out=bt.ids[:w.shards * w.samples], stream=stream)
        lz.unique(bt.ids, w.V, out=ures, ws=self.ws_u, stream=stream)
        if u0 is not None:
            lz.unique(bt.ids0, w.V, out=u0, ws=self.ws_u, stream=stream)

    def back(self, b, j):
        """The rest of step b on the current stream, from output set j."""
        w, lz, st = self.w, self.lz, self.state
        bt = self.batches[b % len(self.batches)]
        ures, u0 = self.sets[j]
        err = ures.dev_err
        self.reduce(bt, ures, err, 1 + b)
        if w.step in ("sgd", "softmax_sgd") and not self.fused:
            lz.sparse_apply(st["table"], ures.uniq, ures.num_unique, self.out, "sgd", lr=w.lr,
                            dev_err=err)
        elif w.step == "adam" and not self.fused:
            b1, b2, eps = w.adam
            lz.sparse_apply(st["table"], ures.uniq, ures.num_unique, self.out, "adam", lr=w.lr,
                            beta1=b1, beta2=b2, eps=eps, step=1 + b, m=st["m"], v=st["v"],
                            dev_err=err)
        elif w.step == "scatter" and not self.fused:
            lz.fill_values(self.out, ures.uniq, ures.num_unique, st["table"], None, None,
                           "scatter", dev_err=err)
        elif w.step in ("expand", "expand_f16"):
            lz.segsum(bt.grad0, u0.perm, u0.inverse, u0.offsets, u0.num_unique, out=st["out0"],
                      dev_err=err, ws=self.ws)
            if w.step == "expand":
                lz.fill_values(st["out0"], u0.uniq, u0.num_unique, st["M"], ures.uniq,
                               ures.num_unique, "expand", dev_err=err)
            else:
                lz.fill_values_f16(st["out0"], u0.uniq, u0.num_unique, st["M"], ures.uniq,
                                   ures.num_unique, "expand", scale=w.scale, dev_err=err)

    def check(self):
        for ures, _ in (self.sets or [(self.ures, None)]):
            self.lz.check(ures.dev_err)

    def run_overlapped(self, first, steps, torch, main, side, sync):
        """Steps first .. first + steps - 1 in groups of G = len(sets) / 2
        consecutive steps; step i uses set i % 2G. The Unique calls of group
        g run on `side`, one after another, then event 2g + 1 marks them
        done; `main` waits for that event once, runs the group's Seg-Sums and
        updates, and event 2g + 2 marks them done, which frees the group's
        half of the sets for group g + 2. So the side stream runs up to
        2G - 1 steps ahead, and the streams meet once per group, not once
        per step. Event 0 starts the side stream no earlier than what is
        already on `main`."""
        G = len(self.sets) // 2
        if G < 1 or len(self.sets) != 2 * G:
            raise ValueError(f"the grouped schedule takes an even number of sets, not {len(self.sets)}")
        ngroups = (steps + G - 1) // G

        def members(g):
            return range(g * G, min(steps, (g + 1) * G))

        def fronts(g):
            for i in members(g):
                self.front(first + i, i % (2 * G), side)
            sync.record(2 * g + 1, side)

        sync.record(0, main)
        sync.wait(0, side)
        if ngroups:
            fronts(0)
        for g in range(ngroups):
            if g + 1 < ngroups:
                if g >= 1:
                    sync.wait(2 * g, side)  # group g - 1 done: its sets are free
                fronts(g + 1)
            sync.wait(2 * g + 1, main)
            for i in members(g):
                self.back(first + i, i % (2 * G))
            sync.record(2 * g + 2, main)

    def step(self, b, ev=None):
        w, lz, st, ures, err = self.w, self.lz, self.state, self.ures, self.dev_err
        bt = self.batches[b % len(self.batches)]
        if ev: ev(0)
        if w.samples:
            lz.sample_ids(bt.words, w.V, out=bt.ids[:w.shards * w.samples])
        lz.unique(bt.ids, w.V, out=ures, ws=self.ws)
        if ev: ev(1)
        self.reduce(bt, ures, err, 1 + b)
        if ev: ev(2)
        if w.step in ("sgd", "softmax_sgd") and not self.fused:
            lz.sparse_apply(st["table"], ures.uniq, ures.num_unique, self.out, "sgd", lr=w.lr,
                            dev_err=err)
        elif w.step == "adam" and not self.fused:
            b1, b2, eps = w.adam
            lz.sparse_apply(st["table"], ures.uniq, ures.num_unique, self.out, "adam", lr=w.lr,
                            beta1=b1, beta2=b2, eps=eps, step=1 + b, m=st["m"], v=st["v"],
                            dev_err=err)
        elif w.step == "scatter" and not self.fused:
            lz.fill_values(self.out, ures.uniq, ures.num_unique, st["table"], None, None,
                           "scatter", dev_err=err)
        elif w.step in ("expand", "expand_f16"):
            u0 = st["u0"]
            lz.unique(bt.ids0, w.V, out=u0, ws=self.ws)
            lz.segsum(bt.grad0, u0.perm, u0.inverse, u0.offsets, u0.num_unique, out=st["out0"],
                      dev_err=err, ws=self.ws)
            if w.step == "expand":
                lz.fill_values(st["out0"], u0.uniq, u0.num_unique, st["M"], ures.uniq,
                               ures.num_unique, "expand", dev_err=err)
            else:
                lz.fill_values_f16(st["out0"], u0.uniq, u0.num_unique, st["M"], ures.uniq,
                                   ures.num_unique, "expand", scale=w.scale, dev_err=err)
        if ev: ev(3)


_SIDE_STREAM = []


def side_stream(torch, dev):
    """The overlapped schedule's second stream (default priority, like the
    first), created once per process and used by every workload: with a new
    stream per pass, about one pass in six ran with the two streams on one
    hardware queue (a process gets four), which serialises them (the word
    step at 160.8 us per step against 130.6)."""
    if not _SIDE_STREAM:
        _SIDE_STREAM.append(torch.cuda.Stream(device=dev))
    return _SIDE_STREAM[0]


# Steps per group of the overlapped schedule (run_overlapped), per
# workload. Each wait of one stream for the other's event leaves the
# waiting stream idle for a few microseconds, so the streams meet once per
# group of steps rather than once per step. Measured in one process against
# one meeting per step with four sets (us per step): the tiny workload 26.7
# -> 23.9 at groups of 8, the word step 109.9 -> 103.8, the 2M vocabulary
# 972 -> 965, the merge 1,472 -> 1,466; the char workload, on its CU split,
# 1,441 -> 1,434 at groups of 2 (1,439 at 8).
OVERLAP_GROUP_DEFAULT = 8
OVERLAP_GROUP = {"char_heavy_1m": 2}


# The overlapped schedule's CU split, per workload: the Unique calls run on
# CUs [0, n) and the rest of the step on the others (two streams created
# with CU masks), where that measured faster than two streams sharing every
# CU: char_heavy_1m 1,427 against 1,445 us per step. On a CU of its own, a
# Unique kernel that needs a whole CU (the 1024-thread sort tiles, the
# per-id counters in LDS) no longer waits for the walk's waves to leave
# one. The word step and the merge, whose Seg-Sums need every CU, measured
# slower split (133 -> 141 and 1,480 -> 1,500 us at 32 CUs), and so does
# the 2M vocabulary since its Seg-Sum applies Adam itself (967 -> 1,328 us
# at 64 CUs; with the separate apply it had gained, 1,118 -> 1,082).
SIDE_CUS = {"char_heavy_1m": 32}


def cu_mask_words(first, count, ncu):
    """hipExtStreamCreateWithCUMask's mask of CUs [first, first + count)
    as 32-bit words, bit c of the mask being CU c."""
    if count <= 0 or first < 0 or first + count > ncu:
        raise ValueError(f"CU range [{first}, {first + count}) outside the {ncu} CUs")
    words = [0] * ((ncu + 31) // 32)
    for c in range(first, first + count):
        words[c // 32] |= 1 << (c % 32)
    return words


class CuSplit:
    """Two streams on disjoint CUs: `side` on CUs [0, n), `main` on
    [n, N), both at the default priority. A mask of every eighth CU was
    refused (hipErrorOutOfMemory), as is one that leaves an XCD without a
    CU: the mask's bits interleave the 8 XCDs, so a contiguous range of 32*j
    bits takes 4*j CUs of each. Other range sizes measured slower for the
    Seg-Sum (its chunks are sized for whole rounds of waves, and an XCD
    with a CU count not a multiple of 4 finished its share late). Created
    for one pass and destroyed after it."""

    def __init__(self, torch, n):
        import ctypes
        self.ct, self.torch = ctypes, torch
        ncu = torch.cuda.get_device_properties(0).multi_processor_count
        if n % 32 or not 0 < n < ncu:
            raise ValueError(f"a CU split takes a multiple of 32 CUs below {ncu}, not {n}")
        hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch already loaded
        hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.c_void_p, ctypes.c_uint32,
                                                     ctypes.c_void_p]
        hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
        self.hip, self.handles = hip, []
        self.side = self._stream(cu_mask_words(0, n, ncu))
        self.main = self._stream(cu_mask_words(n, ncu - n, ncu))

    def _stream(self, words):
        ct = self.ct
        mask = (ct.c_uint32 * len(words))(*words)
        h = ct.c_void_p()
        rc = self.hip.hipExtStreamCreateWithCUMask(ct.byref(h), len(words), ct.byref(mask))
        if rc != 0:
            self.close()
            raise RuntimeError(f"hipExtStreamCreateWithCUMask failed ({rc})")
        self.handles.append(h)
        return self.torch.cuda.ExternalStream(h.value)

    def close(self):
        self.torch.cuda.synchronize()
        for h in self.handles:
            self.hip.hipStreamDestroy(h)
        self.handles = []


def run_overlap_pass(pipe, steps, warmup, torch, main, side):
    """Warm-up, then K timed steps of the overlapped schedule; ms in total."""
    sync = HipEvents(2 * max(steps, warmup) + 2, timing=False)
    ev = HipEvents(2)
    with torch.cuda.stream(main):
        pipe.run_overlapped(0, warmup, torch, main, side, sync)
        torch.cuda.synchronize()
        ev.record(0, main)
        pipe.run_overlapped(0, steps, torch, main, side, sync)
        ev.record(1, main)
        torch.cuda.synchronize()
    pipe.check()
    ms = ev.ms(0, 1)
    ev.close()
    sync.close()
    return ms


class HostInputs:
    """Batch 0 of a workload on the host: the arrays copied to the GPU and
    handed to the CPU oracle, so both sides see the very same values."""

    def __init__(self, w):
        self.words = None
        if w.samples:
            from paper_1810_10045_amd import seeding
            self.words = w.sampler_words(seeding.seed_of_gpus(w.shards, w.seed_rule))
        self.true_ids = w.ids()
        self.grads = w.grads()      # storage dtype (bf16 as uint16 bits)
        self.table = w.table() if w.step in ("sgd", "adam", "softmax_sgd") else None

    def oracle_ids(self, w, oracle):
        if self.words is None:
            return self.true_ids
        return np.concatenate([oracle.sample_ids(self.words, w.V), self.true_ids])


def run_gpu(w, steps, warmup, nbatch, torch, lz, host):
    """The three timed passes of one workload (serial; serial with an event
    around each entry point; overlapped), then one more step over batch 0
    whose Unique and Seg-Sum outputs are returned for the oracle check."""
    dev = torch.device("cuda:0")
    log(f"workload {w.name}: K={w.tokens} V={w.V} D={w.D} s={w.s} {w.grad_dtype}/{w.id_dtype} "
        f"step={w.step}, {nbatch} resident batches")
    t0 = time.time()
    batches = [Batch(w, torch, dev, ids=None if w.samples else host.true_ids, grads=host.grads,
                     words=host.words)]
    batches += [Batch(w.batch(b), torch, dev) for b in range(1, nbatch)]
    log(f"inputs generated and copied in {time.time() - t0:.1f}s")
    K, D = w.tokens, w.D
    pipe = Pipeline(w, batches, torch, lz, dev, table=host.table)
    ures, dev_err, step = pipe.ures, pipe.dev_err, pipe.step
    stream = torch.cuda.current_stream()

    # Types per batch (read once, outside the timed region).
    U_of = []
    for b in range(nbatch):
        step(b)
        torch.cuda.synchronize()
        U_of.append(int(ures.num_unique.item()))
    lz.check(dev_err)
    log(f"types per batch: {U_of}")
    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()

    # Pass 1, the serial schedule: K steps between two events and nothing
    # else on the stream (an event record costs the GPU a few microseconds).
    ev = HipEvents(2)
    torch.cuda.synchronize()
    ev.record(0, stream)
    for i in range(steps):
        step(i)
    ev.record(1, stream)
    torch.cuda.synchronize()
    lz.check(dev_err)
    total_ms = ev.ms(0, 1)
    ev.close()
    # Pass 2, the same K steps with an event around every entry point: the
    # per-stage times and the Seg-Sum launch time of the roofline.
    ev = HipEvents(4 * steps)
    torch.cuda.synchronize()
    for i in range(steps):
        step(i, lambda k, i=i: ev.record(4 * i + k, stream))
    torch.cuda.synchronize()
    lz.check(dev_err)
    st = np.array([[ev.ms(4 * i, 4 * i + 1), ev.ms(4 * i + 1, 4 * i + 2), ev.ms(4 * i + 2, 4 * i + 3)]
                   for i in range(steps)])
    ev.close()
    unfused = None
    if pipe.fused:
        # For comparison, passes 1 and 2 again with the SCATTER as its own
        # call after lm_segsum (the stage the fused call replaces).
        pipe.fused = False
        for i in range(warmup):
            step(i)
        ev = HipEvents(2 + 4 * steps)
        torch.cuda.synchronize()
        ev.record(0, stream)
        for i in range(steps):
            step(i)
        ev.record(1, stream)
        torch.cuda.synchronize()
        for i in range(steps):
            step(i, lambda k, i=i: ev.record(2 + 4 * i + k, stream))
        torch.cuda.synchronize()
        lz.check(dev_err)
        ust = np.array([[ev.ms(2 + 4 * i + k, 2 + 4 * i + k + 1) for k in range(3)]
                        for i in range(steps)])
        unfused = dict(serial_ms=ev.ms(0, 1), stage_ms=ust.mean(axis=0).tolist())
        ev.close()
        pipe.fused = True
    # Pass 3, the headline: the same K steps with the Unique calls on a
    # second stream (default priority, like the first), running ahead in
    # groups of steps; at the workloads of SIDE_CUS with the two streams on
    # disjoint CUs (and, for comparison, both on every CU).
    pipe.enable_overlap()
    group = len(pipe.sets) // 2
    overlap_ms = overlap_all_ms = run_overlap_pass(pipe, steps, warmup, torch, stream,
                                                   side_stream(torch, dev))
    side_cus = SIDE_CUS.get(w.name)
    if side_cus:
        try:
            split = CuSplit(torch, side_cus)
        except (RuntimeError, ValueError) as e:
            # no CU-masked streams here: the line keeps the shared-CU figure
            log(f"{w.name}: no CU split ({e}); the overlapped figure is the shared-CU one")
            side_cus = None
        else:
            try:
                overlap_ms = run_overlap_pass(pipe, steps, warmup, torch, split.main, split.side)
            finally:
                split.close()
    # One more serial step over batch 0: the outputs the oracle checks.
    step(0)
    torch.cuda.synchronize()
    lz.check(dev_err)
    U0 = int(ures.num_unique.item())
    outputs = dict(U=U0, uniq=ures.uniq[:U0].cpu().numpy().astype(np.int64),
                   counts=ures.counts[:U0].cpu().numpy(), offsets=ures.offsets[:U0 + 1].cpu().numpy(),
                   inverse=ures.inverse[:K].cpu().numpy(), perm=ures.perm[:K].cpu().numpy(),
                   out=pipe.reduced_rows(U0).cpu().numpy())
    fused = pipe.fused
    del pipe, batches
    torch.cuda.empty_cache()
    gb = 2 if w.grad_dtype == "bf16" else 4
    ib = 8 if w.id_dtype == "i64" else 4
    Us = [U_of[i % nbatch] for i in range(steps)]
    # the fused call also reads the U row ids (and with SGD the table rows)
    seg_bytes = np.mean([segsum_bytes(K, D, U, gb) + (fused_extra_bytes(w, D, U, ib) if fused else 0)
                         for U in Us])
    seg_ms = float(st[:, 1].mean())
    uniq_bytes = float(np.mean([unique_bytes(K, U, ib) for U in Us]))
    rows = AFTER_ROWS.get(w.step)
    after_bytes = float(np.mean([rows * U * D * 4 for U in Us])) if rows else None
    if unfused:
        ub = float(np.mean([segsum_bytes(K, D, U, gb) for U in Us]))
        unfused.update(seg_bytes=ub, seg_gbps=ub / (unfused["stage_ms"][1] / 1e3) / 1e9,
                       ms_per_step=unfused["serial_ms"] / steps,
                       value=K / (unfused["serial_ms"] / steps / 1e3))
    return dict(total_ms=total_ms, overlap_ms=overlap_ms, overlap_all_ms=overlap_all_ms,
                side_cus=side_cus, group=group, stage_ms=st.mean(axis=0).tolist(), seg_ms=seg_ms,
                seg_bytes=float(seg_bytes), uniq_bytes=uniq_bytes, after_bytes=after_bytes,
                U=U_of, outputs=outputs, fused=fused, unfused=unfused)


def host_threads() -> int:
    """Threads of the all-core oracle leg: the cores this process may run on,
    at most 16 (a one-GPU share of the host)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def oracle_pass(w, oracle, ids, host, threads):
    """One whole step of the oracle over batch 0: unique, then segsum and the
    stage after it, on one thread (threads = 1) or with the columns of the
    reduction and the rows of the update split over `threads` threads (the
    unique stays on one thread). Returns the unique outputs and the sums."""
    grads = host.grads
    uniq, counts, offsets, inverse, perm = oracle.unique(ids, w.V)
    U = len(uniq)
    if threads == 1:
        red = oracle.segsum(grads, inverse, U)
    else:
        red = oracle.segsum_threads(grads, inverse, U, threads)
    if w.step in ("sgd", "softmax_sgd"):
        p = host.table[uniq]
        (oracle.sgd(p, red, w.lr) if threads == 1 else oracle.sgd_threads(p, red, w.lr, threads))
    elif w.step == "adam":
        p, z = host.table[uniq], np.zeros((U, w.D))
        if threads == 1:
            oracle.adam(p, z, z, red, w.lr, *w.adam, 0.0, 1)
        else:
            oracle.adam_threads(p, z, z, red, w.lr, *w.adam, 0.0, 1, threads)
    elif w.step == "scatter":
        dense = np.zeros((w.V, w.D))
        (oracle.scatter(red, uniq, dense) if threads == 1
         else oracle.scatter_threads(red, uniq, dense, threads))
    return (uniq, counts, offsets, inverse, perm), red


def run_cpu_baseline(w, host, budget_s):
    """The CPU oracle as it stands on whole copies of batch 0, until about
    budget_s seconds of work are done (at least one pass), in two legs: one
    thread, and every core of the process (the reduction's columns and the
    update's rows split over the threads). Returns both legs and the first
    pass's outputs."""
    import oracle
    ids = host.oracle_ids(w, oracle)
    legs, first = {}, None
    for threads in (1, host_threads()):
        done, t_used = 0, 0.0
        while t_used < budget_s and done < 1000:
            t0 = time.perf_counter()
            res = oracle_pass(w, oracle, ids, host, threads)
            t_used += time.perf_counter() - t0
            done += 1
            if first is None:
                first = res
            del res
        what = ("1 thread" if threads == 1 else
                f"{threads} threads (unique on one; the reduction's columns and the update's rows "
                f"split over the threads)")
        legs[threads] = dict(value=done * len(ids) / t_used, unit="tokens/s", cores=threads,
                             kind="oracle",
                             sample=f"{done} whole {w.name} batch(es) of {len(ids)} tokens, "
                                    f"unique+segsum+{w.step}, fp64, {what} of {cpu_model()}, "
                                    f"{t_used:.1f}s")
    return legs, first, ids


def check_outputs(w, gpu, ora):
    """The timed kernels' outputs for batch 0 against the oracle's: every
    integer output of Unique bit for bit, and every Seg-Sum row within the
    per-row normwise tolerance of its gradient dtype (with count-1 rows
    exact)."""
    (uniq, counts, offsets, inverse, perm), red = ora
    ok_int = (gpu["U"] == len(uniq) and np.array_equal(gpu["uniq"], uniq)
              and np.array_equal(gpu["counts"], counts) and np.array_equal(gpu["offsets"], offsets)
              and np.array_equal(gpu["inverse"], inverse) and np.array_equal(gpu["perm"], perm))
    err, ones_exact = None, False
    if ok_int:
        got = gpu["out"].astype(np.float64)
        scale = np.abs(red).max(axis=1)
        diff = np.abs(got - red).max(axis=1)
        nz = scale > 0
        err = float((diff[nz] / scale[nz]).max()) if nz.any() else 0.0
        if not np.all(diff[~nz] == 0):
            err = float("inf")
        single = counts == 1
        ones_exact = bool(np.array_equal(got[single], red[single]))
    tol = 2e-3 if w.grad_dtype == "bf16" else 1e-5
    ok = bool(ok_int and err is not None and err <= tol and ones_exact)
    return {"ok": ok, "unique_bit_exact": bool(ok_int), "segsum_rows": int(len(red)),
            "segsum_max_row_rel_err": err, "tolerance": tol, "count1_rows_exact": ones_exact}


def cpu_model() -> str:
    """The host CPU's model name (and how many cores the host has)."""
    name = "unknown CPU"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{name} ({os.cpu_count()} cores)"


def load_traffic(workload):
    """HBM bytes per lm_segsum call (all its kernels) from the committed
    rocprofv3 counter summary (FETCH_SIZE + WRITE_SIZE, scaled by a plain
    copy), only while the Seg-Sum sources are unchanged since the counters
    were taken."""
    path = TRAFFIC_FILE.format(workload=workload)
    if not os.path.exists(path):
        return None
    rec = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].strip().split(": ", 1)
                rec[k.strip("`")] = v.strip("`")
    if rec.get("segsum_sources_sha256_16") != segsum_source_hash():
        return None
    try:
        return float(rec["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_calibration(torch, reps=3):
    """Plain device copies of COPY_BYTES (read COPY_BYTES, write COPY_BYTES)
    whose counter readings scale FETCH_SIZE / WRITE_SIZE to bytes."""
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: {reps} copies of {COPY_BYTES} bytes")
    del src, dst
    torch.cuda.empty_cache()


def segsum_kernels(w, fused=False):
    """The kernels of one lm_segsum (or, fused with SCATTER, SGD or Adam,
    lm_segsum_rows, lm_segsum_sgd or lm_segsum_adam) call at this workload's
    shape (rows of up to 4096 columns on the 16-byte path: one launch)."""
    name = ("lm_segsum" if not fused else "lm_segsum_rows" if w.step == "scatter" else
            "lm_segsum_adam" if w.step == "adam" else "lm_segsum_sgd")
    k = (SEGSUM_KERNELS if w.D <= 4096 else "lm_segsum (k_segsum walk, then k_segsum_fix)")
    k = k.replace("lm_segsum", name, 1)
    if not fused:
        return k
    return k + (", each type row written to its table row" if w.step == "scatter" else
                ", each type row applied to its table row (Adam, with its m and v rows)"
                if w.step == "adam" else ", each type row applied to its table row (SGD)")


def stages(w, r):
    """Per-stage ms of the event pass, named for what each stage runs."""
    ms = r["stage_ms"]
    if r["fused"]:
        return {"unique": ms[0], fused_stage(w): ms[1]}
    return {"unique": ms[0], "segsum": ms[1], w.step: ms[2]}


def unfused_entry(w, r):
    """The same workload with the SCATTER or SGD update as its own call after
    lm_segsum."""
    u = r["unfused"]
    if not u:
        return None
    then = {"scatter": "lm_fill_values SCATTER", "adam": "lm_sparse_apply Adam"}.get(
        w.step, "lm_sparse_apply SGD")
    return {"value": u["value"], "ms_per_step": u["ms_per_step"],
            "stages_ms": {"unique": u["stage_ms"][0], "segsum": u["stage_ms"][1],
                          w.step: u["stage_ms"][2]},
            "segsum_gbps": u["seg_gbps"], "segsum_frac": u["seg_gbps"] / HBM_PEAK_GBPS,
            "schedule": f"one stream; lm_segsum into a U x D buffer, then {then}"}


def measure(w, args, torch, lz, cpu_budget):
    """Everything the bench reports for one workload."""
    gb = 2 if w.grad_dtype == "bf16" else 4
    nbatch = args.batches or max(1, min(8, math.ceil((2 << 30) / (w.tokens * w.D * gb))))
    t0 = time.time()
    host = HostInputs(w)
    log(f"{w.name}: batch 0 generated on the host in {time.time() - t0:.1f}s")
    r = run_gpu(w, args.steps, args.warmup, nbatch, torch, lz, host)
    ms = r["overlap_ms"] / args.steps
    serial_ms = r["total_ms"] / args.steps
    achieved = r["seg_bytes"] / (r["seg_ms"] / 1e3) / 1e9
    res = dict(w=w, nbatch=nbatch, r=r, ms=ms, serial_ms=serial_ms, achieved=achieved, steps=args.steps,
               value=w.tokens / (ms / 1e3), traffic=load_traffic(w.name), cpu=None, check=None)
    if not args.no_cpu:
        t0 = time.time()
        legs, ora, _ = run_cpu_baseline(w, host, cpu_budget)
        res["cpu"] = legs
        res["check"] = check_outputs(w, r["outputs"], ora)
        log(f"{w.name}: oracle legs and check in {time.time() - t0:.1f}s: "
            f"{legs[1]['value']:.3g} / {legs[max(legs)]['value']:.3g} tokens/s; "
            f"check {res['check']}")
        del ora
    del host, r["outputs"]
    return res


def schedule_text(r):
    """The overlapped schedule the headline figure was measured with."""
    g = r["group"]
    t = (f"unique on a second stream, in groups of {g} steps ({2 * g} sets of its outputs): "
         f"the streams meet once per group, the second up to {2 * g - 1} steps ahead")
    n = r["side_cus"]
    if n:
        t += f"; the second stream on CUs 0-{n - 1}, the first on the others (CU-masked streams)"
    return t


def all_cus_entry(res):
    """With a CU split: the same overlapped schedule with both streams on
    every CU, for comparison."""
    r = res["r"]
    if not r["side_cus"]:
        return None
    ms = r["overlap_all_ms"] / res["steps"]
    return {"value": res["w"].tokens / (ms / 1e3), "ms_per_step": ms,
            "schedule": "the same, both streams on every CU"}


def cpu_baseline_entry(res):
    """The cpu_baseline object: the all-core leg, with the one-thread leg and
    the GPU/CPU ratios beside it."""
    legs = res["cpu"]
    if not legs:
        return None
    allc = legs[max(legs)]
    one = legs[1]
    return {**allc, "one_thread": one,
            "gpu_over_cpu": {"all_cores": res["value"] / allc["value"],
                             "one_thread": res["value"] / one["value"]}}


def workload_summary(res):
    """One workload's figures for the per-workload table of the line."""
    w, r = res["w"], res["r"]
    legs = res["cpu"] or {}
    return {
        "tokens": w.tokens, "V": w.V, "D": w.D, "zipf_s": w.s, "ids": w.id_dtype,
        "grad": w.grad_dtype, "after_segsum": w.step, "resident_batches": res["nbatch"],
        "types_batch0": r["U"][0],
        "value": res["value"], "ms_per_step": res["ms"], "schedule": schedule_text(r),
        "overlapped_all_cus": all_cus_entry(res),
        "serial_value": w.tokens / (res["serial_ms"] / 1e3), "serial_ms_per_step": res["serial_ms"],
        "stages_ms": stages(w, r),
        "segsum": {"kernels": segsum_kernels(w, r["fused"]), "achieved_gbps": res["achieved"],
                   "frac": res["achieved"] / HBM_PEAK_GBPS, "bytes_per_launch": r["seg_bytes"],
                   "avg_launch_ms": r["seg_ms"], "traffic": res["traffic"]},
        "cpu_tokens_per_s": {str(k): v["value"] for k, v in legs.items()},
        "gpu_over_cpu_all_cores": (res["value"] / legs[max(legs)]["value"]) if legs else None,
        "oracle_check": res["check"],
        "unfused_serial": unfused_entry(w, r),
    }


FIVE = ("word_tiny_8k", "word_step_64k", "merge_64x32k_bf16", "char_heavy_1m", "vocab2m_adam_i64")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="char_heavy_1m",
                    help="the headline workload (default: char_heavy_1m, the largest fp32 one)")
    ap.add_argument("--workloads", default=",".join(FIVE),
                    help="workloads measured after the headline for the per-workload table "
                         "(comma-separated; 'none' for the headline alone)")
    ap.add_argument("--batches", type=int, default=0, help="resident batches (0: auto)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle time per leg for the headline (other workloads: at most 3 s)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle legs and check")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run plain 1 GiB copies (scale for HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library does not implement the multi-GPU "
              "collectives of the method (the all-gather of the ids and the all-reduce of the "
              "reduced rows); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_1810_10045_amd import lmzipf as lz
    from paper_1810_10045_amd import synth

    side_stream(torch, torch.device("cuda:0"))  # the process's first stream
    if args.copy_calibration:
        copy_calibration(torch)
    w = synth.WORKLOADS[args.workload]
    head = measure(w, args, torch, lz, args.cpu_seconds)
    others = [] if args.workloads == "none" else [n for n in args.workloads.split(",") if n]
    table = {}
    for name in others:
        if name == w.name:
            table[name] = workload_summary(head)
            continue
        table[name] = workload_summary(measure(synth.WORKLOADS[name], args, torch, lz,
                                               min(args.cpu_seconds, 3.0)))
    r = head["r"]
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.grad_dtype == "f32" else "bf16->f32",
        "data": "synthetic",
        "config": {"workload": w.name, "tokens": w.tokens, "V": w.V, "D": w.D, "zipf_s": w.s,
                   "ids": w.id_dtype, "grad": w.grad_dtype, "after_segsum": w.step,
                   **({"gpus_simulated": w.shards, "samples_per_gpu": w.samples,
                       "seed_rule": w.seed_rule} if w.samples else {}),
                   "resident_batches": head["nbatch"], "types_per_batch": r["U"]},
        "stages_ms": stages(w, r),
        # algorithmic bytes of each stage / its event-measured time (GB/s)
        "stages_gbps": ({"unique": r["uniq_bytes"] / (r["stage_ms"][0] / 1e3) / 1e9,
                         fused_stage(w): head["achieved"]} if r["fused"] else
                        {"unique": r["uniq_bytes"] / (r["stage_ms"][0] / 1e3) / 1e9,
                         "segsum": head["achieved"],
                         w.step: (r["after_bytes"] / (r["stage_ms"][2] / 1e3) / 1e9
                                  if r["after_bytes"] else None)}),
        "roofline": {"bound": "hbm", "kernel": segsum_kernels(w, r["fused"]),
                     "achieved": head["achieved"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": head["achieved"] / HBM_PEAK_GBPS,
                     "bytes_per_launch": r["seg_bytes"], "avg_launch_ms": r["seg_ms"],
                     "traffic": head["traffic"]},
        "cpu_baseline": cpu_baseline_entry(head),
        "oracle_check": head["check"],
        "schedule": schedule_text(r),
        "overlapped_all_cus": all_cus_entry(head),
        "serial": {"value": w.tokens / (head["serial_ms"] / 1e3), "ms_per_step": head["serial_ms"],
                   "schedule": "one stream, the steps one after another"},
        "unfused_serial": unfused_entry(w, r),
        "workloads": table,
    }
    print(json.dumps(line), flush=True)
    checks = [head["check"]] + [t["oracle_check"] for t in table.values()]
    if any(c is not None and not c["ok"] for c in checks):
        log("the GPU outputs differ from the oracle's (oracle_check): see the line")
        sys.exit(1)


if __name__ == "__main__":
    main()
