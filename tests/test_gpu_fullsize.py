"""GPU parity at the full sizes of the five synthetic workloads, through the
very launches that bench.py times (its Batch and Pipeline, batch 0).

* Unique: every integer output bit-exact against the oracle, whole input.
* Seg-Sum: every row against the oracle's fp64 sums (the oracle's column
  split over the host's cores for the largest inputs), within the contract
  for the gradient dtype and within the fp32 accumulation bound for bf16
  inputs too; rows of types with one token must be exact copies.
* Map J^ -> I^ at the merge's real shape (shard 0's types into the merged
  list), bit-exact.
* What follows Seg-Sum, end to end from the oracle's own sums: SCATTER into a
  dense table, done by Seg-Sum's own writes (lm_segsum_rows; against the
  dense per-token scatter-add for the 100K x 512 case), SGD, applied by
  Seg-Sum itself (lm_segsum_sgd; its sums read back from the same call with
  lr = -1 on a zero table), the first lazy-Adam step (moments too, every touched row),
  EXPAND of shard 0 into the merged type list; rows the step must not touch
  are compared exactly.
"""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import gpu_helpers as H  # noqa: E402
import oracle  # noqa: E402
from paper_1810_10045_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

# Host threads for the oracle's column-split Seg-Sum (at most the 16 cores a
# one-GPU share of the host has).
THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module")
def lz():
    from paper_1810_10045_amd import lmzipf
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return lmzipf


def _say(msg):
    print(msg, flush=True)


def _f32(x):
    return float(np.float32(x))


def _run(lz, w, ids, grads, table=None):
    """One bench step over batch 0 of workload w (inputs given as host arrays)."""
    import bench
    dev = torch.device("cuda:0")
    _say(f"[fullsize] {w.name}: K={w.tokens} V={w.V} D={w.D} {w.grad_dtype}/{w.id_dtype} {w.step}")
    pipe = bench.Pipeline(w, [bench.Batch(w, torch, dev, ids=ids, grads=grads)], torch, lz, dev,
                          table=table)
    pipe.step(0)
    torch.cuda.synchronize()
    lz.check(pipe.dev_err)
    return pipe


def _release(pipe):
    del pipe
    torch.cuda.empty_cache()


def test_full_word_tiny_8k(lz):
    """8,192 tokens over 100K words, D = 512: Seg-Sum with the SCATTER into
    the dense V x 512 table in the same call (lm_segsum_rows), every written
    row against the oracle's Seg-Sum and the whole table against the
    per-token scatter-add."""
    w = synth.WORKLOADS["word_tiny_8k"]
    ids, g = w.ids(), w.grads()
    pipe = _run(lz, w, ids, g)
    o = H.assert_unique_matches(pipe.ures, ids, w.V, oracle, w.name)
    U = len(o[0])
    S = oracle.segsum(g, o[3], U)
    sq = H.sum_of_squares(g, o[3], U, oracle)
    got = pipe.reduced_rows(U).cpu().numpy()
    H.check_rows(got, S, sq)
    H.assert_single_rows_exact(got, S, o[1])
    dense = oracle.dense_scatter(g, ids, w.V)
    T = pipe.state["table"].cpu().numpy()
    others = np.ones(w.V, bool)
    others[o[0]] = False
    assert np.array_equal(T[others], dense[others]) and not T[others].any()
    assert H.row_rel_err(T[o[0]], dense[o[0]], sq) <= H.TOL_F32
    _release(pipe)


@pytest.mark.parametrize("name", ["word_step_64k", "word_step_64k_perm"])
def test_full_word_step_64k(lz, name):
    """The per-GPU word-LM step: 65,536 tokens over 800K words, D = 1024,
    every Seg-Sum row, then SGD (lr 0.1) into the 800K x 1024 table; also
    with the word ranks permuted over the vocabulary."""
    w = synth.WORKLOADS[name]
    ids, g, table0 = w.ids(), w.grads(), w.table()
    pipe = _run(lz, w, ids, g, table0)
    o = H.assert_unique_matches(pipe.ures, ids, w.V, oracle, w.name)
    U = len(o[0])
    S = oracle.segsum(g, o[3], U)
    sq = H.sum_of_squares(g, o[3], U, oracle)
    got = pipe.reduced_rows(U).cpu().numpy()
    H.check_rows(got, S, sq)
    H.assert_single_rows_exact(got, S, o[1])
    lr = _f32(w.lr)
    ref = oracle.sgd(table0[o[0]], S, lr)
    table = pipe.state["table"]
    rows_t = torch.from_numpy(o[0]).to(table.device)
    H.assert_sgd_rows(table[rows_t].cpu().numpy(), ref, S, lr, H.row_delta(S, H.TOL_F32, sq))
    others = torch.ones(w.V, dtype=torch.bool, device=table.device)
    others[rows_t] = False
    t0 = torch.from_numpy(table0).to(table.device)
    assert torch.equal(table[others], t0[others]), "untouched rows must be bit-unchanged"
    del t0
    _release(pipe)


@pytest.mark.parametrize("name", ["merge_64x32k_bf16", "merge_64x32k_f16"])
def test_full_merge_64x32k_bf16(lz, name):
    """64 concatenated shards of 32,768 tokens (2,097,152), bf16 gradients:
    Unique of the concatenation and of shard 0, every Seg-Sum row of the
    concatenation (326K types) and of shard 0, the map of shard 0's types
    into the merged list (lm_map_ids) and the EXPAND of shard 0's rows into
    it, as fp32 or as the binary16 payload of Sec. III-C (F = 64). With
    1024 columns a row's largest |sum| always exceeds the rms of its
    summands, so the rows are scaled by their largest entry alone."""
    w = synth.WORKLOADS[name]
    ids, g = w.ids(), w.grads()
    pipe = _run(lz, w, ids, g)
    o = H.assert_unique_matches(pipe.ures, ids, w.V, oracle, w.name)
    UG = len(o[0])
    S = oracle.segsum_threads(g, o[3], UG, THREADS)
    got = pipe.reduced_rows(UG).cpu().numpy()
    H.check_rows(got, S, None, w.grad_dtype, "merged rows")
    H.assert_single_rows_exact(got, S, o[1], "merged rows")
    del S, got
    # shard 0: steps 1-2 on its own tokens, step 4's map, step 5 into the
    # merged rows
    ids0, g0 = ids[:w.K], g[:w.K]
    u0 = pipe.state["u0"]
    o0 = H.assert_unique_matches(u0, ids0, w.V, oracle, w.name + " shard 0")
    U0 = len(o0[0])
    S0 = oracle.segsum(g0, o0[3], U0)
    sq0 = H.sum_of_squares(g0, o0[3], U0, oracle)
    got0 = pipe.state["out0"][:U0].cpu().numpy()
    H.check_rows(got0, S0, sq0, w.grad_dtype, "shard 0 rows")
    H.assert_single_rows_exact(got0, S0, o0[1], "shard 0 rows")
    mp, missing = oracle.map_ids(o0[0], o[0])
    assert not missing
    gmap = lz.map_ids(u0.uniq, u0.num_unique, pipe.ures.uniq, pipe.ures.num_unique,
                      dev_err=pipe.dev_err)
    torch.cuda.synchronize()
    lz.check(pipe.dev_err)
    assert np.array_equal(gmap[:U0].cpu().numpy(), mp), "lm_map_ids at the merge's shape"
    want = oracle.expand(S0, o0[0], o[0])
    others = np.ones(UG, bool)
    others[mp] = False
    if w.step == "expand":
        M = pipe.state["M"][:UG].cpu().numpy()
        assert not M[others].any() and not want[others].any(), "EXPAND must zero the other rows"
        H.check_rows(M[mp], want[mp], sq0, w.grad_dtype, "EXPAND rows")
    else:
        # The payload codes from the GPU's fp32 sums against the oracle's
        # compression of its fp64 sums: a code may sit one binary16 step away.
        F = w.scale
        got = pipe.state["M"][:UG].view(torch.int16).cpu().numpy().view(np.uint16)
        assert not got[others].any(), "EXPAND must zero the other rows"
        dg = oracle.decompress(got[mp], 1.0 / F)
        dr = oracle.decompress(oracle.compress(want[mp], F), 1.0 / F)
        delta = H.row_delta(S0, H.TOL_F32, sq0)
        bound = delta[:, None] + 2.0 ** -10 * np.abs(dr) + 2.0 ** -24 / F
        assert np.all(np.abs(dg - dr) <= bound)
    _release(pipe)


def test_full_char_heavy_1m(lz):
    """1,048,576 tokens over 20K characters (Zipf 1.2, the top type holds
    about a fifth of the tokens), D = 2048: every Seg-Sum row, written into
    the dense 20K x 2048 table by the same call (lm_segsum_rows). No floor on the row scale here: with
    2048 columns the largest |sum| always exceeds the rms of the summands."""
    w = synth.WORKLOADS["char_heavy_1m"]
    ids, g = w.ids(), w.grads()
    pipe = _run(lz, w, ids, g)
    o = H.assert_unique_matches(pipe.ures, ids, w.V, oracle, w.name)
    U = len(o[0])
    S = oracle.segsum_threads(g, o[3], U, THREADS)
    got = pipe.reduced_rows(U).cpu().numpy()
    H.check_rows(got, S)
    H.assert_single_rows_exact(got, S, o[1])
    T = pipe.state["table"].cpu().numpy()
    others = np.ones(w.V, bool)
    others[o[0]] = False
    assert not T[others].any()
    assert H.row_rel_err(T[o[0]], S) <= H.TOL_F32
    _release(pipe)


def test_full_vocab2m_adam_i64(lz):
    """262,144 int64 ids over a 2M vocabulary (Zipf 0.9), D = 1024: every
    Seg-Sum row, then the first lazy-Adam step (beta1 0.9, beta2 0.999,
    eps 1e-8, lr 1e-3, zero moments) on every touched row of the 2M x 1024
    param, m and v tables; every untouched row is compared exactly."""
    w = synth.WORKLOADS["vocab2m_adam_i64"]
    ids, g, table0 = w.ids(), w.grads(), w.table()
    pipe = _run(lz, w, ids, g, table0)
    o = H.assert_unique_matches(pipe.ures, ids, w.V, oracle, w.name)
    U = len(o[0])
    S = oracle.segsum_threads(g, o[3], U, THREADS)
    got = pipe.reduced_rows(U).cpu().numpy()
    H.check_rows(got, S)
    H.assert_single_rows_exact(got, S, o[1])
    del got
    sel = o[0]
    lr, (b1, b2, eps) = _f32(w.lr), (_f32(x) for x in w.adam)
    z = np.zeros_like(S)
    rp, rm, rv = oracle.adam_threads(table0[sel], z, z, S, lr, b1, b2, eps, 0.0, 1, THREADS)
    del z
    dev = pipe.out.device
    sel_t = torch.from_numpy(sel).to(dev)
    st = pipe.state
    H.assert_adam_first_step(st["table"][sel_t].cpu().numpy(), st["m"][sel_t].cpu().numpy(),
                             st["v"][sel_t].cpu().numpy(), rp, rm, rv, S, lr, b1, b2, eps,
                             H.row_delta(S, H.TOL_F32))
    del rp, rm, rv
    others = torch.ones(w.V, dtype=torch.bool, device=dev)
    others[sel_t] = False
    t0 = torch.from_numpy(table0).to(dev)
    assert torch.equal(st["table"][others], t0[others]), "untouched rows must be bit-unchanged"
    del t0
    assert int(torch.count_nonzero(st["m"][others])) == 0
    assert int(torch.count_nonzero(st["v"][others])) == 0
    _release(pipe)


# Sec. III-B at G = 64 GPUs, restated here rather than taken from the
# package: the number of sampler seeds of each rule (ceil of the rule's
# value, at least one), and GPU g of G using seed j when g lies in
# [ceil(j G / n), ceil((j + 1) G / n)) -- n contiguous groups of equal size
# to within one.
SEEDS_AT_64 = {"G": 64, "pow0.64": 15, "log2": 6, "ln": 5, "log10": 2, "one": 1}


def _seed_table(G, n):
    bounds = [-(-j * G // n) for j in range(n + 1)]
    return [j for j in range(n) for _ in range(bounds[j], bounds[j + 1])]


@pytest.mark.parametrize("rule", list(SEEDS_AT_64))
def test_full_sampled_softmax(lz, rule):
    """The output embedding under sampled softmax (Sec. III-B) for 64 GPUs on
    one GPU: each samples 1024 candidates from 800K words with its group's
    seed and adds its 640 batch words; the GPU's sampled ids equal the
    oracle's sampler on the same random words, then Unique, every Seg-Sum
    row (D = 512) and the SGD update are checked as for the word step. The
    seed of each GPU comes from the table above, for every rule."""
    w = synth.WORKLOADS["sampled_softmax_64x1024_" + rule]
    seeds = _seed_table(w.shards, SEEDS_AT_64[rule])
    assert len(seeds) == w.shards and len(set(seeds)) == SEEDS_AT_64[rule]
    words = w.sampler_words(seeds)
    ids = np.concatenate([oracle.sample_ids(words, w.V).astype(np.int32), w.ids()])
    g, table0 = w.grads(), w.table()
    import bench
    dev = torch.device("cuda:0")
    _say(f"[fullsize] {w.name}: {w.tokens} rows, {SEEDS_AT_64[rule]} seeds")
    pipe = bench.Pipeline(w, [bench.Batch(w, torch, dev, ids=ids, grads=g, words=words)], torch,
                          lz, dev, table=table0)
    pipe.step(0)
    torch.cuda.synchronize()
    lz.check(pipe.dev_err)
    assert np.array_equal(pipe.batches[0].ids.cpu().numpy(), ids), "sampled ids"
    o = H.assert_unique_matches(pipe.ures, ids, w.V, oracle, w.name)
    U = len(o[0])
    S = oracle.segsum(g, o[3], U)
    sq = H.sum_of_squares(g, o[3], U, oracle)
    got = pipe.reduced_rows(U).cpu().numpy()
    H.check_rows(got, S, sq)
    H.assert_single_rows_exact(got, S, o[1])
    lr = _f32(w.lr)
    ref = oracle.sgd(table0[o[0]], S, lr)
    table = pipe.state["table"]
    rows_t = torch.from_numpy(o[0]).to(table.device)
    H.assert_sgd_rows(table[rows_t].cpu().numpy(), ref, S, lr, H.row_delta(S, H.TOL_F32, sq))
    _release(pipe)


def _overlap_case(name):
    w = synth.WORKLOADS[name if name in synth.WORKLOADS else "merge_64x32k_bf16"]
    if name == "merge_8x32k_bf16":
        import dataclasses
        w = dataclasses.replace(w, name=name, shards=8)
    return w


def _final_state(pipe, ures):
    """What the steps leave behind: the table for SGD, else the EXPAND
    destination rows of the last step's merged types (rows past them are
    never written)."""
    if "table" in pipe.state:
        return pipe.state["table"]
    U = int(ures.num_unique.item())
    return pipe.state["M"][:U]


@pytest.mark.parametrize("name", ["word_step_64k", "sampled_softmax_64x1024_G", "merge_8x32k_bf16"])
def test_overlapped_schedule_matches_serial(lz, name):
    """bench.py's overlapped schedule (the Unique calls on a second stream,
    here in groups of two steps over four sets of their outputs) leaves the
    same result, bit for bit, as the serial steps: every Seg-Sum reads the
    Unique of its own batch and no Unique overwrites a set still in use.
    Seven steps wrap around the four sets, the last group a short one. The sampled-softmax case also
    draws its candidate ids on the second stream; the merge runs two Unique
    calls per step (the merged list and shard 0's own)."""
    import bench
    w = _overlap_case(name)
    dev = torch.device("cuda:0")
    nb, steps = 3, 7
    _say(f"[fullsize] overlapped vs serial: {w.name}, {nb} batches, {steps} steps")
    batches = [bench.Batch(w.batch(b), torch, dev) for b in range(nb)]
    table0 = w.table() if w.step in ("sgd", "softmax_sgd") else None
    serial = bench.Pipeline(w, batches, torch, lz, dev, table=table0)
    for i in range(steps):
        serial.step(i)
    torch.cuda.synchronize()
    serial.check()
    want = _final_state(serial, serial.ures)
    pipe = bench.Pipeline(w, batches, torch, lz, dev, table=table0)
    pipe.enable_overlap(group=2)
    main, side = torch.cuda.current_stream(), torch.cuda.Stream(device=dev)
    sync = bench.HipEvents(2 * steps + 2, timing=False)
    pipe.run_overlapped(0, steps, torch, main, side, sync)
    torch.cuda.synchronize()
    sync.close()
    pipe.check()
    last = pipe.sets[(steps - 1) % len(pipe.sets)][0]
    got = _final_state(pipe, last)
    U = int(serial.ures.num_unique.item())
    assert int(last.num_unique.item()) == U and torch.equal(last.uniq[:U], serial.ures.uniq[:U])
    assert got.shape == want.shape and torch.equal(got, want)
    if table0 is not None:
        assert not torch.equal(want, torch.from_numpy(table0).to(dev)), "the steps changed the table"
    del serial, pipe, want, got, batches
    torch.cuda.empty_cache()
