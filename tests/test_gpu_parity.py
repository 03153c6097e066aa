"""GPU parity: every entry point of liblmzipf.so against the CPU oracle on the
same seeded inputs, at sizes that span several tiles/chunks plus ragged
tails, and on the edge cases of the method. Integer outputs bit-exact; fp32
sums within the per-row tolerance of gpu_helpers."""
import itertools
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


@pytest.fixture(scope="module")
def lz():
    from paper_1810_10045_amd import lmzipf
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return lmzipf


DEV = "cuda"


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _say(msg):
    print(msg, flush=True)


# ---------------------------------------------------------------------------
# Unique
# ---------------------------------------------------------------------------

def test_unique_worked_example(lz):
    for J in ([0, 1, 2, 3, 0, 1], [17, 5, 42, 9, 17, 5]):
        ids = np.array(J, np.int32)
        res = lz.unique(_t(ids), 100)
        torch.cuda.synchronize()
        lz.check(res.dev_err)
        o = H.assert_unique_matches(res, ids, 100, oracle, f"J={J}")
        assert len(o[0]) == 4 and int(o[1].sum()) == 6


def test_unique_brute_force(lz):
    """Every J in [0, V)^K for V <= 4, K <= 6 (bit-exact against the oracle)."""
    cases = []
    for V, Kmax in ((1, 4), (2, 5), (3, 5), (4, 6)):
        for K in range(0, Kmax + 1):
            for J in itertools.product(range(V), repeat=K):
                ids = np.array(J, np.int32)
                cases.append((ids, V, lz.unique(_t(ids), V)))
    torch.cuda.synchronize()
    _say(f"brute force: {len(cases)} cases")
    for ids, V, res in cases:
        lz.check(res.dev_err)
        H.assert_unique_matches(res, ids, V, oracle, f"J={ids.tolist()} V={V}")


UNIQUE_CASES = [
    # (K, V, s, id dtype, seed)
    (1, 10, 1.0, np.int32, 1), (63, 100, 1.0, np.int32, 2), (64, 100, 1.0, np.int32, 3),
    (65, 7, 1.0, np.int32, 4), (255, 1000, 1.0, np.int32, 5), (257, 1, 1.0, np.int32, 6),
    (4095, 2, 1.0, np.int32, 7), (4096, 100_000, 1.0, np.int32, 8),
    (4097, 100_000, 1.0, np.int32, 9), (8205, 100_000, 1.0, np.int32, 10),
    (65536, 800_000, 1.0, np.int32, 11), (100_003, 20_000, 1.2, np.int32, 12),
    (262_144 + 77, 2_000_000, 0.9, np.int64, 13), (50_000, 2**31 - 1, 0.8, np.int32, 14),
    (30_001, 2**40, 0.9, np.int64, 15), (12_345, 256, 0.5, np.int32, 16),
    (20_000, 257, 1.0, np.int64, 17),
    # 1024-thread tiles from 2^14 + 1 keys: 10-bit digits where they save a
    # pass (40-bit int64 keys: 4 passes of 10; 20 bits: 2 of 10; 17 bits: a
    # 9-bit and an 8-bit pass), and the last K that still takes small tiles
    (150_001, 2**40, 0.9, np.int64, 18), (140_000, 1 << 20, 1.0, np.int32, 19),
    (131_073, 1 << 17, 1.0, np.int32, 20), (131_072, 800_000, 1.0, np.int32, 21),
    (16_385, 1 << 17, 1.0, np.int32, 25), (16_384, 800_000, 1.0, np.int32, 26),
    (16_385, 2**40, 0.9, np.int64, 27), (16_383, 2**40, 0.9, np.int64, 28),
    # the larger tile shapes (4 keys per thread above 512K ids, 8 above 1.5M)
    # with ragged last tiles
    (700_001, 800_000, 1.0, np.int32, 22), (1_600_003, 800_000, 1.0, np.int32, 23),
    (1_700_001, 2**40, 0.9, np.int64, 24),
    # heads on the first item of a thread, tails several threads later (the
    # case a compiler miscompile of the dedup scan once got wrong)
    (4096, 50, 1.0, np.int32, 3), (5000, 30, 1.0, np.int32, 8),
    # the one-workgroup path: every keys-per-thread shape, its last K and the
    # first K past it, all-distinct types filling the block, 64-bit keys
    (1024, 1 << 20, 0.0, np.int32, 29), (1025, 100_000, 1.0, np.int32, 30),
    (2049, 100_000, 1.0, np.int32, 31), (8192, 100_000, 1.0, np.int32, 32),
    (8193, 100_000, 1.0, np.int32, 33), (8192, 2**40, 0.9, np.int64, 34),
    (3000, 2**40, 0.0, np.int64, 35), (8192, 3, 1.0, np.int32, 36),
    # its digit widths: 8 bits over 2 and 4 passes (15- and 31-bit keys),
    # 9 bits (17-bit keys above, and 62-bit keys in 7 passes), 10 bits
    # (20- and 40-bit keys above)
    (7000, 20_000, 1.2, np.int32, 37), (8000, 2**31 - 1, 0.0, np.int32, 38),
    (5000, 2**62, 0.8, np.int64, 39),
    # tile-local passes joined by gathers, 12 to 64 tiles (the cases above
    # from 22,529 to 131,072 ids take them too). Up to 65,536 ids: tiles of
    # 1,024 keys on 256 threads, digits of at most 8 bits; the last K before
    # them (11 tiles of 2,048: look-back passes, two 10-bit digits) and the
    # first (23 tiles, 7 + 7 + 6 bits), one pass over 0 key bits, 9-bit keys
    # as 5 + 4 bits, 18-bit int64 keys as 6 + 6 + 6 bits.
    (22_528, 800_000, 1.0, np.int32, 43), (22_529, 800_000, 1.0, np.int32, 44),
    (40_000, 1, 1.0, np.int32, 40), (40_000, 300, 1.0, np.int32, 45),
    (65_536, 1 << 18, 1.0, np.int64, 46),
    # From 65,537 to 131,072 ids: tiles of 2,048 keys on 1024 threads, digits
    # of up to 9 bits: 21-bit keys as 7 + 7 + 7 bits; one 9-bit pass; 17-bit
    # keys as 9 + 8 bits; two 9-bit passes (int32 and int64); three 9-bit
    # passes over 27-bit int64 keys; 64 tiles of 40-bit keys in 8-bit passes.
    (70_001, 1 << 21, 1.0, np.int32, 41), (70_001, 512, 1.0, np.int32, 47),
    (100_000, 1 << 17, 1.0, np.int32, 48), (100_000, 1 << 18, 1.0, np.int32, 49),
    (100_000, 1 << 18, 1.0, np.int64, 50), (131_072, 1 << 27, 0.9, np.int64, 51),
    (131_072, 2**40, 0.9, np.int64, 42),
    # Vocabularies of at most 32,768 ids past one workgroup and outside the
    # tile-local passes: a count per id gives the types (no dedup), and the
    # first radix pass writes the inverse map. The char workload's shape
    # (15-bit keys as 8 + 7 bits) at 2 and 8 keys per thread, the largest
    # vocabulary with int64 ids at 4 keys per thread, one id (no key bits),
    # five ids, all ids nearly uniform, 1024-thread tiles too few for the
    # tile-local passes (9 tiles), 256-thread tiles; (12,345, 256) and
    # (20,000, 257) above take this path too.
    (150_000, 20_000, 1.2, np.int32, 52), (2_000_001, 20_000, 1.2, np.int32, 53),
    (1_048_579, 32_768, 1.0, np.int64, 54), (600_001, 1, 1.0, np.int32, 55),
    (300_000, 5, 1.0, np.int32, 56), (262_145, 32_767, 0.0, np.int32, 57),
    (16_385, 1_000, 1.0, np.int32, 58), (9_000, 32_768, 1.0, np.int64, 59),
    # Two passes over int32 ids with the counts per id write the second
    # pass's digit and the position as one word: on 256-thread tiles too.
    (12_000, 20_000, 1.2, np.int32, 66), (16_384, 32_768, 1.0, np.int32, 67),
    # From 524,288 ids on, vocabularies of up to 2^24 ids past the counts per
    # id: the dedup writes each type to a table indexed by id, and the
    # inverse map is written in token order from it. 20-bit keys at 4 keys
    # per thread, the first K to take it (21-bit int64 keys), the last K
    # before it (the dedup's scatter of the inverse map), the largest
    # vocabulary to take it (a 64 MiB table) and the first above it; 600,003
    # ids write the inverse map in 16-byte stores with a scalar tail.
    (600_000, 800_000, 1.0, np.int32, 60), (524_288, 2_000_000, 0.9, np.int64, 61),
    (600_003, 800_000, 1.0, np.int32, 65),
    (524_287, 800_000, 1.0, np.int32, 62), (600_000, 1 << 24, 1.0, np.int32, 63),
    (600_000, (1 << 24) + 1, 1.0, np.int64, 64),
]


@pytest.mark.parametrize("K,V,s,dt,seed", UNIQUE_CASES,
                         ids=[f"K{c[0]}-V{c[1]}-{c[3].__name__}" for c in UNIQUE_CASES])
def test_unique_random(lz, K, V, s, dt, seed):
    ids = synth.zipf_ids(K, min(V, 4_000_000), s, seed, dt)
    if V > 4_000_000:
        # spread the ranks over the whole id range (and above 2^32 for int64)
        ids = (ids.astype(np.int64) * (V // 4_000_000) + (V - 4_000_000 * (V // 4_000_000))).astype(dt)
        assert ids.max() < V
    _say(f"unique K={K} V={V} dtype={dt.__name__}")
    res = lz.unique(_t(ids), V)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    H.assert_unique_matches(res, ids, V, oracle, f"K={K} V={V}")


@pytest.mark.parametrize("K", [70_000, 9000, 8192, 1024])
def test_unique_all_same_and_all_distinct(lz, K):
    # 8192 and 1024: a full one-workgroup tile, every id its own type
    same = np.full(K, 4242, np.int32)
    res = lz.unique(_t(same), 5000)
    perm_ids = np.random.Generator(np.random.PCG64(5)).permutation(K).astype(np.int32)
    res2 = lz.unique(_t(perm_ids), K)
    top = np.full(K, 4999, np.int32)  # every id is V - 1
    res3 = lz.unique(_t(top), 5000)
    torch.cuda.synchronize()
    for r, ids, V in ((res, same, 5000), (res2, perm_ids, K), (res3, top, 5000)):
        lz.check(r.dev_err)
        H.assert_unique_matches(r, ids, V, oracle)


def test_unique_empty(lz):
    res = lz.unique(torch.zeros(0, dtype=torch.int32, device=DEV), 10)
    torch.cuda.synchronize()
    assert int(res.num_unique.item()) == 0 and int(res.offsets[0].item()) == 0


def test_unique_out_of_range_sets_error(lz):
    ids = np.array([1, 2, 99, 3], np.int32)
    res = lz.unique(_t(ids), 10)
    torch.cuda.synchronize()
    assert int(res.dev_err.item()) & lz.DEVERR_ID_RANGE
    ids = np.array([1, -4, 3], np.int64)
    res = lz.unique(_t(ids), 10)
    torch.cuda.synchronize()
    assert int(res.dev_err.item()) & lz.DEVERR_ID_RANGE


@pytest.mark.parametrize("K,V", [(12_000, 1000), (70_000, 1000), (300_000, 1000),
                                 (300_000, 20_000), (600_000, 800_000)])
def test_unique_out_of_range_sets_error_multi_tile(lz, K, V):
    # 256-thread tiles, tile-local passes, 1024-thread look-back passes (the
    # first and the last with counts per id, V = 1000; V = 20,000 with the
    # counts per id and the packed two passes; V = 800,000 with the type
    # table): one id past V in the last tile, one negative id in the first
    ids = synth.zipf_ids(K, V, 1.0, 62, np.int32)
    ids[K - 1] = V
    res = lz.unique(_t(ids), V)
    ids2 = ids.copy()
    ids2[K - 1] = 7
    ids2[3] = -1
    res2 = lz.unique(_t(ids2), V)
    torch.cuda.synchronize()
    assert int(res.dev_err.item()) & lz.DEVERR_ID_RANGE
    assert int(res2.dev_err.item()) & lz.DEVERR_ID_RANGE


@pytest.mark.parametrize("K,V,dt", [(70_000, 800_000, np.int32), (9000, 100_000, np.int64),
                                     (5000, 100_000, np.int32), (600_001, 800_000, np.int32),
                                     (600_001, 2_000_000, np.int64)])
def test_unique_outputs_not_16_byte_aligned(lz, K, V, dt):
    """Output buffers that start one element into their allocation (4- or
    8-byte aligned, not 16): the dedup then reads the permutation with
    scalar loads, the inverse map from the type table (600,001 ids) is
    written with scalar stores, and every output lands where the caller
    asked."""
    ids = synth.zipf_ids(K, V, 1.0, 61, dt)
    tdt = torch.int64 if dt == np.int64 else torch.int32
    cap = min(K, V)

    def shifted(n, dtype):
        return torch.full((n + 1,), -7, dtype=dtype, device=DEV)[1:]

    out = lz.UniqueResult(shifted(cap, tdt), shifted(cap, torch.int32), shifted(cap + 1, torch.int32),
                          shifted(K, torch.int32), shifted(K, torch.int32),
                          torch.zeros(1, dtype=torch.int64, device=DEV),
                          torch.zeros(1, dtype=torch.int32, device=DEV))
    assert out.perm.data_ptr() % 16 != 0
    _say(f"unique unaligned outputs K={K} V={V} dtype={dt.__name__}")
    res = lz.unique(_t(ids), V, out=out)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    H.assert_unique_matches(res, ids, V, oracle, f"unaligned K={K}")


@pytest.mark.parametrize("K,V", [(70_000, 800_000), (300_000, 20_000)])
def test_unique_wait_failure_is_reported(lz, K, V):
    """The failure path of the look-backs of the multi-workgroup Unique,
    forced from the host: with the test hook set, every predecessor reads as
    not ready, each look-back gives up after 64 polls with LM_DEVERR_SPIN,
    and the kernels still finish inside their buffers. With the hook
    cleared, the next call on the same workspace is exact again. Tile-local
    passes with the gathering dedup; look-back passes with the key scan."""
    ids = synth.zipf_ids(K, V, 1.0, 73, np.int32)
    ws = lz.Workspace(DEV)
    _say("unique with forced look-back failures")
    lz.force_wait_failure(True, 64)
    try:
        bad = lz.unique(_t(ids), V, ws=ws)
        torch.cuda.synchronize()
    finally:
        lz.force_wait_failure(False)
    assert int(bad.dev_err.item()) & lz.DEVERR_SPIN
    res = lz.unique(_t(ids), V, ws=ws)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    H.assert_unique_matches(res, ids, V, oracle, "after the forced failures")


def test_unique_workspace_reuse_and_determinism(lz):
    """Back-to-back calls on one workspace, with different sizes and a
    workspace full of garbage, stay exact."""
    ws = lz.Workspace(DEV)
    ws.get(1 << 24).fill_(0xA5)
    outs = []
    for K, V, seed in ((70_000, 800_000, 21), (5000, 30, 22), (70_000, 800_000, 21), (1, 3, 23)):
        ids = synth.zipf_ids(K, V, 1.0, seed, np.int32)
        outs.append((ids, V, lz.unique(_t(ids), V, ws=ws)))
    torch.cuda.synchronize()
    for ids, V, r in outs:
        lz.check(r.dev_err)
        H.assert_unique_matches(r, ids, V, oracle)
    assert torch.equal(outs[0][2].perm, outs[2][2].perm)


# ---------------------------------------------------------------------------
# Seg-Sum
# ---------------------------------------------------------------------------

SEG_CASES = [
    # (K, V, s, D, grad dtype, seed)
    (1, 5, 1.0, 16, "f32", 31), (6, 4, 1.0, 3, "f32", 32), (257, 30, 1.0, 1, "f32", 33),
    (1000, 50, 1.0, 17, "f32", 34), (5000, 100, 1.2, 64, "f32", 35),
    (20_000, 300, 1.2, 96, "f32", 36), (20_000, 300, 1.2, 1100, "f32", 37),
    (40_000, 2000, 1.0, 512, "f32", 38), (65_536, 800_000, 1.0, 1024, "f32", 39),
    (150_000, 20_000, 1.2, 256, "f32", 40), (30_000, 5000, 1.0, 2048, "f32", 41),
    (3000, 100, 1.0, 4096, "f32", 42),
    (5000, 100, 1.2, 64, "bf16", 43), (20_000, 300, 1.2, 1024, "bf16", 44),
    (70_000, 800_000, 1.0, 1024, "bf16", 45), (9000, 500, 1.0, 100, "bf16", 46),
    (2000, 50, 1.0, 7, "bf16", 47),
    # rows wider than one 1024-column tile, walked and fixed up in one launch
    # (ragged last tiles, bf16 too), and wider than that one launch takes
    (40_000, 300, 1.2, 2048, "bf16", 48), (12_000, 800, 1.0, 1536, "bf16", 49),
    (4000, 100, 1.0, 5000, "f32", 50),
]


def _segsum_case(lz, K, V, s, D, gdt, seed, ws=None, perm_seed=0):
    ids = (synth.zipf_ids_permuted(K, V, s, seed, perm_seed, np.int32) if perm_seed
           else synth.zipf_ids(K, V, s, seed, np.int32))
    g32 = synth.normal_rows(K, D, seed + 1000)
    grad = synth.bf16_bits(g32) if gdt == "bf16" else g32
    tgrad = _t(g32).to(torch.bfloat16) if gdt == "bf16" else _t(g32)
    if gdt == "bf16":  # torch's fp32->bf16 is round-to-nearest-even, like the generator
        assert np.array_equal(tgrad.view(torch.int16).cpu().numpy().view(np.uint16), grad)
    res = lz.unique(_t(ids), V, ws=ws)
    out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, dev_err=res.dev_err, ws=ws)
    return ids, grad, res, out


@pytest.mark.parametrize("K,V,s,D,gdt,seed", SEG_CASES,
                         ids=[f"K{c[0]}-V{c[1]}-D{c[3]}-{c[4]}" for c in SEG_CASES])
def test_segsum_random(lz, K, V, s, D, gdt, seed, perm_seed=0):
    _say(f"segsum K={K} V={V} D={D} {gdt} perm_seed={perm_seed}")
    ids, grad, res, out = _segsum_case(lz, K, V, s, D, gdt, seed, perm_seed=perm_seed)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    o = H.assert_unique_matches(res, ids, V, oracle)
    U = len(o[0])
    ref = oracle.segsum(grad, o[3], U)
    got = out[:U].double().cpu().numpy()
    H.check_rows(got, ref, H.sum_of_squares(grad, o[3], U, oracle), gdt)
    H.assert_single_rows_exact(got, ref, o[1])


PERM_CASES = [
    # Zipf ranks spread over the ids by a fixed permutation: the long runs of
    # the heads fall anywhere in the sorted order, among short ones.
    (65_536, 800_000, 1.0, 1024, "f32", 51), (150_000, 20_000, 1.2, 256, "f32", 52),
    (70_000, 800_000, 1.0, 1024, "bf16", 53), (20_000, 300, 1.2, 96, "f32", 54),
]


@pytest.mark.parametrize("K,V,s,D,gdt,seed", PERM_CASES,
                         ids=[f"K{c[0]}-V{c[1]}-D{c[3]}-{c[4]}" for c in PERM_CASES])
def test_segsum_permuted_ids(lz, K, V, s, D, gdt, seed):
    test_segsum_random(lz, K, V, s, D, gdt, seed, perm_seed=seed + 500)


@pytest.mark.parametrize("gdt", ["bf16", "f32"])
def test_segsum_chunks_inside_short_segments(lz, gdt):
    """One head of 30,000 tokens and 600 types of 15 (just under the
    long-segment threshold of 16 at this K): with so few types for the
    capacity, a bf16 chunk holds about 13.6 positions, and some chunks lie
    wholly inside a short segment owned by an earlier chunk."""
    base = np.concatenate([np.full(30_000, 0)] + [np.full(15, 1000 * t) for t in range(1, 601)])
    ids = np.random.Generator(np.random.PCG64(81)).permutation(base).astype(np.int32)
    K, V, D = len(ids), 800_000, 64
    _say(f"segsum short segments K={K} {gdt}")
    g32 = synth.normal_rows(K, D, 82)
    grad = synth.bf16_bits(g32) if gdt == "bf16" else g32
    tgrad = _t(g32).to(torch.bfloat16) if gdt == "bf16" else _t(g32)
    res = lz.unique(_t(ids), V)
    out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, dev_err=res.dev_err)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    o = H.assert_unique_matches(res, ids, V, oracle)
    U = len(o[0])
    ref = oracle.segsum(grad, o[3], U)
    H.check_rows(out[:U].double().cpu().numpy(), ref, H.sum_of_squares(grad, o[3], U, oracle), gdt)


def _piece_counts(ids, V, rw, ww):
    """Host restatement of the walk's cost partition (a position costs rw,
    a segment end ww; R the power of two near K/1024 in 16..512, T = R/4):
    for every segment of at least T rows that spans chunks, the number of
    chunks after its first that it reaches, and its first chunk."""
    K = len(ids)
    _, c = np.unique(ids, return_counts=True)
    U = len(c)
    off = np.concatenate([[0], np.cumsum(c)])
    R = 16
    while R < (K + 1023) // 1024 and R < 512:
        R *= 2
    T = R // 4
    n = -(-(rw * K + ww * min(K, V)) // (rw * R))
    Q = -(-(rw * K + ww * U) // n)
    f = rw * off[:-1] + ww * np.arange(U)
    cs, ce = f // Q, np.minimum((f + rw * (c - 1)) // Q, n - 1)
    lg = (c >= T) & (ce > cs)
    return (ce - cs)[lg], cs[lg]


@pytest.mark.parametrize("gdt", ["f32", "bf16"])
def test_segsum_fixup_piece_counts(lz, gdt):
    """Long segments of graded lengths: 1, 15 and 16 further pieces (the
    last count summed by one wave and the first summed by a workgroup), a
    head of more than 128 (several rounds per wave), and 8-chunk fix-up
    groups that start both a head and a shorter long segment."""
    rng = np.random.Generator(np.random.PCG64(3))
    sc, lens = 45, []
    for k in range(1, 22):
        lens += [1] * int(rng.integers(3, 40)) + [16 + sc * k + int(rng.integers(0, sc))]
    for _ in range(12):
        lens += [1] * int(rng.integers(3, 40)) + [int(rng.integers(sc + 20, 2 * sc)),
                                                 int(rng.integers(17 * sc, 20 * sc))]
    lens += [1] * 20 + [160 * sc]
    lens += [1] * (60_000 - sum(lens))
    ids = rng.permutation(np.repeat(np.arange(len(lens)) * 7 + 3, lens)).astype(np.int32)
    K, V, D = len(ids), 800_000, 96
    # (rw, ww): a read row costs 2 * sizeof(grad), a written fp32 row 8 (its
    # bytes) with fp32 rows and 16 with bf16 rows
    P, cs = _piece_counts(ids, V, *((4, 16) if gdt == "bf16" else (8, 8)))
    grp = cs // 8
    assert {1, 15, 16} <= set(P.tolist()) and P.max() > 128
    assert any((P[grp == g] >= 16).any() and (P[grp == g] < 16).any() for g in set(grp.tolist()))
    _say(f"segsum fix-up piece counts K={K} {gdt}: {len(P)} long segments, max {P.max()} pieces")
    g32 = synth.normal_rows(K, D, 91)
    grad = synth.bf16_bits(g32) if gdt == "bf16" else g32
    tgrad = _t(g32).to(torch.bfloat16) if gdt == "bf16" else _t(g32)
    res = lz.unique(_t(ids), V)
    out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, dev_err=res.dev_err)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    o = H.assert_unique_matches(res, ids, V, oracle)
    U = len(o[0])
    ref = oracle.segsum(grad, o[3], U)
    H.check_rows(out[:U].double().cpu().numpy(), ref, H.sum_of_squares(grad, o[3], U, oracle), gdt)


def test_segsum_workspace_reuse(lz):
    """One workspace through calls of different shapes: each layout puts the
    per-chunk flags of the one-launch path where another call left partial
    rows or flags, and a call must never take an earlier call's flag for its
    own. Each result is checked against the oracle."""
    ws = lz.Workspace(DEV)
    cases = [(65_536, 800_000, 1.0, 1024, "f32", 101), (20_000, 300, 1.2, 96, "f32", 102),
             (70_000, 800_000, 1.0, 1024, "bf16", 103), (65_536, 800_000, 1.0, 1024, "f32", 104),
             (9000, 500, 1.0, 100, "bf16", 105), (65_536, 800_000, 1.0, 1024, "f32", 101)]
    for K, V, s, D, gdt, seed in cases:
        _say(f"segsum workspace reuse K={K} D={D} {gdt}")
        ids, grad, res, out = _segsum_case(lz, K, V, s, D, gdt, seed, ws=ws)
        torch.cuda.synchronize()
        lz.check(res.dev_err)
        o = H.assert_unique_matches(res, ids, V, oracle)
        U = len(o[0])
        ref = oracle.segsum(grad, o[3], U)
        H.check_rows(out[:U].double().cpu().numpy(), ref, H.sum_of_squares(grad, o[3], U, oracle),
                     gdt)


def test_segsum_wait_failure_is_reported(lz):
    """The failure path of the one-launch form's bounded waits, forced from
    the host: with the test hook set, the fix-up workgroups wait for a flag
    value no walk writes, give up after 64 polls and raise LM_DEVERR_SPIN,
    and the launch still finishes. With the hook cleared, the next call on
    the same workspace is exact again."""
    K, V, D = 65_536, 800_000, 1024
    ids = synth.zipf_ids(K, V, 1.0, 71, np.int32)
    g32 = synth.normal_rows(K, D, 72)
    ws = lz.Workspace(DEV)
    res = lz.unique(_t(ids), V, ws=ws)
    grad = _t(g32)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    _say("segsum with forced wait failures")
    lz.force_wait_failure(True, 64)
    try:
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        lz.segsum(grad, res.perm, res.inverse, res.offsets, res.num_unique, dev_err=err, ws=ws)
        torch.cuda.synchronize()
    finally:
        lz.force_wait_failure(False)
    assert int(err.item()) & lz.DEVERR_SPIN
    err2 = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = lz.segsum(grad, res.perm, res.inverse, res.offsets, res.num_unique, dev_err=err2, ws=ws)
    torch.cuda.synchronize()
    lz.check(err2)
    o = oracle.unique(ids, V)
    U = len(o[0])
    ref = oracle.segsum(g32, o[3], U)
    rel = H.row_rel_err(out[:U].double().cpu().numpy(), ref, H.sum_of_squares(g32, o[3], U, oracle))
    assert rel <= H.TOL_F32


def test_segsum_deterministic(lz):
    _, _, ra, a = _segsum_case(lz, 60_000, 500, 1.2, 1024, "f32", 51)
    _, _, rb, b = _segsum_case(lz, 60_000, 500, 1.2, 1024, "f32", 51)
    torch.cuda.synchronize()
    U = int(ra.num_unique.item())
    assert U == int(rb.num_unique.item())
    assert torch.equal(a[:U], b[:U])  # rows past U are never written


@pytest.mark.parametrize("D,gdt", [(2048, "f32"), (1024, "bf16")])
def test_segsum_on_cu_masked_stream(lz, D, gdt):
    """On a stream limited to 32 CUs (a contiguous mask: 4 CUs of each XCD)
    the walk's chunks are sized for whole rounds of the waves that fit on
    those CUs, several rounds here where the whole device holds them in one.
    Checked against the oracle, bit-identical from run to run on that
    stream, and lm_segsum_rows, lm_segsum_sgd (lr = -1 on zeros: the sums)
    and lm_segsum_adam (beta1 = 0 on zeros: the sums in m) bit-identical to
    lm_segsum there too: all four size their chunks for the same CUs."""
    K, V, s, seed = 100_000, 5000, 1.2, 131
    _say(f"segsum on a 32-CU stream K={K} D={D} {gdt}")
    ids = synth.zipf_ids(K, V, s, seed, np.int32)
    g32 = synth.normal_rows(K, D, seed + 1000)
    grad = synth.bf16_bits(g32) if gdt == "bf16" else g32
    tgrad = _t(g32).to(torch.bfloat16) if gdt == "bf16" else _t(g32)
    res = lz.unique(_t(ids), V)
    torch.cuda.synchronize()
    U = int(res.num_unique.item())
    ms = H.CuMaskedStream(torch, 0, 32)
    try:
        outs = [lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique,
                          dev_err=res.dev_err, stream=ms.stream) for _ in range(2)]
        table = torch.zeros((V, D), dtype=torch.float32, device=DEV)
        lz.segsum_rows(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq,
                       table, dev_err=res.dev_err, stream=ms.stream)
        tsgd = torch.zeros((V, D), dtype=torch.float32, device=DEV)
        lz.segsum_sgd(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq,
                      tsgd, -1.0, dev_err=res.dev_err, stream=ms.stream)
        pmv = [torch.zeros((V, D), dtype=torch.float32, device=DEV) for _ in range(3)]
        lz.segsum_adam(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq,
                       pmv[0], pmv[1], pmv[2], lr=0.0, beta1=0.0, step=1, dev_err=res.dev_err,
                       stream=ms.stream)
        ms.stream.synchronize()
    finally:
        ms.close()
    lz.check(res.dev_err)
    o = H.assert_unique_matches(res, ids, V, oracle)
    ref = oracle.segsum(grad, o[3], U)
    got = outs[0][:U].double().cpu().numpy()
    H.check_rows(got, ref, H.sum_of_squares(grad, o[3], U, oracle), gdt, "32-CU stream")
    H.assert_single_rows_exact(got, ref, o[1])
    assert torch.equal(outs[0][:U], outs[1][:U]), "not deterministic on the masked stream"
    assert torch.equal(table[res.uniq[:U].long()], outs[0][:U]), "rows variant differs"
    assert torch.equal(tsgd, table), "SGD variant's sums differ"
    assert torch.equal(pmv[1], table), "Adam variant's sums differ"


@pytest.mark.parametrize("K,V,s,D,gdt,seed", [(65_536, 800_000, 1.0, 1024, "f32", 121),
                                               (60_000, 500, 1.2, 1024, "f32", 122),
                                               (70_000, 800_000, 1.0, 1024, "bf16", 123)])
def test_segsum_two_launch_switch(lz, K, V, s, D, gdt, seed):
    """lm_segsum_set_two_launches: shapes that take the one-launch form by
    default run as the walk plus a separate fix-up kernel while the switch
    is on. Both forms are checked against the oracle; the two-launch form is
    bit-identical from run to run; switching back restores the default."""
    _say(f"segsum two-launch switch K={K} D={D} {gdt}")
    assert lz.segsum_two_launches(True) is False, "the switch is off by default"
    try:
        ids, grad, res, two = _segsum_case(lz, K, V, s, D, gdt, seed)
        again = _segsum_case(lz, K, V, s, D, gdt, seed)[3]
        torch.cuda.synchronize()
        lz.check(res.dev_err)
    finally:
        assert lz.segsum_two_launches(False) is True
    one = _segsum_case(lz, K, V, s, D, gdt, seed)[3]
    torch.cuda.synchronize()
    o = H.assert_unique_matches(res, ids, V, oracle)
    U = len(o[0])
    ref = oracle.segsum(grad, o[3], U)
    sq = H.sum_of_squares(grad, o[3], U, oracle)
    assert torch.equal(two[:U], again[:U]), "two-launch form not deterministic"
    H.check_rows(two[:U].double().cpu().numpy(), ref, sq, gdt, "two launches")
    H.check_rows(one[:U].double().cpu().numpy(), ref, sq, gdt, "one launch")


def test_segsum_special_rows(lz):
    """One type: the column sum; every id distinct: the permuted rows."""
    K, D = 30_000, 160
    g = synth.normal_rows(K, D, 61)
    same = np.full(K, 3, np.int32)
    r1 = lz.unique(_t(same), 10)
    o1 = lz.segsum(_t(g), r1.perm, r1.inverse, r1.offsets, r1.num_unique, dev_err=r1.dev_err)
    dist = np.random.Generator(np.random.PCG64(62)).permutation(K).astype(np.int32)
    r2 = lz.unique(_t(dist), K)
    o2 = lz.segsum(_t(g), r2.perm, r2.inverse, r2.offsets, r2.num_unique, dev_err=r2.dev_err)
    torch.cuda.synchronize()
    lz.check(r1.dev_err)
    lz.check(r2.dev_err)
    colsum = g.astype(np.float64).sum(0, keepdims=True)
    assert H.row_rel_err(o1[:1].double().cpu().numpy(), colsum) <= H.TOL_F32
    assert np.array_equal(o2[:K].cpu().numpy(), g[np.argsort(dist)])


def test_segsum_strided_and_capacity(lz):
    """Row strides larger than D (a column slice of a wider matrix), the
    scalar path (unaligned stride), and u_cap below U."""
    K, V, D = 9000, 700, 40
    ids = synth.zipf_ids(K, V, 1.0, 71, np.int32)
    wide = synth.normal_rows(K, 3 * D + 1, 72)
    res = lz.unique(_t(ids), V)
    tw = _t(wide)
    out_a = lz.segsum(tw[:, 5:5 + D], res.perm, res.inverse, res.offsets, res.num_unique, dev_err=res.dev_err)
    out_b = lz.segsum(tw[:, 8:8 + D], res.perm, res.inverse, res.offsets, res.num_unique, dev_err=res.dev_err)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    o = oracle.unique(ids, V)
    U = len(o[0])
    for out, c0 in ((out_a, 5), (out_b, 8)):
        ref = oracle.segsum(np.ascontiguousarray(wide[:, c0:c0 + D]), o[3], U)
        assert H.row_rel_err(out[:U].double().cpu().numpy(), ref) <= H.TOL_F32
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    small = torch.full((10, D), 7.0, device=DEV)
    lz.segsum(tw[:, :D], res.perm, res.inverse, res.offsets, res.num_unique, u_cap=10, out=small, dev_err=err)
    torch.cuda.synchronize()
    assert int(err.item()) & lz.DEVERR_CAPACITY
    # the same on the vector path (walk and fix-up in one launch): the
    # capacity error, and no fix-up wait that gave up
    g64 = _t(synth.normal_rows(K, 64, 73))
    err2 = torch.zeros(1, dtype=torch.int32, device=DEV)
    small2 = torch.full((10, 64), 7.0, device=DEV)
    lz.segsum(g64, res.perm, res.inverse, res.offsets, res.num_unique, u_cap=10, out=small2, dev_err=err2)
    torch.cuda.synchronize()
    assert int(err2.item()) == lz.DEVERR_CAPACITY


ROWS_CASES = [
    # (K, V, s, D, grad dtype, id dtype, seed): one-workgroup Unique and a
    # 512-column walk; rows of two 1024-column tiles in one launch (f32 and
    # bf16, int64 row ids); narrow rows; rows wider than the one-launch form
    # takes (walk, then the separate fix-up); a single token.
    (8192, 100_000, 1.0, 512, "f32", np.int32, 131),
    (60_000, 20_000, 1.2, 2048, "f32", np.int32, 132),
    (40_000, 300, 1.2, 2048, "bf16", np.int64, 133),
    (20_000, 300, 1.2, 96, "f32", np.int64, 134),
    (4000, 100, 1.0, 5000, "f32", np.int32, 135),
    (1, 5, 1.0, 16, "f32", np.int32, 136),
]


def _rows_case(lz, K, V, s, D, gdt, dt, seed):
    ids = synth.zipf_ids(K, V, s, seed, dt)
    g32 = synth.normal_rows(K, D, seed + 1000)
    grad = synth.bf16_bits(g32) if gdt == "bf16" else g32
    tgrad = _t(g32).to(torch.bfloat16) if gdt == "bf16" else _t(g32)
    res = lz.unique(_t(ids), V)
    return ids, grad, tgrad, res


@pytest.mark.parametrize("K,V,s,D,gdt,dt,seed", ROWS_CASES,
                         ids=[f"K{c[0]}-V{c[1]}-D{c[3]}-{c[4]}-{np.dtype(c[5]).name}"
                              for c in ROWS_CASES])
def test_segsum_rows_is_segsum_then_scatter(lz, K, V, s, D, gdt, dt, seed):
    """lm_segsum_rows into a dense V x D table with row_ids = uniq: the same
    table, bit for bit, as lm_segsum followed by Fill-Values SCATTER (each
    launch form against lm_segsum in that form: the forms group the heads'
    partial rows differently); the written rows match the oracle's steps 2
    and 5; every other row keeps its value."""
    _say(f"segsum_rows K={K} V={V} D={D} {gdt} {np.dtype(dt).name}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, s, D, gdt, dt, seed)
    base = _t(synth.normal_rows(V, D, seed + 2000))
    out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, dev_err=res.dev_err)
    want = base.clone()
    lz.fill_values(out, res.uniq, res.num_unique, want, None, None, "scatter", dev_err=res.dev_err)
    got = base.clone()
    lz.segsum_rows(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, got,
                   dev_err=res.dev_err)
    assert lz.segsum_two_launches(True) is False
    try:
        out2 = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique,
                         dev_err=res.dev_err)
        want2 = base.clone()
        lz.fill_values(out2, res.uniq, res.num_unique, want2, None, None, "scatter",
                       dev_err=res.dev_err)
        got2 = base.clone()
        lz.segsum_rows(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, got2,
                       dev_err=res.dev_err)
        torch.cuda.synchronize()
    finally:
        assert lz.segsum_two_launches(False) is True
    lz.check(res.dev_err)
    o = H.assert_unique_matches(res, ids, V, oracle)
    U = len(o[0])
    assert torch.equal(got, want), "not the table of lm_segsum + SCATTER"
    assert torch.equal(got2, want2), "two-launch form: not lm_segsum + SCATTER"
    touched = torch.zeros(V, dtype=torch.bool, device=DEV)
    touched[_t(o[0].astype(np.int64))] = True
    assert torch.equal(got[~touched], base[~touched]), "a row no type names was written"
    ref = oracle.segsum(grad, o[3], U)
    rows = got[_t(o[0].astype(np.int64))].double().cpu().numpy()
    H.check_rows(rows, ref, H.sum_of_squares(grad, o[3], U, oracle), gdt)
    if V * D <= 1 << 20:  # the oracle's dense table, whole
        dense = oracle.scatter(ref, o[0], base.double().cpu().numpy())
        assert H.row_rel_err(got.double().cpu().numpy(), dense) <= (
            H.TOL_BF16 if gdt == "bf16" else H.TOL_F32)


@pytest.mark.parametrize("D,dt", [(512, np.int32), (2048, np.int64), (5000, np.int32)])
def test_segsum_rows_any_row_map(lz, D, dt):
    """row_ids need not be the uniq ids: type u to row U-1-u of a U-row
    output is lm_segsum's output (u_cap = U, the same chunks) upside down,
    bit for bit."""
    K, V = 20_000, 3000
    _say(f"segsum_rows reversed D={D}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, 1.0, D, "f32", dt, 141)
    U = int(res.num_unique.item())
    out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, u_cap=U,
                    dev_err=res.dev_err)
    rev = torch.arange(U - 1, -1, -1, device=DEV).to(torch.int64 if dt == np.int64 else torch.int32)
    got = torch.full((U, D), float("nan"), device=DEV)
    lz.segsum_rows(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, rev, got,
                   dev_err=res.dev_err)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    assert torch.equal(got, out[:U].flip(0))


@pytest.mark.parametrize("D", [512, 2048, 5000])
def test_segsum_rows_bad_row_id(lz, D):
    """A row id outside [0, out_rows) sets LM_DEVERR_ID_RANGE and leaves that
    type unwritten; the other types are written as usual. The longest type
    (summed by the fix-up) and a short one (ended inside the walk), and a
    negative id; then rows_cap below the number of types: the capacity
    error."""
    K, V = 30_000, 2000
    _say(f"segsum_rows bad ids D={D}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, 1.2, D, "f32", np.int64, 151)
    U = int(res.num_unique.item())
    counts = res.counts[:U].cpu().numpy()
    head, short = int(np.argmax(counts)), int(np.argmin(counts))
    # lm_segsum with u_cap = rows_cap: the same chunks, so the same sums
    out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, u_cap=U,
                    dev_err=res.dev_err)
    e10 = torch.zeros(1, dtype=torch.int32, device=DEV)
    out10 = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, u_cap=10,
                      out=torch.empty((10, D), device=DEV), dev_err=e10)
    base = _t(synth.normal_rows(V, D, 152))
    uniq = res.uniq[:U].clone()
    for bad_u, bad_id in ((head, V), (short, V + 99), (short, -1)):
        rid = uniq.clone()
        rid[bad_u] = bad_id
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        got = base.clone()
        lz.segsum_rows(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, rid, got,
                       dev_err=err)
        torch.cuda.synchronize()
        assert int(err.item()) == lz.DEVERR_ID_RANGE, (bad_u, bad_id)
        keep = torch.ones(U, dtype=torch.bool, device=DEV)
        keep[bad_u] = False
        assert torch.equal(got[uniq[keep]], out[:U][keep])
        assert torch.equal(got[uniq[bad_u]], base[uniq[bad_u]]), "the bad type was written"
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    got = base.clone()
    lz.segsum_rows(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, uniq[:10].clone(),
                   got, dev_err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == lz.DEVERR_CAPACITY == int(e10.item())
    assert torch.equal(got[uniq[:10]], out10)
    rest = torch.ones(V, dtype=torch.bool, device=DEV)
    rest[uniq[:10]] = False
    assert torch.equal(got[rest], base[rest]), "a type past rows_cap was written"


SGD_CASES = [
    # (K, V, s, D, grad dtype, id dtype, seed): the word step's ids over a
    # 100K vocabulary (many segment ends per gather batch); rows of two
    # 1024-column tiles in one launch (f32, and bf16 with int64 ids); rows
    # not a multiple of 4 wide (the scalar path); rows wider than the
    # one-launch form takes; one-workgroup Unique; a single token.
    (65_536, 100_000, 1.0, 1024, "f32", np.int32, 161),
    (60_000, 20_000, 1.2, 2048, "f32", np.int32, 162),
    (40_000, 300, 1.2, 2048, "bf16", np.int64, 163),
    (20_000, 3000, 1.0, 97, "f32", np.int32, 164),
    (9000, 500, 1.0, 100, "bf16", np.int64, 165),
    (4000, 100, 1.0, 5000, "f32", np.int32, 166),
    (8192, 100_000, 1.0, 512, "f32", np.int32, 167),
    (1, 5, 1.0, 16, "f32", np.int32, 168),
]


@pytest.mark.parametrize("K,V,s,D,gdt,dt,seed", SGD_CASES,
                         ids=[f"K{c[0]}-V{c[1]}-D{c[3]}-{c[4]}-{np.dtype(c[5]).name}"
                              for c in SGD_CASES])
def test_segsum_sgd_is_segsum_then_sgd(lz, K, V, s, D, gdt, dt, seed):
    """lm_segsum_sgd on a V x D table with row_ids = uniq: the same table, bit
    for bit, as lm_segsum followed by lm_sparse_apply SGD with the same lr
    (each launch form against lm_segsum in that form); the updated rows match
    the oracle's Seg-Sum and SGD; every other row keeps its value."""
    _say(f"segsum_sgd K={K} V={V} D={D} {gdt} {np.dtype(dt).name}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, s, D, gdt, dt, seed)
    lr = float(np.float32(0.1))
    p0 = synth.normal_rows(V, D, seed + 2000)
    base = _t(p0)

    def both():
        out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique,
                        dev_err=res.dev_err)
        want = base.clone()
        lz.sparse_apply(want, res.uniq, res.num_unique, out, "sgd", lr=lr, dev_err=res.dev_err)
        got = base.clone()
        lz.segsum_sgd(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, got,
                      lr, dev_err=res.dev_err)
        return want, got

    want, got = both()
    assert lz.segsum_two_launches(True) is False
    try:
        want2, got2 = both()
        torch.cuda.synchronize()
    finally:
        assert lz.segsum_two_launches(False) is True
    lz.check(res.dev_err)
    o = H.assert_unique_matches(res, ids, V, oracle)
    U = len(o[0])
    assert torch.equal(got, want), "not the table of lm_segsum + lm_sparse_apply SGD"
    assert torch.equal(got2, want2), "two-launch form: not lm_segsum + lm_sparse_apply SGD"
    rows_t = _t(o[0].astype(np.int64))
    touched = torch.zeros(V, dtype=torch.bool, device=DEV)
    touched[rows_t] = True
    assert torch.equal(got[~touched], base[~touched]), "a row no type names was updated"
    S = oracle.segsum(grad, o[3], U)
    sq = H.sum_of_squares(grad, o[3], U, oracle)
    ref = oracle.sgd(p0[o[0]], S, lr)
    H.assert_sgd_rows(got[rows_t].cpu().numpy(), ref, S, lr, H.row_delta(S, H.TOL_F32, sq))


@pytest.mark.parametrize("D", [512, 2048, 5000])
def test_segsum_sgd_minus_one_on_zeros_is_segsum_rows(lz, D):
    """With lr = -1 on a zero table each updated row is 0 + 1 * sum, which
    rounds to the sum itself: lm_segsum_rows's table, bit for bit."""
    K, V = 30_000, 2000
    _say(f"segsum_sgd lr=-1 D={D}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, 1.2, D, "f32", np.int32, 171)
    want = torch.zeros((V, D), device=DEV)
    lz.segsum_rows(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, want,
                   dev_err=res.dev_err)
    got = torch.zeros((V, D), device=DEV)
    lz.segsum_sgd(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, got, -1.0,
                  dev_err=res.dev_err)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    assert torch.equal(got, want)


@pytest.mark.parametrize("D", [512, 2048, 5000])
def test_segsum_sgd_bad_row_id(lz, D):
    """A row id outside [0, V) sets LM_DEVERR_ID_RANGE and leaves that row
    as it was, as lm_sparse_apply does; the other rows are updated as usual.
    The longest type (finished by the fix-up) and a short one (finished in
    the walk); then rows_cap below the number of types: the capacity
    error, and only the first rows_cap types are applied."""
    K, V = 30_000, 2000
    _say(f"segsum_sgd bad ids D={D}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, 1.2, D, "f32", np.int64, 172)
    U = int(res.num_unique.item())
    counts = res.counts[:U].cpu().numpy()
    head, short = int(np.argmax(counts)), int(np.argmin(counts))
    lr = 0.25
    # lm_segsum with u_cap = rows_cap: the same chunks, so the same sums
    out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, u_cap=U,
                    dev_err=res.dev_err)
    base = _t(synth.normal_rows(V, D, 173))
    uniq = res.uniq[:U].clone()
    for bad_u, bad_id in ((head, V), (short, V + 99), (short, -1)):
        rid = uniq.clone()
        rid[bad_u] = bad_id
        e_want = torch.zeros(1, dtype=torch.int32, device=DEV)
        want = base.clone()
        lz.sparse_apply(want, rid, res.num_unique, out, "sgd", lr=lr, dev_err=e_want)
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        got = base.clone()
        lz.segsum_sgd(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, rid, got, lr,
                      dev_err=err)
        torch.cuda.synchronize()
        assert int(err.item()) == lz.DEVERR_ID_RANGE == int(e_want.item()), (bad_u, bad_id)
        assert torch.equal(got, want)
    e10 = torch.zeros(1, dtype=torch.int32, device=DEV)
    out10 = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, u_cap=10,
                      out=torch.empty((10, D), device=DEV), dev_err=e10)
    want = base.clone()
    lz.sparse_apply(want, uniq[:10].clone(), torch.tensor([10], dtype=torch.int64, device=DEV),
                    out10, "sgd", lr=lr, dev_err=torch.zeros(1, dtype=torch.int32, device=DEV))
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    got = base.clone()
    lz.segsum_sgd(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, uniq[:10].clone(),
                  got, lr, dev_err=err)
    torch.cuda.synchronize()
    assert int(err.item()) == lz.DEVERR_CAPACITY == int(e10.item())
    assert torch.equal(got, want)


ADAM_CASES = [
    # (K, V, s, D, grad dtype, id dtype, seed): ids over a 100K vocabulary
    # (a segment end on most rows); rows of two 1024-column tiles (f32, and
    # bf16 with int64 ids); chunks of 512 positions; rows not a multiple of
    # 4 wide (the scalar path); rows wider than the one-launch form takes; a
    # single token.
    (65_536, 100_000, 0.9, 1024, "f32", np.int64, 181),
    (60_000, 20_000, 1.2, 2048, "f32", np.int32, 182),
    (40_000, 300, 1.2, 2048, "bf16", np.int64, 183),
    (300_000, 20_000, 1.2, 1024, "f32", np.int32, 184),
    (20_000, 3000, 1.0, 97, "f32", np.int32, 185),
    (4000, 100, 1.0, 5000, "f32", np.int32, 186),
    (1, 5, 1.0, 16, "f32", np.int32, 187),
]
ADAM_KW = dict(lr=float(np.float32(1e-3)), beta1=float(np.float32(0.9)),
               beta2=float(np.float32(0.999)), eps=float(np.float32(1e-8)),
               weight_decay=float(np.float32(0.01)), step=3)


def _adam_tables(V, D, seed):
    """Parameters and non-zero moments, as a later step sees them."""
    return (synth.normal_rows(V, D, seed, 0.02), synth.normal_rows(V, D, seed + 1, 0.01),
            np.abs(synth.normal_rows(V, D, seed + 2, 0.01)))


@pytest.mark.parametrize("K,V,s,D,gdt,dt,seed", ADAM_CASES,
                         ids=[f"K{c[0]}-V{c[1]}-D{c[3]}-{c[4]}-{np.dtype(c[5]).name}"
                              for c in ADAM_CASES])
def test_segsum_adam_is_segsum_then_adam(lz, K, V, s, D, gdt, dt, seed):
    """lm_segsum_adam on V x D parameter, m and v tables with row_ids = uniq,
    at step 3 with weight decay: the same three tables, bit for bit, as
    lm_segsum followed by lm_sparse_apply Adam with the same arguments (each
    launch form against lm_segsum in that form); every row no type names
    keeps its value in all three."""
    _say(f"segsum_adam K={K} V={V} D={D} {gdt} {np.dtype(dt).name}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, s, D, gdt, dt, seed)
    base = [_t(a) for a in _adam_tables(V, D, seed + 2000)]

    def both():
        out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique,
                        dev_err=res.dev_err)
        want = [b.clone() for b in base]
        lz.sparse_apply(want[0], res.uniq, res.num_unique, out, "adam", m=want[1], v=want[2],
                        dev_err=res.dev_err, **ADAM_KW)
        got = [b.clone() for b in base]
        lz.segsum_adam(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq,
                       got[0], got[1], got[2], dev_err=res.dev_err, **ADAM_KW)
        return want, got

    want, got = both()
    assert lz.segsum_two_launches(True) is False
    try:
        want2, got2 = both()
        torch.cuda.synchronize()
    finally:
        assert lz.segsum_two_launches(False) is True
    lz.check(res.dev_err)
    o = H.assert_unique_matches(res, ids, V, oracle)
    for name, a, b in zip("pmv", got, want):
        assert torch.equal(a, b), f"{name}: not lm_segsum + lm_sparse_apply Adam"
    for name, a, b in zip("pmv", got2, want2):
        assert torch.equal(a, b), f"{name}, two-launch form: not lm_segsum + lm_sparse_apply Adam"
    touched = torch.zeros(V, dtype=torch.bool, device=DEV)
    touched[_t(o[0].astype(np.int64))] = True
    for name, a, b in zip("pmv", got, base):
        assert torch.equal(a[~touched], b[~touched]), f"{name}: a row no type names was updated"


def test_segsum_adam_first_step_matches_oracle(lz):
    """End to end against the oracle's Seg-Sum and lazy Adam: the first step
    from zero moments, every touched row of the three tables within the
    bounds that the Seg-Sum tolerance allows."""
    K, V, D = 60_000, 20_000, 1024
    _say("segsum_adam first step against the oracle")
    ids, grad, tgrad, res = _rows_case(lz, K, V, 1.0, D, "f32", np.int32, 188)
    p0 = synth.normal_rows(V, D, 189, 0.02)
    p, m, v = _t(p0), torch.zeros((V, D), device=DEV), torch.zeros((V, D), device=DEV)
    kw = dict(ADAM_KW, weight_decay=0.0, step=1)
    lz.segsum_adam(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, p, m, v,
                   dev_err=res.dev_err, **kw)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    o = H.assert_unique_matches(res, ids, V, oracle)
    U = len(o[0])
    S = oracle.segsum(grad, o[3], U)
    sq = H.sum_of_squares(grad, o[3], U, oracle)
    z = np.zeros_like(S)
    rp, rm, rv = oracle.adam(p0[o[0]], z, z, S, kw["lr"], kw["beta1"], kw["beta2"], kw["eps"],
                             0.0, 1)
    sel = _t(o[0].astype(np.int64))
    H.assert_adam_first_step(p[sel].cpu().numpy(), m[sel].cpu().numpy(), v[sel].cpu().numpy(),
                             rp, rm, rv, S, kw["lr"], kw["beta1"], kw["beta2"], kw["eps"],
                             H.row_delta(S, H.TOL_F32, sq))


@pytest.mark.parametrize("D", [512, 2048, 5000])
def test_segsum_adam_reads_back_the_sums(lz, D):
    """With beta1 = 0 on zero tables each updated m row is 0 * 0 + 1 * sum,
    the sum itself: lm_segsum_rows's table, bit for bit (how the bench reads
    the sums of its fused Adam step back for the oracle check)."""
    K, V = 30_000, 2000
    _say(f"segsum_adam beta1=0 D={D}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, 1.2, D, "f32", np.int32, 190)
    want = torch.zeros((V, D), device=DEV)
    lz.segsum_rows(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, want,
                   dev_err=res.dev_err)
    p, m, v = (torch.zeros((V, D), device=DEV) for _ in range(3))
    lz.segsum_adam(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, p, m, v,
                   lr=0.0, beta1=0.0, step=1, dev_err=res.dev_err)
    torch.cuda.synchronize()
    lz.check(res.dev_err)
    assert torch.equal(m, want)


@pytest.mark.parametrize("D", [512, 2048])
def test_segsum_adam_bad_row_id(lz, D):
    """A row id outside [0, V) sets LM_DEVERR_ID_RANGE and leaves that row of
    all three tables as it was, as lm_sparse_apply does; the other rows are
    updated as usual (the longest type, finished by the fix-up, and a short
    one, finished in the walk)."""
    K, V = 30_000, 2000
    _say(f"segsum_adam bad ids D={D}")
    ids, grad, tgrad, res = _rows_case(lz, K, V, 1.2, D, "f32", np.int64, 191)
    U = int(res.num_unique.item())
    counts = res.counts[:U].cpu().numpy()
    out = lz.segsum(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, u_cap=U,
                    dev_err=res.dev_err)
    base = [_t(a) for a in _adam_tables(V, D, 192)]
    for bad_u, bad_id in ((int(np.argmax(counts)), V), (int(np.argmin(counts)), -1)):
        rid = res.uniq[:U].clone()
        rid[bad_u] = bad_id
        e_want = torch.zeros(1, dtype=torch.int32, device=DEV)
        want = [b.clone() for b in base]
        lz.sparse_apply(want[0], rid, res.num_unique, out, "adam", m=want[1], v=want[2],
                        dev_err=e_want, **ADAM_KW)
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        got = [b.clone() for b in base]
        lz.segsum_adam(tgrad, res.perm, res.inverse, res.offsets, res.num_unique, rid, got[0],
                       got[1], got[2], dev_err=err, **ADAM_KW)
        torch.cuda.synchronize()
        assert int(err.item()) == lz.DEVERR_ID_RANGE == int(e_want.item()), (bad_u, bad_id)
        for a, b in zip(got, want):
            assert torch.equal(a, b)


def test_segsum_updates_special_inputs(lz):
    """The update variants on degenerate inputs, against lm_segsum followed
    by lm_sparse_apply: no tokens (nothing is touched), a single type (one
    segment across every chunk: the fix-up's head), every id distinct (a
    segment end on every row: each gather batch closes at its last end)."""
    D = 256
    _say("segsum_sgd / segsum_adam special inputs")
    empty = lz.unique(torch.zeros(0, dtype=torch.int32, device=DEV), 10)
    g0 = torch.zeros((0, D), device=DEV)
    t = torch.ones((10, D), device=DEV)
    lz.segsum_sgd(g0, empty.perm, empty.inverse, empty.offsets, empty.num_unique, empty.uniq, t,
                  0.5, dev_err=empty.dev_err)
    pmv = [torch.ones((10, D), device=DEV) for _ in range(3)]
    lz.segsum_adam(g0, empty.perm, empty.inverse, empty.offsets, empty.num_unique, empty.uniq,
                   pmv[0], pmv[1], pmv[2], dev_err=empty.dev_err)
    torch.cuda.synchronize()
    lz.check(empty.dev_err)
    assert all(bool((x == 1).all()) for x in [t] + pmv), "no tokens, yet a row was touched"
    K = 30_000
    g = _t(synth.normal_rows(K, D, 63))
    dist = np.random.Generator(np.random.PCG64(64)).permutation(K).astype(np.int32)
    for ids, V in ((np.full(K, 3, np.int32), 10), (dist, K)):
        res = lz.unique(_t(ids), V)
        out = lz.segsum(g, res.perm, res.inverse, res.offsets, res.num_unique, dev_err=res.dev_err)
        base = _t(synth.normal_rows(V, D, 65))
        want = base.clone()
        lz.sparse_apply(want, res.uniq, res.num_unique, out, "sgd", lr=0.1, dev_err=res.dev_err)
        got = base.clone()
        lz.segsum_sgd(g, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, got, 0.1,
                      dev_err=res.dev_err)
        wa = [base.clone(), torch.zeros_like(base), torch.zeros_like(base)]
        lz.sparse_apply(wa[0], res.uniq, res.num_unique, out, "adam", m=wa[1], v=wa[2],
                        dev_err=res.dev_err, **ADAM_KW)
        ga = [base.clone(), torch.zeros_like(base), torch.zeros_like(base)]
        lz.segsum_adam(g, res.perm, res.inverse, res.offsets, res.num_unique, res.uniq, ga[0],
                       ga[1], ga[2], dev_err=res.dev_err, **ADAM_KW)
        torch.cuda.synchronize()
        lz.check(res.dev_err)
        assert torch.equal(got, want), f"SGD, V={V}"
        assert all(torch.equal(a, b) for a, b in zip(ga, wa)), f"Adam, V={V}"


# ---------------------------------------------------------------------------
# Map, Fill-Values, the G-shard merge
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dt", [np.int32, np.int64])
def test_shard_merge_and_expand(lz, dt):
    """Steps 1-5 for G shards on one GPU: Unique over the concatenation, the
    local->global map, EXPAND of each shard's reduction, and the sum of the
    expansions equals the Seg-Sum of the concatenation (the AllReduce)."""
    G, K, V, D = 6, 7000, 50_000, 136
    shards = [synth.zipf_ids(K, V, 1.0, 80 + g, dt) for g in range(G)]
    grads = [synth.normal_rows(K, D, 90 + g) for g in range(G)]
    I = np.concatenate(shards)
    rI = lz.unique(_t(I), V)
    MI = lz.segsum(_t(np.concatenate(grads)), rI.perm, rI.inverse, rI.offsets, rI.num_unique, dev_err=rI.dev_err)
    total = torch.zeros((rI.uniq.numel(), D), dtype=torch.float64, device=DEV)
    keep = []
    for J, g in zip(shards, grads):
        r = lz.unique(_t(J), V)
        s = lz.segsum(_t(g), r.perm, r.inverse, r.offsets, r.num_unique, dev_err=r.dev_err)
        mp = lz.map_ids(r.uniq, r.num_unique, rI.uniq, rI.num_unique, dev_err=r.dev_err)
        M = torch.full((rI.uniq.numel(), D), float("nan"), device=DEV)
        lz.fill_values(s, r.uniq, r.num_unique, M, rI.uniq, rI.num_unique, "expand", dev_err=r.dev_err)
        total += M.double().nan_to_num(0.0)
        keep.append((J, r, s, mp, M))
    torch.cuda.synchronize()
    lz.check(rI.dev_err)
    oI = H.assert_unique_matches(rI, I, V, oracle)
    UG = len(oI[0])
    for (J, r, s, mp, M), g in zip(keep, grads):
        lz.check(r.dev_err)
        oj = H.assert_unique_matches(r, J, V, oracle)
        Ui = len(oj[0])
        omap, missing = oracle.map_ids(oj[0], oI[0])
        assert not missing and np.array_equal(mp[:Ui].cpu().numpy(), omap)
        Mn = M[:UG].cpu().numpy()
        assert not np.isnan(Mn).any(), "EXPAND must write every row"
        # the oracle's steps 2 and 5 on the same shard
        want = oracle.expand(oracle.segsum(g, oj[3], Ui), oj[0], oI[0])
        others = np.ones(UG, bool)
        others[omap] = False
        assert not Mn[others].any() and not want[others].any()
        assert H.row_rel_err(Mn[omap], want[omap]) <= H.TOL_F32
    ref = oracle.segsum(np.concatenate(grads), oI[3], UG)
    assert H.row_rel_err(total[:UG].cpu().numpy(), ref) <= 2 * H.TOL_F32
    assert H.row_rel_err(MI[:UG].double().cpu().numpy(), ref) <= H.TOL_F32


@pytest.mark.parametrize("dt", [np.int32, np.int64])
def test_fill_modes(lz, dt):
    """Step 5 and the row scatters on seeded source rows (the same arrays go
    to the oracle): every mode is a copy or one fp32 add, so bit-exact."""
    U, V, D = 3000, 40_000, 72
    src_ids = synth.distinct_ids(U, V, 101, dt)
    src = synth.normal_rows(U, D, 102)
    base = synth.normal_rows(V, D, 103)
    n_src = torch.tensor([U], dtype=torch.int64, device=DEV)
    sid, s = _t(src_ids), _t(src)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    t1 = _t(base)
    lz.fill_values(s, sid, n_src, t1, None, None, "scatter", dev_err=err)
    t2 = _t(base)
    lz.fill_values(s, sid, n_src, t2, None, None, "scatter_add", dev_err=err)
    # the row space of a superset id list: scatter, and EXPAND (zero fill)
    sup = np.union1d(src_ids, synth.distinct_ids(9000, V, 104, dt)).astype(dt)
    n_sup = torch.tensor([len(sup)], dtype=torch.int64, device=DEV)
    t3 = torch.zeros((len(sup), D), device=DEV)
    lz.fill_values(s, sid, n_src, t3, _t(sup), n_sup, "scatter", dev_err=err)
    t4 = torch.full((len(sup) + 5, D), float("nan"), device=DEV)
    lz.fill_values(s, sid, n_src, t4, _t(sup), n_sup, "expand", dev_err=err)
    torch.cuda.synchronize()
    lz.check(err)
    s64 = src.astype(np.float64)
    assert np.array_equal(t1.cpu().numpy().astype(np.float64), oracle.scatter(s64, src_ids, base))
    want_add = oracle.scatter(s64, src_ids, base, add=True).astype(np.float32)
    assert np.array_equal(t2.cpu().numpy(), want_add)
    assert np.array_equal(t3.cpu().numpy().astype(np.float64),
                          oracle.scatter(s64, src_ids, np.zeros((len(sup), D)), dst_ids=sup))
    got4 = t4.cpu().numpy()
    assert np.array_equal(got4[:len(sup)].astype(np.float64), oracle.expand(s64, src_ids, sup))
    assert np.isnan(got4[len(sup):]).all(), "EXPAND wrote past the merged rows"


def test_fill_and_map_errors(lz):
    ids = _t(np.array([2, 5, 9], np.int32))
    n3 = torch.tensor([3], dtype=torch.int64, device=DEV)
    sup = _t(np.array([1, 2, 5, 8], np.int32))
    n4 = torch.tensor([4], dtype=torch.int64, device=DEV)
    src = torch.ones((3, 8), device=DEV)
    e1 = torch.zeros(1, dtype=torch.int32, device=DEV)
    mp = lz.map_ids(ids, n3, sup, n4, dev_err=e1)
    e2 = torch.zeros(1, dtype=torch.int32, device=DEV)
    lz.fill_values(src, ids, n3, torch.zeros((4, 8), device=DEV), sup, n4, "expand", dev_err=e2)
    e3 = torch.zeros(1, dtype=torch.int32, device=DEV)
    lz.fill_values(src, ids, n3, torch.zeros((6, 8), device=DEV), None, None, "scatter", dev_err=e3)
    torch.cuda.synchronize()
    assert mp.cpu().tolist() == [1, 2, -1]
    assert int(e1.item()) & lz.DEVERR_NOT_FOUND
    assert int(e2.item()) & lz.DEVERR_NOT_FOUND
    assert int(e3.item()) & lz.DEVERR_ID_RANGE


# ---------------------------------------------------------------------------
# Sparse apply (step 7)
# ---------------------------------------------------------------------------

def _apply_case(lz, opt, dt, U, V, D, seed, step=1, wd=0.0):
    """Step 7 on seeded touched rows and update values (the same arrays go to
    the oracle, which works in fp64)."""
    rows = synth.distinct_ids(U, V, seed, dt)
    g = synth.normal_rows(U, D, seed + 1)
    p0 = synth.normal_rows(V, D, seed + 2, 0.02)
    n_rows = torch.tensor([U], dtype=torch.int64, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    table = _t(p0)
    kw = {}
    m0 = v0 = None
    if opt == "adam":
        m0 = synth.normal_rows(V, D, seed + 3, 0.01) if step > 1 else np.zeros((V, D), np.float32)
        v0 = np.abs(synth.normal_rows(V, D, seed + 4, 0.01)) if step > 1 else np.zeros((V, D), np.float32)
        kw = dict(m=_t(m0), v=_t(v0), step=step)
    # The kernel receives fp32 hyperparameters; the oracle gets the same
    # fp32-rounded values (1 - fp32(0.999) differs from 0.001 by 1.3e-5).
    f32 = lambda x: float(np.float32(x))
    lr = f32(0.1 if opt == "sgd" else 1e-3)
    b1, b2, eps = f32(0.9), f32(0.999), f32(1e-8)
    if opt == "adam":
        kw["weight_decay"] = f32(wd)
    lz.sparse_apply(table, _t(rows), n_rows, _t(g), opt, lr=lr, beta1=b1, beta2=b2, eps=eps,
                    dev_err=err, **kw)
    torch.cuda.synchronize()
    lz.check(err)
    got = table.cpu().numpy()
    untouched = np.ones(V, bool)
    untouched[rows] = False
    assert np.array_equal(got[untouched], p0[untouched]), "untouched rows must be bit-unchanged"
    if opt == "sgd":
        ref = oracle.sgd(p0[rows], g, float(lr))
        np.testing.assert_allclose(got[rows], ref, rtol=0, atol=float(np.abs(ref).max()) * 2.4e-7)
    else:
        pr, mr, vr = oracle.adam(p0[rows], m0[rows], v0[rows], g, lr, b1, b2, eps, f32(wd), step)
        dp = np.abs(got[rows] - pr)
        assert float(dp.max()) <= 2e-6 * float(lr) + 2.4e-7 * float(np.abs(pr).max())
        # Each moment is a two-term fp32 update: its rounding error is bounded
        # by the size of the terms, not of the (possibly cancelling) result.
        u = 2.0 ** -24
        bm = 3 * u * (b1 * np.abs(m0[rows]) + (1 - b1) * np.abs(g.astype(np.float64)))
        bv = 4 * u * (b2 * v0[rows] + (1 - b2) * np.square(g.astype(np.float64)))
        assert (np.abs(kw["m"].cpu().numpy()[rows] - mr) <= bm).all(), "Adam m"
        assert (np.abs(kw["v"].cpu().numpy()[rows] - vr) <= bv).all(), "Adam v"
        assert np.array_equal(kw["m"].cpu().numpy()[untouched], m0[untouched])
        assert np.array_equal(kw["v"].cpu().numpy()[untouched], v0[untouched])


@pytest.mark.parametrize("dt", [np.int32, np.int64])
def test_apply_sgd(lz, dt):
    _apply_case(lz, "sgd", dt, 7_000, 30_000, 256, 111)


@pytest.mark.parametrize("step,wd", [(1, 0.0), (10, 0.0), (10, 0.01)])
def test_apply_adam(lz, step, wd):
    _apply_case(lz, "adam", np.int64, 7_000, 30_000, 200, 121, step, wd)


def test_apply_sgd_odd_width(lz):
    _apply_case(lz, "sgd", np.int32, 900, 2000, 13, 131)


# ---------------------------------------------------------------------------
# Candidate sampler (Sec. III-B)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("V,dt", [(800_000, np.int32), (1, np.int32), (97, np.int32),
                                  (1 << 31, np.int32), ((1 << 40) + 3, np.int64)])
def test_sample_ids(lz, V, dt):
    r = np.random.Generator(np.random.PCG64(401)).bit_generator.random_raw(70_001).astype(np.uint64)
    r[:4] = [0, 2**64 - 1, 2**63, 1]
    out = lz.sample_ids(_t(r.view(np.int64)), V, id_dtype=torch.int32 if dt == np.int32 else torch.int64)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().astype(np.int64), oracle.sample_ids(r, V))
