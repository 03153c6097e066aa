"""Pins of the CPU oracle against facts fixed outside it.

Each ``check_*`` raises AssertionError when the oracle disagrees with the
paper's worked examples, a closed form, an independent library routine, a
brute-force definition or an invariant of the method. The same checks run
against deliberately broken copies of the oracle (test_oracle_mutants.py),
which they must reject.
"""
from __future__ import annotations

import itertools
import json
import math
import os

import numpy as np

import oracle
from paper_1810_10045_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _brute_unique(J):
    """Types of a token list straight from the definition (Python built-ins)."""
    J = [int(x) for x in J]
    uniq = sorted(set(J))
    counts = [J.count(x) for x in uniq]
    inverse = [uniq.index(x) for x in J]
    offsets = [0]
    for c in counts:
        offsets.append(offsets[-1] + c)
    perm = sorted(range(len(J)), key=lambda k: (J[k], k))
    return uniq, counts, offsets, inverse, perm


def _assert_unique_equals(got, want, what=""):
    names = ("uniq", "counts", "offsets", "inverse", "perm")
    for n, g, w in zip(names, got, want):
        assert list(np.asarray(g).tolist()) == list(w), f"{what}: {n} {list(g)} != {list(w)}"


def _int_rows(K, D, seed):
    """Small integer-valued fp32 rows: every fp64 sum of them is exact."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(-50, 51, size=(K, D)).astype(np.float32)


# ----------------------------------------------------------------------------
# Unique (steps 1 and 4)
# ----------------------------------------------------------------------------

def check_to_be_or_not_to_be():
    """Sec. I: "to be or not to be" has four types and six tokens."""
    g = _golden("to_be_or_not_to_be.json")
    words = g["tokens"]
    first = {}
    for w in words:
        first.setdefault(w, len(first))
    for ids in ({w: first[w] for w in first},               # by first appearance
                {"to": 17, "be": 5, "or": 42, "not": 9}):    # shuffled ids
        J = [ids[w] for w in words]
        got = oracle.unique(J, 100)
        uniq, counts = got[0], got[1]
        assert len(uniq) == g["paper_types"]
        assert int(np.sum(counts)) == g["paper_tokens"] == len(J)
        _assert_unique_equals(got, _brute_unique(J), "to be or not to be")


def check_numpy_unique():
    """Against numpy's unique (return_inverse, return_counts) and its stable
    argsort, on Zipf batches of several sizes."""
    for K, V, s, seed in ((1, 5, 1.0, 1), (17, 3, 1.0, 2), (1000, 50, 1.0, 3),
                          (4097, 100_000, 1.0, 4), (20000, 20_000, 1.2, 5),
                          (3000, 2_000_000, 0.9, 6)):
        J = synth.zipf_ids(K, V, s, seed, np.int64)
        uniq, counts, offsets, inverse, perm = oracle.unique(J, V)
        nu, ninv, ncnt = np.unique(J, return_inverse=True, return_counts=True)
        assert np.array_equal(uniq, nu)
        assert np.array_equal(counts, ncnt)
        assert np.array_equal(inverse, ninv.reshape(-1))
        assert np.array_equal(perm, np.argsort(J, kind="stable"))
        assert np.array_equal(offsets, np.concatenate([[0], np.cumsum(ncnt)]))


def check_brute_force_unique():
    """Every token list J in [0, V)^K for small V and K."""
    for V, Kmax in ((1, 5), (2, 5), (3, 5), (4, 6)):
        for K in range(0, Kmax + 1):
            for J in itertools.product(range(V), repeat=K):
                _assert_unique_equals(oracle.unique(list(J), V), _brute_unique(J), f"J={J}")


def check_unique_invariants():
    """Sec. III-A: types are totally ordered, U <= min(K, V), every token maps
    to its own word, and the permutation lists each type's tokens in order."""
    for K, V, s, seed in ((5000, 1000, 1.0, 11), (8192, 100_000, 1.0, 12)):
        J = synth.zipf_ids(K, V, s, seed, np.int64)
        uniq, counts, offsets, inverse, perm = oracle.unique(J, V)
        U = len(uniq)
        assert U <= min(K, V)
        assert np.all(np.diff(uniq) > 0)
        assert np.array_equal(uniq[inverse], J)
        assert int(counts.sum()) == K and np.all(counts >= 1)
        assert np.array_equal(np.diff(offsets), counts)
        assert np.array_equal(np.sort(perm), np.arange(K))
        assert np.all(np.diff(J[perm]) >= 0)
        for u in range(0, U, max(1, U // 50)):
            seg = perm[offsets[u]:offsets[u + 1]]
            assert np.all(J[seg] == uniq[u]) and np.all(np.diff(seg) > 0)


def check_unique_rejects_out_of_range():
    for J, V in (([0, 1, 5], 5), ([-1, 0], 3)):
        try:
            oracle.unique(J, V)
        except oracle.OracleError:
            continue
        raise AssertionError(f"ids {J} with V={V} accepted")


# ----------------------------------------------------------------------------
# Seg-Sum (step 2) and the baseline reverse map (Sec. II-A)
# ----------------------------------------------------------------------------

def check_fig2_i_want_a_pen_and_a():
    """Sec. II-A / Fig. 2: "a" (word 1) at positions 3 and 6 -> rows 3 and 6
    of the gradient accumulate into row 1 of E; "I" is word 4343."""
    g = _golden("i_want_a_pen_and_a.json")
    ids = dict(g["paper_ids"], **g["placeholder_ids"])
    J = [ids[w] for w in g["tokens"]]
    K, D = len(J), 3
    Delta = (np.arange(1, K + 1, dtype=np.float32)[:, None]
             * np.array([1, 10, 100], np.float32)[None, :])
    uniq, counts, offsets, inverse, perm = oracle.unique(J, 10_000)
    assert len(uniq) == 5
    a = int(np.searchsorted(uniq, g["paper_row_of_a"]))
    i = int(np.searchsorted(uniq, g["paper_row_of_I"]))
    assert uniq[a] == 1 and uniq[i] == 4343
    assert counts[a] == 2
    p3, p6 = (p - 1 for p in g["paper_positions_of_a_1based"])
    assert list(perm[offsets[a]:offsets[a + 1]]) == [p3, p6]
    out = oracle.segsum(Delta, inverse, len(uniq))
    assert np.array_equal(out[a], Delta[p3].astype(np.float64) + Delta[p6])
    assert np.array_equal(out[i], Delta[0].astype(np.float64))
    dense = oracle.dense_scatter(Delta, J, 10_000)
    assert np.array_equal(dense[1], out[a]) and np.array_equal(dense[4343], out[i])


def check_segsum_numpy():
    """fp64 accumulation equals numpy's add.at over the same token order
    (fp32 and bf16 gradients)."""
    for K, V, D, s, seed in ((3000, 500, 7, 1.0, 21), (4096, 100_000, 64, 1.0, 22),
                             (2500, 40, 33, 1.2, 23)):
        J = synth.zipf_ids(K, V, s, seed, np.int64)
        G = synth.normal_rows(K, D, seed + 100)
        uniq, counts, offsets, inverse, perm = oracle.unique(J, V)
        for grad, vals in ((G, G), (synth.bf16_bits(G), synth.bf16_to_f32(synth.bf16_bits(G)))):
            want = np.zeros((len(uniq), D), np.float64)
            np.add.at(want, inverse, vals.astype(np.float64))
            got = oracle.segsum(grad, inverse, len(uniq))
            assert np.array_equal(got, want)
            dense = np.zeros((V, D), np.float64)
            np.add.at(dense, J, vals.astype(np.float64))
            assert np.array_equal(oracle.dense_scatter(grad, J, V), dense)


def check_segsum_special_cases():
    """Exact identities on integer-valued rows: column sums are preserved,
    one type gives the column sum, all-distinct ids give the permuted rows,
    and the reduction expanded into V rows is the dense scatter-add with
    every other row zero (Sec. V-A: uniqueness changes how the update is
    computed, not its value)."""
    K, D, V = 777, 19, 300
    G = _int_rows(K, D, 31)
    J = synth.zipf_ids(K, V, 1.0, 32, np.int64)
    uniq, counts, offsets, inverse, perm = oracle.unique(J, V)
    out = oracle.segsum(G, inverse, len(uniq))
    assert np.array_equal(out.sum(0), G.astype(np.float64).sum(0))
    dense = oracle.dense_scatter(G, J, V)
    mask = np.zeros(V, bool)
    mask[uniq] = True
    assert np.array_equal(dense[uniq], out) and np.all(dense[~mask] == 0)
    # a single type
    J1 = np.full(K, 7, np.int64)
    u1 = oracle.unique(J1, V)
    o1 = oracle.segsum(G, u1[3], 1)
    assert np.array_equal(o1[0], G.astype(np.float64).sum(0))
    # every id distinct (a permutation of 0..K-1)
    Jp = np.random.Generator(np.random.PCG64(33)).permutation(K).astype(np.int64)
    up = oracle.unique(Jp, K)
    assert np.array_equal(up[0], np.arange(K)) and np.array_equal(up[3], Jp)
    op = oracle.segsum(G, up[3], K)
    assert np.array_equal(op, G[up[4]].astype(np.float64))
    # empty batch
    u0 = oracle.unique(np.zeros(0, np.int64), V)
    assert len(u0[0]) == 0 and list(u0[2]) == [0]
    assert oracle.segsum(np.zeros((0, D), np.float32), u0[3], 0).shape == (0, D)


def check_segsum_columns():
    """The all-core form of step 2: every column range equals numpy's fp64
    add.at on those columns and leaves the other columns untouched, and any
    split of the columns over threads gives the one-thread result bit for
    bit (each column is summed in the same token order). The row-split
    updates equal their one-thread forms."""
    for K, V, D, s, seed in ((3000, 500, 7, 1.0, 51), (5000, 20_000, 256, 1.2, 52),
                             (700, 40, 1, 1.0, 53)):
        J = synth.zipf_ids(K, V, s, seed, np.int64)
        G = synth.normal_rows(K, D, seed + 100)
        uniq, counts, offsets, inverse, perm = oracle.unique(J, V)
        U = len(uniq)
        for grad, vals in ((G, G), (synth.bf16_bits(G), synth.bf16_to_f32(synth.bf16_bits(G)))):
            one = oracle.segsum(grad, inverse, U)
            for threads in (1, 2, 3, 8):
                assert np.array_equal(oracle.segsum_threads(grad, inverse, U, threads), one)
            d0, d1 = D // 3, D - D // 4
            part = oracle.segsum_cols(grad, inverse, U, d0, d1)
            want = np.zeros((U, d1 - d0), np.float64)
            np.add.at(want, inverse, vals[:, d0:d1].astype(np.float64))
            assert np.array_equal(part[:, d0:d1], want)
            assert np.isnan(part[:, :d0]).all() and np.isnan(part[:, d1:]).all()
        table = synth.normal_rows(V, D, seed + 200, 0.02).astype(np.float64)
        g = oracle.segsum(G, inverse, U)
        assert np.array_equal(oracle.sgd_threads(table[uniq], g, 0.1, 3),
                              oracle.sgd(table[uniq], g, 0.1))
        m0 = np.full((U, D), 0.01)
        a = oracle.adam_threads(table[uniq], m0, m0, g, 1e-3, 0.9, 0.999, 1e-8, 0.0, 3, 5)
        b = oracle.adam(table[uniq], m0, m0, g, 1e-3, 0.9, 0.999, 1e-8, 0.0, 3)
        assert all(np.array_equal(x, y) for x, y in zip(a, b))
        assert np.array_equal(oracle.scatter_threads(g, uniq, table, 4),
                              oracle.scatter(g, uniq, table))


def check_segsum_select():
    K, D, V = 2000, 11, 97
    G = synth.normal_rows(K, D, 41)
    J = synth.zipf_ids(K, V, 1.0, 42, np.int64)
    uniq, counts, offsets, inverse, perm = oracle.unique(J, V)
    full = oracle.segsum(G, inverse, len(uniq))
    assert np.array_equal(oracle.segsum_select(G, J, uniq), full)
    assert np.array_equal(oracle.segsum_select(G, J, uniq[1::3]), full[1::3])
    absent = np.setdiff1d(np.arange(V), uniq)
    if absent.size:
        assert np.all(oracle.segsum_select(G, J, absent[:1]) == 0)


# ----------------------------------------------------------------------------
# Merge across GPUs (steps 3-6 on one host) and Fill-Values (step 5)
# ----------------------------------------------------------------------------

def check_fig3_two_gpus():
    """Sec. II-B / Fig. 3 and Sec. III-A steps 4-6: word 1234 occurs on both
    GPUs; after the merge it is one type that both GPUs map to the same row,
    and the all-reduced row is the sum of both GPUs' rows for it."""
    g = _golden("two_gpu_fig3.json")
    J1 = [g["gpu1_first"]] + g["placeholder_rest"]["gpu1"]
    J2 = [g["gpu2_first"], g["gpu2_second"]] + g["placeholder_rest"]["gpu2"]
    V, D = 10_000, 4
    D1, D2 = _int_rows(len(J1), D, 51), _int_rows(len(J2), D, 52)
    I = J1 + J2
    Ihat = oracle.unique(I, V)[0]
    assert list(Ihat).count(1234) == 1
    row = int(np.searchsorted(Ihat, 1234))
    M = []
    for J, Dl in ((J1, D1), (J2, D2)):
        uj, cj, oj, ij, pj = oracle.unique(J, V)
        mp, missing = oracle.map_ids(uj, Ihat)
        assert not missing
        assert mp[int(np.searchsorted(uj, 1234))] == row
        M.append(oracle.expand(oracle.segsum(Dl, ij, len(uj)), uj, Ihat))
    uI, cI, oI, iI, pI = oracle.unique(I, V)
    Mhat = oracle.segsum(np.concatenate([D1, D2]), iI, len(uI))
    assert np.array_equal(M[0] + M[1], Mhat)
    assert np.array_equal(Mhat[row], D1[0].astype(np.float64) + D2[1])
    # rows of words absent on a GPU are zero in its expansion (step 5)
    for J, Mi in zip((J1, J2), M):
        absent = np.setdiff1d(Ihat, J)
        for w in absent:
            assert np.all(Mi[int(np.searchsorted(Ihat, w))] == 0)


def check_shards_merge():
    """Steps 3-6 with G shards: the sum of the expanded local reductions
    equals the reduction of the concatenated batch (exact on integers)."""
    G_, K, V, D = 5, 300, 400, 6
    shards = [synth.zipf_ids(K, V, 1.0, 60 + g, np.int64) for g in range(G_)]
    rows = [_int_rows(K, D, 70 + g) for g in range(G_)]
    I = np.concatenate(shards)
    uI, cI, oI, iI, pI = oracle.unique(I, V)
    total = np.zeros((len(uI), D))
    for J, R in zip(shards, rows):
        uj, cj, oj, ij, pj = oracle.unique(J, V)
        assert len(uj) <= len(uI) <= G_ * K
        mp, missing = oracle.map_ids(uj, uI)
        assert not missing and np.array_equal(uI[mp], uj)
        total += oracle.expand(oracle.segsum(R, ij, len(uj)), uj, uI)
    assert np.array_equal(total, oracle.segsum(np.concatenate(rows), iI, len(uI)))


def check_map_and_fill():
    """map = numpy searchsorted on present ids; missing ids flagged; expand
    writes every destination row (zero where absent); scatter writes or adds
    only the named rows."""
    sup = np.array([2, 3, 5, 8, 13, 21, 34], np.int64)
    sub = np.array([3, 8, 34], np.int64)
    mp, missing = oracle.map_ids(sub, sup)
    assert not missing and list(mp) == list(np.searchsorted(sup, sub))
    mp2, missing2 = oracle.map_ids(np.array([4], np.int64), sup)
    assert missing2 and mp2[0] == -1
    D = 3
    src = np.array([[1, 2, 3], [4, 5, 6], [7, 8, 9]], np.float64)
    ex = oracle.expand(src, sub, sup)
    want = np.zeros((len(sup), D))
    want[[1, 3, 6]] = src
    assert np.array_equal(ex, want)
    base = np.arange(40 * D, dtype=np.float64).reshape(40, D)
    sc = oracle.scatter(src, sub, base)
    w = base.copy()
    w[sub] = src
    assert np.array_equal(sc, w)
    sa = oracle.scatter(src, sub, base, add=True)
    w = base.copy()
    w[sub] += src
    assert np.array_equal(sa, w)
    dsc = oracle.scatter(src, sub, np.zeros((len(sup), D)), dst_ids=sup)
    assert np.array_equal(dsc, want)


# ----------------------------------------------------------------------------
# Update (step 7)
# ----------------------------------------------------------------------------

def check_sgd():
    p = np.array([[1.0, -2.0], [0.5, 4.0]])
    g = np.array([[2.0, 2.0], [-1.0, 0.0]])
    assert np.array_equal(oracle.sgd(p, g, 0.25), np.array([[0.5, -2.5], [0.75, 4.0]]))


def check_adam_closed_forms():
    rng = np.random.Generator(np.random.PCG64(81))
    p = rng.standard_normal((4, 5))
    g = rng.standard_normal((4, 5))
    z = np.zeros_like(p)
    lr, b1, b2, eps = 0.01, 0.9, 0.999, 0.5
    # t = 1 from zero moments: the bias corrections make m^ = g, v^ = g^2
    pn, m, v = oracle.adam(p, z, z, g, lr, b1, b2, eps, 0.0, 1)
    assert np.allclose(pn, p - lr * g / (np.abs(g) + eps), rtol=1e-13, atol=1e-15)
    assert np.allclose(m, (1 - b1) * g, rtol=1e-15) and np.allclose(v, (1 - b2) * g * g, rtol=1e-15)
    # beta1 = beta2 = 0: the moments are the last gradient at any step
    pn, m, v = oracle.adam(p, p, p, g, lr, 0.0, 0.0, eps, 0.0, 10)
    assert np.allclose(pn, p - lr * g / (np.abs(g) + eps), rtol=1e-13, atol=1e-15)
    # zero gradient and moments: only the decoupled weight decay acts
    pn, m, v = oracle.adam(p, z, z, z, lr, b1, b2, eps, 0.1, 3)
    assert np.allclose(pn, p * (1 - lr * 0.1), rtol=1e-15)
    # odd symmetry in (g, m)
    m0 = rng.standard_normal((4, 5))
    v0 = rng.random((4, 5))
    a = oracle.adam(z, m0, v0, g, lr, b1, b2, 1e-8, 0.0, 7)[0]
    b = oracle.adam(z, -m0, v0, -g, lr, b1, b2, 1e-8, 0.0, 7)[0]
    assert np.allclose(a, -b, rtol=1e-15, atol=0)
    # a late step: bias corrections -> 1; one step from (m0, v0) by hand on
    # one element, written from the update rule's definition
    t = 10_000
    pn, m, v = oracle.adam(p, m0, v0, g, lr, b1, b2, 1e-8, 0.0, t)
    e_m = b1 * m0[1, 2] + (1 - b1) * g[1, 2]
    e_v = b2 * v0[1, 2] + (1 - b2) * g[1, 2] ** 2
    e_p = p[1, 2] - lr * (e_m / (1 - b1 ** t)) / (math.sqrt(e_v / (1 - b2 ** t)) + 1e-8)
    assert math.isclose(pn[1, 2], e_p, rel_tol=1e-12)


# ----------------------------------------------------------------------------
# Closed form of the paper's memory example (reading of the text)
# ----------------------------------------------------------------------------

def check_memory_example():
    """Sec. III-A worked example: 35.2 GB for the AllGather of gradients vs
    0.137 GB with uniqueness, a 256x saving, at K = 19,200, D = 1792, G = 256,
    with U_g = (G K)^0.64."""
    g = _golden("memory_example.json")
    K = g["c"] * g["seqs_per_gpu"]
    assert K == 19_200
    ag = g["G"] * K * g["D"] * g["bytes_per_value"] / 1e9
    Ug = (g["G"] * K) ** g["alpha"]
    un = Ug * g["D"] * g["bytes_per_value"] / 1e9
    assert round(ag, 1) == g["paper_allgather_GB"]
    assert round(un, 3) == g["paper_uniqueness_GB"]
    assert round(ag / un) == g["paper_saving_x"]


def check_f16_conversion():
    """Sec. III-C binary16 casts against numpy's (IEEE round to nearest even):
    every binary16 pattern widens to numpy's value and narrows back to itself;
    random fp32 values over 57 binades, and the exact midpoints between
    neighbouring binary16 values (normal and subnormal), narrow like numpy."""
    allh = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    wide = oracle.f32_from_f16(allh)
    ref = allh.view(np.float16).astype(np.float32)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(wide), nan)
    assert np.array_equal(wide[~nan].view(np.uint32), ref[~nan].view(np.uint32))
    back = oracle.f16_from_f32(wide)
    assert np.array_equal(back[~nan], allh[~nan])
    assert np.all((back[nan] & 0x7C00) == 0x7C00) and np.all((back[nan] & 0x3FF) != 0)
    rng = np.random.default_rng(61)
    mag = np.exp2(rng.uniform(-40, 17, size=200_000)).astype(np.float32)
    x = np.where(rng.random(mag.size) < 0.5, -mag, mag).astype(np.float32)
    with np.errstate(over="ignore"):
        want = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(oracle.f16_from_f32(x), want)
    # exact midpoints: ties go to the even neighbour
    fin = ref[np.isfinite(ref) & (ref >= 0)]
    fin = np.unique(fin)
    mid = ((fin[:-1].astype(np.float64) + fin[1:].astype(np.float64)) / 2).astype(np.float32)
    assert np.array_equal(mid.astype(np.float64), (fin[:-1].astype(np.float64) + fin[1:]) / 2)
    with np.errstate(over="ignore"):
        assert np.array_equal(oracle.f16_from_f32(mid), mid.astype(np.float16).view(np.uint16))


def check_compression():
    """Sec. III-C compression-scaling: with a power-of-two F the product is
    exact, so the payload equals numpy's binary16 of x*F and the round trip
    errs by at most 2^-11 |x| while |x F| stays in the normal range; past
    65504 the code saturates to infinity; with any other F the product is
    rounded to fp32 before the cast."""
    rng = np.random.default_rng(62)
    x32 = (rng.standard_normal((300, 40)) * 0.01).astype(np.float32)
    for F in (1.0, 256.0, 1024.0):
        h = oracle.compress(x32.astype(np.float64), F)
        assert np.array_equal(h, (x32 * np.float32(F)).astype(np.float16).view(np.uint16))
        back = oracle.decompress(h, 1.0 / F)
        big = np.abs(x32 * F) >= 2.0 ** -14
        assert np.all(np.abs(back - x32)[big] <= 2.0 ** -11 * np.abs(x32)[big])
        assert np.all(np.abs(back - x32)[~big] <= 2.0 ** -25 / F)
    F = 3.0
    prod = x32 * np.float32(F)
    assert np.array_equal(oracle.compress(x32.astype(np.float64), F),
                          prod.astype(np.float16).view(np.uint16))
    over = np.array([[65519.0 / 256, 65521.0 / 256, -70000.0 / 256, 1e9]], np.float64)
    h = oracle.compress(over, 256.0)
    assert h.tolist() == [[0x7BFF, 0x7C00, 0xFC00, 0x7C00]]
    assert np.all(np.isinf(oracle.decompress(h[:, 1:], 1 / 256.0)))


def check_sample_ids():
    """Sec. III-B uniform candidate sampler: with V = 2^k an id is the top k
    bits of r; 40 V values of r spaced evenly over [0, 2^64) land 40 +- 1
    times on every id, monotonically; and each id equals the exact integer
    floor(r * V / 2^64) (Python's big integers)."""
    rng = np.random.default_rng(71)
    r = rng.integers(0, 2**63, size=5000, dtype=np.uint64) * np.uint64(2) + \
        rng.integers(0, 2, size=5000, dtype=np.uint64)
    for k in (1, 7, 20, 33):
        assert np.array_equal(oracle.sample_ids(r, 1 << k), (r >> np.uint64(64 - k)).astype(np.int64))
    for V in (3, 10, 97, 1021, 800_000):
        if V < 10_000:
            sweep = (np.arange(V * 40, dtype=np.uint64) * np.uint64((2**64 - 1) // (V * 40)))
            ids = oracle.sample_ids(sweep, V)
            assert np.all(np.diff(ids) >= 0) and ids.min() == 0 and ids.max() == V - 1
            c = np.bincount(ids, minlength=V)
            assert np.all(np.abs(c - 40) <= 1)
        exact = [(int(x) * V) >> 64 for x in r[:300]]
        assert oracle.sample_ids(r[:300], V).tolist() == exact
    assert oracle.sample_ids(np.array([0, 2**64 - 1], np.uint64), 5).tolist() == [0, 4]


ALL_CHECKS = [
    check_to_be_or_not_to_be, check_numpy_unique, check_brute_force_unique,
    check_unique_invariants, check_unique_rejects_out_of_range,
    check_fig2_i_want_a_pen_and_a, check_segsum_numpy, check_segsum_special_cases,
    check_segsum_columns, check_segsum_select, check_fig3_two_gpus, check_shards_merge, check_map_and_fill,
    check_sgd, check_adam_closed_forms, check_f16_conversion, check_compression,
    check_sample_ids,
]
