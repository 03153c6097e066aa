"""CPU oracle for the Zipf gradient-compression path (arXiv:1810.10045).

TEST INFRASTRUCTURE ONLY: the plain fp64 reference that the GPU library is
checked against. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the product package never
does, and the two share no code. The arithmetic lives in ``lmoracle.c`` (one
routine per step of Sec. III-A of the paper); this module only marshals numpy
arrays into it.

Parity status per routine (what pins it lives in ``tests/test_oracle_pins.py``):
  unique          pinned (worked examples, numpy, brute force, invariants)
  segsum          pinned (worked examples, fp64 numpy accumulation, dense
                  scatter, column sums, special cases)
  segsum_select   pinned (equal to segsum rows)
  segsum_cols,
  segsum_threads  pinned (equal to segsum bit for bit, any column split;
                  numpy add.at on a column range)
  dense_scatter   pinned (numpy ``add.at``)
  map, expand,
  scatter         pinned (worked two-GPU example, numpy, invariants)
  sgd, adam       pinned (closed forms: t = 1 with zero moments, one step by
                  hand, bias-correction limits)
  f16_from_f32,
  f32_from_f16,
  compress,
  decompress      pinned (numpy's float16 conversion, every binary16 pattern
                  round-tripped, overflow / subnormal / tie cases, power-of-two
                  scales exact)
  sample_ids      pinned (V a power of two: the top bits; exact run lengths of
                  every id for small V over an evenly spaced sweep of r;
                  monotone in r; Python's exact integer product)
"""
from __future__ import annotations

import contextlib
import ctypes
import os

import numpy as np

from .build import build as _build, LIB_PATH

_lib = None
_override = None

OK, BADARG, RANGE, NOTFOUND = 0, 1, 2, 3
F32, BF16 = 0, 1


class OracleError(RuntimeError):
    pass


def _declare(L):
    P = ctypes.c_void_p
    I = ctypes.c_int64
    L.orc_unique.argtypes = [P, I, I, P, P, P, P, P, P]
    L.orc_segsum.argtypes = [P, ctypes.c_int, I, I, I, P, I, P]
    L.orc_segsum_cols.argtypes = [P, ctypes.c_int, I, I, I, P, I, I, I, P]
    L.orc_segsum_select.argtypes = [P, ctypes.c_int, I, I, I, P, P, I, P]
    L.orc_dense_scatter.argtypes = [P, ctypes.c_int, I, I, I, P, I, P]
    L.orc_map.argtypes = [P, I, P, I, P]
    L.orc_expand.argtypes = [P, I, I, P, P, I, P]
    L.orc_scatter.argtypes = [P, I, I, P, P, I, P, I, ctypes.c_int]
    L.orc_sgd.argtypes = [P, P, I, I, ctypes.c_double]
    L.orc_adam.argtypes = [P, P, P, P, I, I] + [ctypes.c_double] * 5 + [I]
    L.orc_f16_from_f32.argtypes = [P, I, P]
    L.orc_f32_from_f16.argtypes = [P, I, P]
    L.orc_compress.argtypes = [P, I, I, ctypes.c_float, P]
    L.orc_decompress.argtypes = [P, I, I, ctypes.c_float, P]
    L.orc_sample_ids.argtypes = [P, I, I, P]
    for f in ("orc_unique", "orc_segsum", "orc_segsum_cols", "orc_segsum_select",
              "orc_dense_scatter", "orc_map", "orc_expand", "orc_scatter",
              "orc_sgd", "orc_adam", "orc_f16_from_f32", "orc_f32_from_f16",
              "orc_compress", "orc_decompress", "orc_sample_ids"):
        getattr(L, f).restype = ctypes.c_int
    return L


def lib():
    """Load ``liblmoracle.so``, compiling it with gcc only if it is absent."""
    global _lib
    if _override is not None:
        return _override
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            _build()
        _lib = _declare(ctypes.CDLL(LIB_PATH))
    return _lib


@contextlib.contextmanager
def loaded_from(path: str):
    """Run the oracle from another build of ``lmoracle.c`` (used by the tests
    that plant a mistake in a copy of the oracle and expect the pins to fail)."""
    global _override
    prev = _override
    _override = _declare(ctypes.CDLL(path))
    try:
        yield
    finally:
        _override = prev


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != OK:
        raise OracleError(f"{what}: oracle status {rc}")


def _ids(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.int64)


def _grad(g: np.ndarray):
    """Return (array, dtype code, row stride). bf16 arrives as uint16 bits."""
    g = np.asarray(g)
    if g.dtype == np.float32:
        code = F32
    elif g.dtype == np.uint16:
        code = BF16
    else:
        raise OracleError(f"gradient dtype {g.dtype} (want float32 or bf16 bits as uint16)")
    if g.ndim != 2:
        raise OracleError("gradient must be K x D")
    if not g.flags.c_contiguous:
        g = np.ascontiguousarray(g)
    return g, code, g.shape[1]


def unique(J, V: int):
    """Steps 1/4: returns (uniq int64, counts, offsets, inverse, perm) (int32)."""
    J = _ids(J)
    K = J.size
    cap = max(K, 1)
    # Outputs start poisoned (-7 / NaN) so that a value the oracle forgets to
    # write cannot pass for a correct zero.
    uniq = np.full(cap, -7, np.int64)
    counts = np.full(cap, -7, np.int32)
    offsets = np.full(cap + 1, -7, np.int32)
    inverse = np.full(cap, -7, np.int32)
    perm = np.full(cap, -7, np.int32)
    U = ctypes.c_int64(0)
    _check(lib().orc_unique(_p(J), K, V, _p(uniq), _p(counts), _p(offsets),
                            _p(inverse), _p(perm), ctypes.byref(U)), "unique")
    n = U.value
    return (uniq[:n].copy(), counts[:n].copy(), offsets[:n + 1].copy(),
            inverse[:K].copy(), perm[:K].copy())


def segsum(grad, inverse, U: int) -> np.ndarray:
    """Step 2: U x D fp64 sums of the gradient rows of each type."""
    g, code, D = _grad(grad)
    inv = np.ascontiguousarray(inverse, dtype=np.int32)
    out = np.full((U, D), np.nan)
    _check(lib().orc_segsum(_p(g), code, g.shape[0], D, D, _p(inv), U, _p(out)), "segsum")
    return out


def segsum_cols(grad, inverse, U: int, d0: int, d1: int, out=None) -> np.ndarray:
    """Step 2 over the columns [d0, d1) of a U x D fp64 matrix ``out`` (a new
    NaN-filled one when None); the other columns are left as they are."""
    g, code, D = _grad(grad)
    inv = np.ascontiguousarray(inverse, dtype=np.int32)
    if out is None:
        out = np.full((U, D), np.nan)
    if out.shape != (U, D) or out.dtype != np.float64 or not out.flags.c_contiguous:
        raise OracleError("segsum_cols: out must be a C-contiguous U x D float64 matrix")
    _check(lib().orc_segsum_cols(_p(g), code, g.shape[0], D, D, _p(inv), U, d0, d1, _p(out)),
           "segsum_cols")
    return out


def column_ranges(D: int, parts: int):
    """[d0, d1) ranges that split D columns into ``parts`` near-equal pieces
    (empty pieces dropped)."""
    parts = max(1, min(parts, max(D, 1)))
    edges = [D * i // parts for i in range(parts + 1)]
    return [(edges[i], edges[i + 1]) for i in range(parts) if edges[i + 1] > edges[i]]


def segsum_threads(grad, inverse, U: int, threads: int) -> np.ndarray:
    """Step 2 with the D columns split over ``threads`` threads, each running
    orc_segsum_cols on its own range (the all-core CPU baseline). The ctypes
    calls release the GIL, so the threads run in parallel; no two write the
    same element, and each column is summed in the same token order as
    segsum, so the result equals it bit for bit."""
    from concurrent.futures import ThreadPoolExecutor
    g, code, D = _grad(grad)
    inv = np.ascontiguousarray(inverse, dtype=np.int32)
    out = np.full((U, D), np.nan)
    ranges = column_ranges(D, threads)
    if len(ranges) <= 1:
        return segsum_cols(g, inv, U, 0, D, out)
    with ThreadPoolExecutor(len(ranges)) as ex:
        list(ex.map(lambda r: segsum_cols(g, inv, U, r[0], r[1], out), ranges))
    return out


def segsum_select(grad, J, sel) -> np.ndarray:
    """Step 2 evaluated only for the word ids in ``sel`` (strictly ascending)."""
    g, code, D = _grad(grad)
    J = _ids(J)
    sel = _ids(sel)
    out = np.full((sel.size, D), np.nan)
    _check(lib().orc_segsum_select(_p(g), code, g.shape[0], D, D, _p(J),
                                   _p(sel), sel.size, _p(out)), "segsum_select")
    return out


def dense_scatter(grad, J, V: int) -> np.ndarray:
    """Sec. II-A baseline: V x D fp64, every token's row added at its word."""
    g, code, D = _grad(grad)
    J = _ids(J)
    out = np.full((V, D), np.nan)
    _check(lib().orc_dense_scatter(_p(g), code, g.shape[0], D, D, _p(J), V, _p(out)),
           "dense_scatter")
    return out


def map_ids(sub, sup):
    """Step 4 map J^ -> I^: int32 positions, -1 where missing; also a flag."""
    sub = _ids(sub)
    sup = _ids(sup)
    m = np.full(max(sub.size, 1), -7, np.int32)
    rc = lib().orc_map(_p(sub), sub.size, _p(sup), sup.size, _p(m))
    if rc not in (OK, NOTFOUND):
        _check(rc, "map")
    return m[:sub.size].copy(), rc == NOTFOUND


def expand(src, src_ids, dst_ids) -> np.ndarray:
    """Step 5: zero-filled len(dst_ids) x D fp64 matrix."""
    src = np.ascontiguousarray(src, dtype=np.float64)
    src_ids = _ids(src_ids)
    dst_ids = _ids(dst_ids)
    D = src.shape[1]
    dst = np.full((dst_ids.size, D), np.nan)
    _check(lib().orc_expand(_p(src), src_ids.size, D, _p(src_ids), _p(dst_ids),
                            dst_ids.size, _p(dst)), "expand")
    return dst


def scatter(src, src_ids, dst, dst_ids=None, add: bool = False) -> np.ndarray:
    """Row write / accumulate into a copy of ``dst`` (fp64)."""
    src = np.ascontiguousarray(src, dtype=np.float64)
    src_ids = _ids(src_ids)
    out = np.array(dst, dtype=np.float64, copy=True, order="C")
    D = src.shape[1]
    if dst_ids is None:
        rc = lib().orc_scatter(_p(src), src_ids.size, D, _p(src_ids), None, 0,
                               _p(out), out.shape[0], int(add))
    else:
        dst_ids = _ids(dst_ids)
        rc = lib().orc_scatter(_p(src), src_ids.size, D, _p(src_ids), _p(dst_ids),
                               dst_ids.size, _p(out), out.shape[0], int(add))
    _check(rc, "scatter")
    return out


def sgd(p, g, lr: float) -> np.ndarray:
    """Step 7, SGD, on the touched rows (fp64 copy returned)."""
    p = np.array(p, dtype=np.float64, copy=True, order="C")
    g = np.ascontiguousarray(g, dtype=np.float64)
    n, D = p.shape
    _check(lib().orc_sgd(_p(p), _p(g), n, D, lr), "sgd")
    return p


def adam(p, m, v, g, lr, beta1, beta2, eps, weight_decay, step):
    """Step 7, lazy Adam, on the touched rows: returns fp64 (p, m, v)."""
    p = np.array(p, dtype=np.float64, copy=True, order="C")
    m = np.array(m, dtype=np.float64, copy=True, order="C")
    v = np.array(v, dtype=np.float64, copy=True, order="C")
    g = np.ascontiguousarray(g, dtype=np.float64)
    n, D = p.shape
    _check(lib().orc_adam(_p(p), _p(m), _p(v), _p(g), n, D, lr, beta1, beta2,
                          eps, weight_decay, step), "adam")
    return p, m, v


def _row_parts(n: int, threads: int):
    parts = max(1, min(threads, max(n, 1)))
    edges = [n * i // parts for i in range(parts + 1)]
    return [(edges[i], edges[i + 1]) for i in range(parts) if edges[i + 1] > edges[i]]


def _run_parts(fn, parts):
    from concurrent.futures import ThreadPoolExecutor
    if len(parts) <= 1:
        for r in parts:
            fn(r)
        return
    with ThreadPoolExecutor(len(parts)) as ex:
        list(ex.map(fn, parts))


def sgd_threads(p, g, lr: float, threads: int) -> np.ndarray:
    """sgd with the rows split over ``threads`` threads (each row is updated
    on its own, so the result equals sgd exactly)."""
    p = np.array(p, dtype=np.float64, copy=True, order="C")
    g = np.ascontiguousarray(g, dtype=np.float64)
    n, D = p.shape

    def part(r):
        _check(lib().orc_sgd(_p(p[r[0]:r[1]]), _p(g[r[0]:r[1]]), r[1] - r[0], D, lr), "sgd")
    _run_parts(part, _row_parts(n, threads))
    return p


def adam_threads(p, m, v, g, lr, beta1, beta2, eps, weight_decay, step, threads: int):
    """adam with the rows split over ``threads`` threads (equal to adam)."""
    p = np.array(p, dtype=np.float64, copy=True, order="C")
    m = np.array(m, dtype=np.float64, copy=True, order="C")
    v = np.array(v, dtype=np.float64, copy=True, order="C")
    g = np.ascontiguousarray(g, dtype=np.float64)
    n, D = p.shape

    def part(r):
        a, b = r
        _check(lib().orc_adam(_p(p[a:b]), _p(m[a:b]), _p(v[a:b]), _p(g[a:b]), b - a, D, lr,
                              beta1, beta2, eps, weight_decay, step), "adam")
    _run_parts(part, _row_parts(n, threads))
    return p, m, v


def scatter_threads(src, src_ids, dst, threads: int) -> np.ndarray:
    """SCATTER of src rows into a copy of the dense table ``dst`` (row = id),
    the source rows split over ``threads`` threads; the ids are distinct, so
    no two threads write the same row (equal to scatter with dst_ids None)."""
    src = np.ascontiguousarray(src, dtype=np.float64)
    src_ids = _ids(src_ids)
    out = np.array(dst, dtype=np.float64, copy=True, order="C")
    D = src.shape[1]

    def part(r):
        a, b = r
        _check(lib().orc_scatter(_p(src[a:b]), b - a, D, _p(src_ids[a:b]), None, 0, _p(out),
                                 out.shape[0], 0), "scatter")
    _run_parts(part, _row_parts(src_ids.size, threads))
    return out


def f16_from_f32(x) -> np.ndarray:
    """Sec. III-C: binary16 bits of fp32 values, round to nearest even."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.full(x.shape, 0xDEAD, np.uint16)
    _check(lib().orc_f16_from_f32(_p(x), x.size, _p(out)), "f16_from_f32")
    return out


def f32_from_f16(h) -> np.ndarray:
    """Exact fp32 values of binary16 bit patterns."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.full(h.shape, np.nan, np.float32)
    _check(lib().orc_f32_from_f16(_p(h), h.size, _p(out)), "f32_from_f16")
    return out


def compress(x, scale: float) -> np.ndarray:
    """Sec. III-C compression of an n x D payload: binary16(fp32(x) * F)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    n, D = x.shape
    out = np.full((n, D), 0xDEAD, np.uint16)
    _check(lib().orc_compress(_p(x), n, D, float(scale), _p(out)), "compress")
    return out


def decompress(h, inv_scale: float) -> np.ndarray:
    """Sec. III-C decompression: fp32(binary16) * (1/F), as fp64."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    n, D = h.shape
    out = np.full((n, D), np.nan)
    _check(lib().orc_decompress(_p(h), n, D, float(inv_scale), _p(out)), "decompress")
    return out


def sample_ids(r, V: int) -> np.ndarray:
    """Sec. III-B sampler: ids floor(r * V / 2^64) of 64-bit random words."""
    r = np.ascontiguousarray(r, dtype=np.uint64)
    out = np.full(r.shape, -7, np.int64)
    _check(lib().orc_sample_ids(_p(r), r.size, V, _p(out)), "sample_ids")
    return out
