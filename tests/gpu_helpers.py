"""Shared helpers of the GPU parity tests (no test functions here)."""
from __future__ import annotations

import numpy as np

# Per-row normwise tolerances of Seg-Sum against the fp64 oracle:
#   max_d |got[u,d] - ref[u,d]| / scale[u],
#   scale[u] = max( max_d |ref[u,d]|,  sqrt(mean_d sum_k grad[k,d]^2) )
# The element-wise relative error is ill-posed here (sums of N(0,1) values
# land near zero), so each row is scaled by its largest entry, floored at the
# root-mean-square size of its summands so that a narrow row (D = 1) whose
# sum happens to cancel is not judged relative to a near-zero number.
# fp32 rows: 1e-5; bf16 inputs are widened exactly, so only the fp32
# accumulation differs, and the looser 2e-3 bound is kept for them.
TOL_F32 = 1e-5
TOL_BF16 = 2e-3


def row_rel_err(got: np.ndarray, ref: np.ndarray, sumsq: np.ndarray = None) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    scale = np.abs(ref).max(axis=1)
    if sumsq is not None:
        scale = np.maximum(scale, np.sqrt(np.asarray(sumsq, np.float64).mean(axis=1)))
    err = np.abs(got - ref).max(axis=1)
    zero = scale == 0
    assert np.all(err[zero] == 0), "rows whose summands are all zero must be exactly zero"
    if not (~zero).any():
        return 0.0
    return float((err[~zero] / scale[~zero]).max())


def unique_to_numpy(res, K):
    U = int(res.num_unique.item())
    return (U, res.uniq[:U].cpu().numpy().astype(np.int64), res.counts[:U].cpu().numpy(),
            res.offsets[:U + 1].cpu().numpy(), res.inverse[:K].cpu().numpy(),
            res.perm[:K].cpu().numpy())


def assert_unique_matches(res, ids_np, V, oracle, what=""):
    K = len(ids_np)
    U, uniq, counts, offsets, inverse, perm = unique_to_numpy(res, K)
    o = oracle.unique(ids_np, V)
    assert U == len(o[0]), f"{what}: U {U} != {len(o[0])}"
    assert np.array_equal(uniq, o[0]), f"{what}: uniq"
    assert np.array_equal(counts, o[1]), f"{what}: counts"
    assert np.array_equal(offsets, o[2]), f"{what}: offsets"
    if K:
        assert np.array_equal(inverse, o[3]), f"{what}: inverse"
        assert np.array_equal(perm, o[4]), f"{what}: perm"
    return o


def sum_of_squares(grad, inverse, U, oracle):
    """U x D fp64 sums of the squared gradient values of every type (the
    floor of the row scale above), through the oracle's own reduction."""
    g = np.asarray(grad)
    vals = (g.astype(np.uint32) << np.uint32(16)).view(np.float32) if g.dtype == np.uint16 else g
    return oracle.segsum(np.square(vals, dtype=np.float32), inverse, U)
