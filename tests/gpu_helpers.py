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
# fp32 rows: 1e-5. bf16 rows: the contract allows 2e-3, but the inputs are
# widened to fp32 exactly, on the GPU and in the oracle alike, so only the
# fp32 accumulation differs and the fp32 bound holds for them as well; both
# are asserted (check_rows). At 2e-3 alone a lost or doubled token in a head
# of ~150K tokens, about 1 / (3 sqrt(150K)) = 9e-4 of its row maximum, could
# pass unseen.
TOL_F32 = 1e-5
TOL_BF16 = 2e-3


def check_rows(got, ref, sumsq=None, gdt="f32", what="segsum"):
    """Per-row normwise error of Seg-Sum rows against the oracle: within the
    contract for the gradient dtype, and within the fp32 accumulation bound
    for every dtype. Returns the error."""
    err = row_rel_err(got, ref, sumsq)
    print(f"  {what}: {len(ref)} rows, max row-relative error {err:.3e}", flush=True)
    assert err <= (TOL_BF16 if gdt == "bf16" else TOL_F32), f"{what}: {err:.3e} above the contract"
    assert err <= TOL_F32, f"{what}: {err:.3e} above the fp32 accumulation bound"
    return err


def assert_single_rows_exact(got, ref, counts, what="segsum"):
    """A type with one token sums one value: its row must be that value,
    bit for bit (no rounding can occur)."""
    ones = np.asarray(counts) == 1
    assert np.array_equal(np.asarray(got, np.float64)[ones], np.asarray(ref)[ones]), \
        f"{what}: count-1 rows must be exact copies"


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


# ---------------------------------------------------------------------------
# End-to-end bounds: the GPU's update computed from its own Seg-Sum against
# the oracle's update computed from the oracle's Seg-Sum. delta[u] bounds
# |S_gpu[u,d] - S_ref[u,d]| (the Seg-Sum tolerance times the row scale); the
# rest is fp32 rounding of the update itself, with unit roundoff U32.
# ---------------------------------------------------------------------------
U32 = 2.0 ** -24


def row_delta(S_ref, tol, sumsq=None):
    """Per-row bound on the Seg-Sum error allowed by the row tolerance."""
    scale = np.abs(S_ref).max(axis=1)
    if sumsq is not None:
        scale = np.maximum(scale, np.sqrt(np.asarray(sumsq, np.float64).mean(axis=1)))
    return tol * scale


def assert_sgd_rows(got, ref, S_ref, lr, delta):
    """ref = oracle.sgd(p0, S_ref, lr). The GPU subtracts fl(lr * S_gpu)
    from p0 and rounds: |got - ref| <= lr*delta + 2u(|ref| + lr|S_ref|)."""
    got = np.asarray(got, np.float64)
    bound = (lr * delta[:, None] + 2 * U32 * (np.abs(ref) + lr * (np.abs(S_ref) + delta[:, None])))
    bad = np.abs(got - ref) > bound * 1.01 + 1e-30
    assert not bad.any(), f"SGD rows: {int(bad.sum())} values outside the bound, first at {np.argwhere(bad)[0]}"


def assert_adam_first_step(got_p, got_m, got_v, ref_p, ref_m, ref_v, S_ref, lr, b1, b2, eps, delta):
    """First lazy-Adam step from zero moments (t = 1, no weight decay):
    m = (1-b1) g, v = (1-b2) g^2 and the update lr * g / (|g| + eps).
    Where |g| > 2 delta the update moves by at most lr*delta*eps/(|g|-delta)^2
    under a perturbation of g by delta; where |g| <= 2 delta its sign is not
    determined by the tolerance and any update in [-lr, lr] is accepted."""
    d = delta[:, None]
    g = np.abs(S_ref)
    got_p, got_m, got_v = (np.asarray(a, np.float64) for a in (got_p, got_m, got_v))
    bm = (1 - b1) * d + 8 * U32 * np.abs(ref_m)
    assert (np.abs(got_m - ref_m) <= bm * 1.01 + 1e-38).all(), "Adam m"
    bv = (1 - b2) * (2 * g * d + d * d) + 8 * U32 * np.abs(ref_v)
    assert (np.abs(got_v - ref_v) <= bv * 1.01 + 1e-38).all(), "Adam v"
    sure = g > 2 * d
    gap = np.where(sure, g - d, 1.0)
    bp = np.where(sure, lr * (d * eps / (gap * gap) + 16 * U32), 2 * lr * (1 + 16 * U32))
    bp = bp + 2 * U32 * np.abs(ref_p)
    bad = np.abs(got_p - ref_p) > bp * 1.01
    assert not bad.any(), f"Adam p: {int(bad.sum())} values outside the bound"


class CuMaskedStream:
    """A stream whose kernels run on CUs [first, first + count) only
    (hipExtStreamCreateWithCUMask, default priority); close() destroys it."""

    def __init__(self, torch, first, count):
        import ctypes
        self.torch, self.ct = torch, ctypes
        hip = ctypes.CDLL("libamdhip64.so.7")  # the runtime torch already loaded
        hip.hipExtStreamCreateWithCUMask.argtypes = [ctypes.c_void_p, ctypes.c_uint32,
                                                     ctypes.c_void_p]
        hip.hipStreamDestroy.argtypes = [ctypes.c_void_p]
        self.hip = hip
        ncu = torch.cuda.get_device_properties(0).multi_processor_count
        assert 0 <= first and 0 < count and first + count <= ncu
        words = [0] * ((ncu + 31) // 32)
        for c in range(first, first + count):
            words[c // 32] |= 1 << (c % 32)
        mask = (ctypes.c_uint32 * len(words))(*words)
        self.h = ctypes.c_void_p()
        rc = hip.hipExtStreamCreateWithCUMask(ctypes.byref(self.h), len(words), ctypes.byref(mask))
        assert rc == 0, f"hipExtStreamCreateWithCUMask failed ({rc})"
        self.stream = torch.cuda.ExternalStream(self.h.value)

    def close(self):
        self.torch.cuda.synchronize()
        self.hip.hipStreamDestroy(self.h)
