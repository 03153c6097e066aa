"""lm_unique_noalloc (the Unique entry point for callers that cannot
allocate) against lm_unique with a caller's workspace, through the C ABI:
every integer output bit for bit, over calls in a row that share the
library's device workspace, each smaller than the one before, so that a
later call sees what the earlier one left there. Also checked against the
oracle, and the host-side rejection of inputs above the maximum."""
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


# Calls in a row, largest first: the maximum with 61-bit int64 keys (the
# largest workspace), the 2M-vocabulary shape, the word step, a merge shard,
# the one-workgroup path and an empty call.
CALLS = [
    (262_144, 2**61, 0.9, np.int64, 301),
    (262_144, 2_000_000, 0.9, np.int64, 302),
    (262_144, 32_768, 1.0, np.int64, 307),   # counts per id: the largest workspace
    (200_000, 20_000, 1.2, np.int32, 308),
    (65_536, 800_000, 1.0, np.int32, 303),
    (32_768, 800_000, 1.0, np.int32, 304),
    (8_192, 100_000, 1.0, np.int32, 305),
    (0, 10, 1.0, np.int32, 306),
]


def _ids(K, V, s, dt, seed):
    ids = synth.zipf_ids(K, min(V, 4_000_000), s, seed, dt)
    if V > 4_000_000:
        ids = (ids.astype(np.int64) * (V // 4_000_000) + 7).astype(dt)
        assert K == 0 or ids.max() < V
    return ids


def _same(a, b, K):
    U = int(a.num_unique.item())
    assert U == int(b.num_unique.item())
    assert torch.equal(a.uniq[:U], b.uniq[:U]) and torch.equal(a.counts[:U], b.counts[:U])
    assert torch.equal(a.offsets[:U + 1], b.offsets[:U + 1])
    assert torch.equal(a.inverse[:K], b.inverse[:K]) and torch.equal(a.perm[:K], b.perm[:K])
    return U


def test_noalloc_matches_lm_unique(lz):
    dev = torch.device("cuda:0")
    for K, V, s, dt, seed in CALLS:
        print(f"noalloc unique K={K} V={V} {dt.__name__}", flush=True)
        ids = _ids(K, V, s, dt, seed)
        t = torch.from_numpy(ids).to(dev)
        tdt = torch.int64 if dt == np.int64 else torch.int32
        got = lz.unique_noalloc(t, V, lz.unique_buffers(K, V, tdt, dev))
        want = lz.unique(t, V, out=lz.unique_buffers(K, V, tdt, dev), ws=lz.Workspace(dev))
        torch.cuda.synchronize()
        lz.check(got.dev_err)
        lz.check(want.dev_err)
        _same(got, want, K)
        H.assert_unique_matches(got, ids, V, oracle, f"noalloc K={K} V={V}")


def test_noalloc_repeat_and_reject(lz):
    """The same input twice after a larger one gives the same result; K above
    the maximum is refused on the host (nothing launched)."""
    dev = torch.device("cuda:0")
    big = torch.from_numpy(_ids(200_000, 800_000, 1.0, np.int32, 311)).to(dev)
    small_np = _ids(20_000, 800_000, 1.0, np.int32, 312)
    small = torch.from_numpy(small_np).to(dev)
    lz.unique_noalloc(big, 800_000, lz.unique_buffers(200_000, 800_000, torch.int32, dev))
    a = lz.unique_noalloc(small, 800_000, lz.unique_buffers(20_000, 800_000, torch.int32, dev))
    b = lz.unique_noalloc(small, 800_000, lz.unique_buffers(20_000, 800_000, torch.int32, dev))
    torch.cuda.synchronize()
    lz.check(a.dev_err)
    lz.check(b.dev_err)
    _same(a, b, 20_000)
    H.assert_unique_matches(a, small_np, 800_000, oracle, "noalloc repeat")
    K = lz.UNIQUE_NOALLOC_MAX_K + 1
    over = torch.zeros(K, dtype=torch.int32, device=dev)
    with pytest.raises(lz.LmError, match="UNSUPPORTED"):
        lz.unique_noalloc(over, 10, lz.unique_buffers(K, 10, torch.int32, dev))
