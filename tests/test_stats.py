"""The types-vs-tokens tool of Fig. 1: the fit recovers exact power laws
(CPU), and the GPU counts equal the oracle's number of types (GPU)."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle  # noqa: E402
from paper_1810_10045_amd import stats, synth  # noqa: E402


def test_fit_recovers_exact_power_laws():
    Ns = np.array([1e3, 1e4, 1e5, 1e6, 1e7])
    for alpha, c in ((0.64, 5.5), (0.5, 1.0), (1.0, 0.3)):
        a, cc = stats.fit_power_law(Ns, c * Ns ** alpha)
        assert abs(a - alpha) < 1e-12 and abs(cc - c) < 1e-9 * c
    with pytest.raises(ValueError):
        stats.fit_power_law([10], [3])


@pytest.mark.gpu
def test_gpu_type_counts_match_the_oracle():
    torch = pytest.importorskip("torch")
    from paper_1810_10045_amd import lmzipf as lz
    ids = synth.zipf_ids(300_000, 800_000, 1.0, 501, np.int32)
    Ns = [1, 63, 1000, 65_536, 131_073, 300_000]
    got = stats.types_vs_tokens(torch.from_numpy(ids).cuda(), 800_000, Ns, lz)
    want = [len(oracle.unique(ids[:n], 800_000)[0]) for n in Ns]
    assert got.tolist() == want
