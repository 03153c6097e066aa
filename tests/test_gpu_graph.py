"""lm_unique and lm_segsum captured in HIP graphs and replayed on changing
inputs, with eager calls on the same workspace in between: every replay is
checked against the oracle. (Under capture lm_segsum takes its two-launch
form: the one-launch form tells its calls apart by a per-call value that a
replay would repeat. lm_unique's first kernel clears the tile tickets and
status words that its later kernels use, inside the graph as well.)"""
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
DEV = "cuda"


@pytest.fixture(scope="module")
def lz():
    from paper_1810_10045_amd import lmzipf
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return lmzipf


def _check(out, ids, grad, V):
    o = oracle.unique(ids, V)
    U = len(o[0])
    ref = oracle.segsum(grad, o[3], U)
    err = H.row_rel_err(out[:U].double().cpu().numpy(), ref, H.sum_of_squares(grad, o[3], U, oracle))
    assert err <= H.TOL_F32, err


def test_segsum_graph_replays(lz):
    K, V, D = 65_536, 800_000, 1024
    ws = lz.Workspace(DEV)
    ids = synth.zipf_ids(K, V, 1.0, 201, np.int32)
    g32 = synth.normal_rows(K, D, 202)
    res = lz.unique(torch.from_numpy(ids).to(DEV), V, ws=ws)
    grad = torch.from_numpy(g32).to(DEV)
    out = torch.empty((res.offsets.numel() - 1, D), dtype=torch.float32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    lz.segsum(grad, res.perm, res.inverse, res.offsets, res.num_unique, out=out, dev_err=err, ws=ws)
    torch.cuda.synchronize()
    lz.check(err)
    _check(out, ids, g32, V)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        lz.segsum(grad, res.perm, res.inverse, res.offsets, res.num_unique, out=out, dev_err=err, ws=ws)
    torch.cuda.synchronize()

    other_ids = synth.zipf_ids(K, V, 1.0, 299, np.int32)
    other_grad = torch.from_numpy(synth.normal_rows(K, D, 298)).to(DEV)
    for i, seed in enumerate((203, 205, 207, 209, 211)):
        print(f"graph replay with inputs of seed {seed}", flush=True)
        ids = synth.zipf_ids(K, V, 1.0, seed, np.int32)
        g32 = synth.normal_rows(K, D, seed + 1)
        lz.unique(torch.from_numpy(ids).to(DEV), V, out=res, ws=ws)  # the graph's input buffers
        grad.copy_(torch.from_numpy(g32))
        out.fill_(float("nan"))
        if i % 2:
            # eager Seg-Sum on the same workspace between two replays (the
            # others follow each other with only new inputs in between)
            r2 = lz.unique(torch.from_numpy(other_ids).to(DEV), V, ws=ws)
            lz.segsum(other_grad, r2.perm, r2.inverse, r2.offsets, r2.num_unique, dev_err=err, ws=ws)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        lz.check(err)
        _check(out, ids, g32, V)


def test_unique_graph_replays(lz):
    K, V = 65_536, 800_000
    ws = lz.Workspace(DEV)
    ids_dev = torch.from_numpy(synth.zipf_ids(K, V, 1.0, 301, np.int32)).to(DEV)
    res = lz.unique(ids_dev, V, ws=ws)
    torch.cuda.synchronize()
    lz.check(res.dev_err)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        lz.unique(ids_dev, V, out=res, ws=ws)
    torch.cuda.synchronize()

    other = torch.from_numpy(synth.zipf_ids(K // 2 + 7, V, 1.0, 399, np.int32)).to(DEV)
    for i, seed in enumerate((303, 305, 307, 309)):
        print(f"unique graph replay with ids of seed {seed}", flush=True)
        ids = synth.zipf_ids(K, V, 1.0, seed, np.int32)
        ids_dev.copy_(torch.from_numpy(ids))
        res.perm.fill_(-1)
        res.inverse.fill_(-1)
        if i % 2:
            # an eager call on the same workspace between replays
            r2 = lz.unique(other, V, ws=ws)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        lz.check(res.dev_err)
        H.assert_unique_matches(res, ids, V, oracle, f"replay {i}")
        if i % 2:
            lz.check(r2.dev_err)
            H.assert_unique_matches(r2, other.cpu().numpy(), V, oracle, f"eager {i}")
