"""Types against tokens (Sec. I, Fig. 1): the number of distinct words U in
the first N tokens of a stream grows as a power of N, U ~ c * N^alpha, which
is what makes the unique-word path pay off (U_g << G*K).

types_vs_tokens counts U for several prefix lengths with lm_unique on the
GPU (one call per N, num_unique read back); fit_power_law fits alpha and c
by least squares on (log N, log U).
"""
from __future__ import annotations

import numpy as np


def types_vs_tokens(ids, V: int, Ns, lz=None) -> np.ndarray:
    """U(N) for each N in Ns: the distinct ids among ids[:N] (a CUDA tensor
    of int32/int64 ids in [0, V)). Raises if a kernel flags an error."""
    import torch
    if lz is None:
        from paper_1810_10045_amd import lmzipf as lz
    Ns = [int(n) for n in Ns]
    if any(n < 1 or n > ids.numel() for n in Ns):
        raise ValueError("every N must lie in [1, len(ids)]")
    ws = lz.Workspace(ids.device)
    out = []
    for n in Ns:
        res = lz.unique(ids[:n], V, ws=ws)
        torch.cuda.synchronize()
        lz.check(res.dev_err)
        out.append(int(res.num_unique.item()))
    return np.array(out, dtype=np.int64)


def fit_power_law(Ns, Us):
    """(alpha, c) minimising the squared error of log U = alpha log N + log c."""
    x = np.log(np.asarray(Ns, np.float64))
    y = np.log(np.asarray(Us, np.float64))
    if x.size < 2:
        raise ValueError("need at least two points")
    A = np.stack([x, np.ones_like(x)], axis=1)
    (alpha, logc), *_ = np.linalg.lstsq(A, y, rcond=None)
    return float(alpha), float(np.exp(logc))


def main(argv=None):
    """Print U(N) and the fitted alpha for the Zipf laws of the synthetic
    workloads (N = 2^13 .. 2^24 tokens, one stream per law)."""
    import argparse
    import torch
    from paper_1810_10045_amd import synth
    ap = argparse.ArgumentParser(description=main.__doc__)
    ap.add_argument("--max-log2", type=int, default=24)
    args = ap.parse_args(argv)
    Ns = [1 << k for k in range(13, args.max_log2 + 1)]
    laws = [(100_000, 1.0), (800_000, 1.0), (20_000, 1.2), (2_000_000, 0.9)]
    print("V          s     alpha   c        " + " ".join(f"U(2^{k})" for k in range(13, args.max_log2 + 1, 3)))
    for V, s in laws:
        ids = torch.from_numpy(synth.zipf_ids(Ns[-1], V, s, 911, np.int32)).cuda()
        Us = types_vs_tokens(ids, V, Ns)
        a, c = fit_power_law(Ns, Us)
        print(f"{V:<10d} {s:<5.1f} {a:6.3f}  {c:7.2f}  " + " ".join(f"{u:7d}" for u in Us[::3]), flush=True)


if __name__ == "__main__":
    main()
