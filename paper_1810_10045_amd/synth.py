"""Seeded synthetic inputs shaped like the paper's workloads.

This module holds no arithmetic of the method: it only draws token ids and
gradient rows, so that the GPU path and the CPU oracle are fed the very same
arrays. The paper's corpora (1-Billion Word, Gutenberg, Tieba) are not
available, so token streams are drawn from a bounded Zipf law, which is the
statistic the method exploits (Sec. III: word frequency inversely
proportional to frequency rank; U grows as a power of the token count,
Fig. 1).

Recipe
------
* Word ids: bounded Zipf over a frequency-ordered vocabulary,
  p(r) proportional to r**-s for ranks r = 1..V, id = r - 1 (rank 1 is the
  most frequent word, like "a" = word 1 in the Fig. 2 example). Drawn by
  inverse CDF: u ~ U[0,1) from PCG64(seed), id = searchsorted(cdf, u,
  side="right"), clipped to V - 1.
* Gradient rows: i.i.d. N(0, std^2) fp32, generated in blocks of
  ``ROW_BLOCK`` rows, block b from PCG64(SeedSequence([seed, b])), so the
  result does not depend on how many threads fill it. bf16 gradients are the
  round-to-nearest-even bf16 of those fp32 values, carried as uint16 bits.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
import dataclasses
from dataclasses import dataclass, field

import numpy as np

ROW_BLOCK = 16384


def zipf_cdf(V: int, s: float) -> np.ndarray:
    """Cumulative bounded-Zipf distribution over ranks 1..V (float64)."""
    r = np.arange(1, V + 1, dtype=np.float64)
    w = r ** (-float(s))
    c = np.cumsum(w)
    return c / c[-1]


def zipf_ids(K: int, V: int, s: float, seed: int, dtype=np.int32) -> np.ndarray:
    """K word ids in [0, V) drawn i.i.d. from the bounded Zipf law."""
    rng = np.random.Generator(np.random.PCG64(seed))
    u = rng.random(K)
    ids = np.searchsorted(zipf_cdf(V, s), u, side="right")
    np.minimum(ids, V - 1, out=ids)
    return ids.astype(dtype)


def zipf_ids_permuted(K: int, V: int, s: float, seed: int, perm_seed: int,
                      dtype=np.int32) -> np.ndarray:
    """Bounded-Zipf ids whose ranks are spread over the vocabulary by a fixed
    random permutation (id = perm[rank - 1]): the same counts as zipf_ids,
    but the frequent words no longer sit at the smallest ids, so in sorted
    order the long runs are scattered among the short ones."""
    perm = np.random.Generator(np.random.PCG64(perm_seed)).permutation(V)
    return perm[zipf_ids(K, V, s, seed, np.int64)].astype(dtype)


def distinct_ids(n: int, V: int, seed: int, dtype=np.int32) -> np.ndarray:
    """n distinct word ids in [0, V), drawn uniformly without replacement and
    listed in ascending order (a stand-in for a type list, as the row list
    of an update or the source ids of a fill)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return np.sort(rng.choice(V, size=n, replace=False)).astype(dtype)


def _threads() -> int:
    n = os.cpu_count() or 1
    return max(1, min(16, n))


def _fill_normal(out: np.ndarray, seed: int, b: int, std: float):
    """Rows [b * ROW_BLOCK, (b + 1) * ROW_BLOCK) of a block-seeded matrix."""
    lo, hi = b * ROW_BLOCK, min(out.shape[0], (b + 1) * ROW_BLOCK)
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, b])))
    rng.standard_normal(out=out[lo:hi], dtype=np.float32)
    if std != 1.0:
        out[lo:hi] *= np.float32(std)


def _blocks(K: int) -> int:
    return (K + ROW_BLOCK - 1) // ROW_BLOCK


def normal_rows(K: int, D: int, seed: int, std: float = 1.0) -> np.ndarray:
    """K x D fp32 rows ~ N(0, std^2), block-seeded (see module docstring)."""
    out = np.empty((K, D), dtype=np.float32)
    nblk = _blocks(K)
    if nblk <= 1:
        for b in range(nblk):
            _fill_normal(out, seed, b, std)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(lambda b: _fill_normal(out, seed, b, std), range(nblk)))
    return out


def stacked_normal_rows(K: int, D: int, seeds) -> np.ndarray:
    """Concatenation of normal_rows(K, D, seed) over ``seeds``, filled by one
    thread pool over every (part, block) pair."""
    seeds = list(seeds)
    out = np.empty((K * len(seeds), D), dtype=np.float32)
    parts = [out[g * K:(g + 1) * K] for g in range(len(seeds))]
    jobs = [(g, b) for g in range(len(seeds)) for b in range(_blocks(K))]
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(lambda j: _fill_normal(parts[j[0]], seeds[j[0]], j[1], 1.0), jobs))
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even bf16 of fp32 values, as uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty(x.shape, dtype=np.uint16)
    flat_in = x.reshape(-1).view(np.uint32)
    flat_out = out.reshape(-1)
    step = 1 << 22

    def conv(lo: int):
        b = flat_in[lo:lo + step]
        bias = ((b >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
        flat_out[lo:lo + step] = ((b + bias) >> np.uint32(16)).astype(np.uint16)

    starts = range(0, flat_in.size, step)
    if len(starts) <= 1:
        for lo in starts:
            conv(lo)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(conv, starts))
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact fp32 values of bf16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclass(frozen=True)
class Workload:
    """One synthetic workload. ``shards`` > 1 concatenates that many
    independently seeded batches of K tokens (the G x K gathered index list
    of Sec. III-A step 3, at real shape on one GPU)."""
    name: str
    K: int
    V: int
    s: float
    D: int
    grad_dtype: str          # "f32" or "bf16"
    id_dtype: str            # "i32" or "i64"
    step: str                # what follows Seg-Sum: "scatter", "sgd", "expand", "adam"
    number: int              # seed base: ids 1000n+1, grads 1000n+2, table 1000n+3, m/v +4/+5
    shards: int = 1
    perm_seed: int = 0       # > 0: ranks spread over the ids by a fixed permutation
    scale: float = 1.0       # compression scale F of a binary16 payload (Sec. III-C)
    samples: int = 0         # > 0: sampled-softmax candidates per GPU (Sec. III-B)
    seed_rule: str = ""      # how many sampler seeds the shards (GPUs) use
    lr: float = 0.0
    table_std: float = 0.02
    adam: tuple = field(default=(0.9, 0.999, 1e-8))

    @property
    def tokens(self) -> int:
        return (self.K + self.samples) * self.shards

    def batch(self, b: int) -> "Workload":
        """The b-th independent batch of this workload (b = 0 is the
        workload itself): every seed moves by 1,000,000 * b."""
        if b == 0:
            return self
        return dataclasses.replace(self, number=self.number + 1000 * b)

    @property
    def np_id_dtype(self):
        return np.int64 if self.id_dtype == "i64" else np.int32

    def _draw(self, seed: int) -> np.ndarray:
        if self.perm_seed:
            return zipf_ids_permuted(self.K, self.V, self.s, seed, self.perm_seed, self.np_id_dtype)
        return zipf_ids(self.K, self.V, self.s, seed, self.np_id_dtype)

    def ids(self) -> np.ndarray:
        if self.shards == 1:
            return self._draw(1000 * self.number + 1)
        return np.concatenate([self.shard_ids(g) for g in range(self.shards)])

    def shard_ids(self, g: int) -> np.ndarray:
        return self._draw(1000 * self.number + 100 + g)

    def sampler_words(self, seed_of_gpu) -> np.ndarray:
        """The sampled-softmax random words, shards x samples uint64: shard g
        takes the raw 64-bit outputs of PCG64(SeedSequence([1000n+6, j])),
        j = seed_of_gpu[g], so shards that share a seed share their words."""
        out = np.empty((self.shards, self.samples), np.uint64)
        streams = {}
        for g, j in enumerate(seed_of_gpu):
            if j not in streams:
                bg = np.random.PCG64(np.random.SeedSequence([1000 * self.number + 6, int(j)]))
                streams[j] = bg.random_raw(self.samples).astype(np.uint64)
            out[g] = streams[j]
        return out.reshape(-1)

    def grads_f32(self) -> np.ndarray:
        """fp32 gradients (before any bf16 rounding), one row per token (for a
        sampled-softmax workload: the shards' sampled rows, then their words)."""
        if self.samples:
            return normal_rows(self.tokens, self.D, 1000 * self.number + 2)
        if self.shards == 1:
            return normal_rows(self.K, self.D, 1000 * self.number + 2)
        return stacked_normal_rows(self.K, self.D,
                                   [1000 * self.number + 200 + g for g in range(self.shards)])

    def grads(self) -> np.ndarray:
        """Gradients in the workload's storage dtype (bf16 as uint16 bits)."""
        g = self.grads_f32()
        return bf16_bits(g) if self.grad_dtype == "bf16" else g

    def table(self) -> np.ndarray:
        return normal_rows(self.V, self.D, 1000 * self.number + 3, self.table_std)


# The five workloads: per-GPU word-LM batches (Sec. IV-B: 1-Billion Word, 100K
# and 800K vocabularies, 512/1024-wide embeddings), the post-gather merge over
# 64 concatenated batches (Sec. III-A step 4 at G = 64), a heavily duplicated
# character-level vocabulary (Sec. IV-B char LM, Tieba-sized 20K), and a 2M
# int64 vocabulary updated with Adam.
WORKLOADS = {
    "word_tiny_8k": Workload("word_tiny_8k", K=8192, V=100_000, s=1.0, D=512,
                             grad_dtype="f32", id_dtype="i32", step="scatter", number=1),
    "word_step_64k": Workload("word_step_64k", K=65536, V=800_000, s=1.0, D=1024,
                              grad_dtype="f32", id_dtype="i32", step="sgd", number=2, lr=0.1),
    "merge_64x32k_bf16": Workload("merge_64x32k_bf16", K=32768, V=800_000, s=1.0, D=1024,
                                  grad_dtype="bf16", id_dtype="i32", step="expand",
                                  number=3, shards=64),
    "char_heavy_1m": Workload("char_heavy_1m", K=1_048_576, V=20_000, s=1.2, D=2048,
                              grad_dtype="f32", id_dtype="i32", step="scatter", number=4),
    "vocab2m_adam_i64": Workload("vocab2m_adam_i64", K=262_144, V=2_000_000, s=0.9, D=1024,
                                 grad_dtype="f32", id_dtype="i64", step="adam", number=5,
                                 lr=1e-3),
    # The merge with the step-5 payload compressed to binary16 (Sec. III-C),
    # same inputs as merge_64x32k_bf16; F = 64 keeps the largest per-word
    # sums of these N(0,1) rows (about +-240) inside binary16's range.
    "merge_64x32k_f16": Workload("merge_64x32k_f16", K=32768, V=800_000, s=1.0, D=1024,
                                 grad_dtype="bf16", id_dtype="i32", step="expand_f16",
                                 number=3, shards=64, scale=64.0),
    # The per-GPU word step with the word ranks permuted over the vocabulary
    # (the robustness variant: heads no longer first in sorted order).
    "word_step_64k_perm": Workload("word_step_64k_perm", K=65536, V=800_000, s=1.0, D=1024,
                                   grad_dtype="f32", id_dtype="i32", step="sgd", number=2,
                                   lr=0.1, perm_seed=77),
}

# The output embedding under sampled softmax (Sec. III-B), at the word-LM
# shape of Sec. IV-B on 64 GPUs: each GPU samples 1024 candidates uniformly
# from the 800K vocabulary and adds the 32 x 20 = 640 words of its batch;
# Unique + Seg-Sum run over the 64 x 1664 gathered rows (D = 512, the
# projection width) and SGD updates the output embedding. One workload per
# seeding rule: all GPUs different, G^0.64, log2 G, ln G, log10 G, one seed.
for _rule in ("G", "pow0.64", "log2", "ln", "log10", "one"):
    _name = "sampled_softmax_64x1024_" + _rule
    WORKLOADS[_name] = Workload(_name, K=640, V=800_000, s=1.0, D=512, grad_dtype="f32",
                                id_dtype="i32", step="softmax_sgd", number=6, shards=64,
                                samples=1024, seed_rule=_rule, lr=0.1)
