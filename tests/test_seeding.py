"""Pins of the controlled-randomness rules of Sec. III-B (CPU only).

The paper has groups of GPUs share a sampler seed: G^0.64 seeds (the
exponent of the type/token power law) keep the accuracy of a seed per GPU,
and it also evaluates log2 G, ln G and log10 G seeds. A rule's value is
rounded up (at least one seed), and the GPUs form that many contiguous
groups of equal size to within one. The expected numbers below were worked
out by hand from those definitions, not by calling the rules.
"""
import math

import pytest

from paper_1810_10045_amd import seeding

# num_seeds(G, rule) for the GPU counts the paper runs on (16 .. 192) and
# the degenerate ones. By hand, for example at G = 64:
#   64^0.64 = e^(0.64 ln 64) = e^2.662 = 14.3 -> 15;  log2 64 = 6 exactly;
#   ln 64 = 4.16 -> 5;  log10 64 = 1.81 -> 2.
# At G = 192: 192^0.64 = e^(0.64 * 5.2575) = e^3.365 = 28.9 -> 29;
#   log2 192 = 7.58 -> 8;  ln 192 = 5.26 -> 6;  log10 192 = 2.28 -> 3.
HAND = {
    #      G   pow0.64 log2  ln  log10 one
    1:   (1,   1,      1,    1,  1,    1),
    2:   (2,   2,      1,    1,  1,    1),
    8:   (8,   4,      3,    3,  1,    1),
    16:  (16,  6,      4,    3,  2,    1),
    64:  (64,  15,     6,    5,  2,    1),
    192: (192, 29,     8,    6,  3,    1),
}
RULES = ("G", "pow0.64", "log2", "ln", "log10", "one")


@pytest.mark.parametrize("G", sorted(HAND))
def test_number_of_seeds_by_hand(G):
    got = tuple(seeding.num_seeds(G, r) for r in RULES)
    assert got == HAND[G], (G, got)


def test_rules_listed():
    assert tuple(seeding.RULES) == RULES


def test_exact_powers_are_not_rounded_up():
    """log2 of a power of two is exact: 2^k GPUs get k seeds, not k + 1."""
    for k in range(1, 11):
        assert seeding.num_seeds(2 ** k, "log2") == k
    assert seeding.num_seeds(100, "log10") == 2
    assert seeding.num_seeds(1000, "log10") == 3


def test_assignment_by_hand():
    """Which seed each GPU uses, for small cases worked out by hand."""
    assert seeding.seed_of_gpus(8, "ln") == [0, 0, 0, 1, 1, 1, 2, 2]
    assert seeding.seed_of_gpus(8, "pow0.64") == [0, 0, 1, 1, 2, 2, 3, 3]
    assert seeding.seed_of_gpus(2, "log2") == [0, 0]
    assert seeding.seed_of_gpus(1, "G") == [0]
    # G = 64, 15 seeds: group j starts at ceil(64 j / 15) = 0, 5, 9, 13, 18,
    # 22, 26, 30, 35, 39, 43, 47, 52, 56, 60 (and 64 ends the last group)
    sizes = [5, 4, 4, 5, 4, 4, 4, 5, 4, 4, 4, 5, 4, 4, 4]
    want = [j for j, n in enumerate(sizes) for _ in range(n)]
    assert seeding.seed_of_gpus(64, "pow0.64") == want


@pytest.mark.parametrize("rule", RULES)
def test_groups_are_contiguous_and_balanced(rule):
    """For every G up to 256: n seeds, each used, in contiguous groups (the
    seed never decreases along the GPUs), of sizes within one of each other
    and of G / n."""
    for G in range(1, 257):
        n = seeding.num_seeds(G, rule)
        s = seeding.seed_of_gpus(G, rule)
        assert len(s) == G and s[0] == 0 and s[-1] == n - 1
        assert all(b - a in (0, 1) for a, b in zip(s, s[1:])), (G, rule)
        sizes = [s.count(j) for j in range(n)]
        assert max(sizes) - min(sizes) <= 1
        assert math.floor(G / n) <= min(sizes) and max(sizes) <= math.ceil(G / n)


def test_bad_arguments():
    with pytest.raises(ValueError):
        seeding.num_seeds(0, "G")
    with pytest.raises(ValueError):
        seeding.seed_index(5, 4, 2)
    with pytest.raises(KeyError):
        seeding.num_seeds(4, "sqrt")
