"""The CPU oracle pinned to the paper's worked examples, closed forms,
independent library routines, brute force and invariants (CPU only)."""
import pytest

import os, sys
sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import oracle_pins as P  # noqa: E402


@pytest.mark.parametrize("check", P.ALL_CHECKS + [P.check_memory_example],
                         ids=lambda c: c.__name__)
def test_pin(check):
    check()
