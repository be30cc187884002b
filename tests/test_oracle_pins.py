"""Pins of the CPU oracle: closed forms, invariants, brute force and the
paper's own worked values (tests/golden).  CPU only."""
import pytest

import oracle_checks as C


@pytest.mark.parametrize("check", C.ALL_CHECKS, ids=lambda f: f.__name__)
def test_oracle_pin(check):
    check()
