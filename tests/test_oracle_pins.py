"""The fp64 oracle against hand-derived values, closed-form reductions and
invariants (no GPU)."""

import pytest

import pins


@pytest.mark.parametrize("name,check", pins.ALL_CHECKS, ids=[n for n, _ in pins.ALL_CHECKS])
def test_oracle_pin(name, check):
    check(None)
