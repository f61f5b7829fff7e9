"""The plan-execution oracle against hand values, closed forms and
invariants (no GPU)."""

import pytest

import sim_pins


@pytest.mark.parametrize("name,check", sim_pins.ALL, ids=[n for n, _ in sim_pins.ALL])
def test_sim_pin(name, check):
    check()
