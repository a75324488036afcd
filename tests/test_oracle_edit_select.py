"""Pins of the edit-selection oracle (CPU only)."""
import pytest

import oracle
import oracle_pins as pins


@pytest.mark.parametrize("check", pins.EDIT_CHECKS, ids=lambda c: c.__name__)
def test_edit_pin(check):
    check(oracle)
