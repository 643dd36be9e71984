"""The fp64 oracle against its pins (worked examples, closed forms, brute force,
invariants); see ``oracle_pins.py`` for what each pin checks and cites."""
import pytest

from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_oracle_pin(pin):
    pin()
