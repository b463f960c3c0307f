"""The float64 oracle against what the paper and mathematics fix (CPU)."""
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS,
                         ids=[p.__name__ for p in oracle_pins.ALL_PINS])
def test_oracle_pin(pin, oracle_lib):
    pin(oracle_lib)
