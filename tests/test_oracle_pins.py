"""The float64 oracle against what the paper and the mathematics fix (no GPU)."""
import pytest

import oracle
import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(oracle.luna_oracle)


import oracle_variant_pins  # noqa: E402


@pytest.mark.parametrize("pin", oracle_variant_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_variant_pin(pin):
    pin(oracle.luna_variants)


import oracle_distill_pins  # noqa: E402


@pytest.mark.parametrize("pin", oracle_distill_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_distill_pin(pin):
    pin(oracle.luna_distill)
