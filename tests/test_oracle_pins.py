"""The fp64 oracles against their pins (closed forms, the paper's worked example, LP and grid
sandwiches, library convolutions, soundness, finite differences).  CPU only."""
import pytest

import oracle
from oracle import alpha64, beta64
from tests import pins, pins_alpha, pins_beta


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle)


@pytest.mark.parametrize("pin", pins_alpha.ALPHA_PINS, ids=lambda p: p.__name__)
def test_alpha_pin(pin):
    pin(alpha64)


@pytest.mark.parametrize("pin", pins_beta.BETA_PINS, ids=lambda p: p.__name__)
def test_beta_pin(pin):
    pin(beta64)
