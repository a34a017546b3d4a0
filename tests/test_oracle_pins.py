"""The fp64 oracle against its pins (closed forms, the paper's worked example, LP and grid
sandwiches, library convolutions, soundness).  CPU only."""
import pytest

import oracle
from tests import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(oracle)
