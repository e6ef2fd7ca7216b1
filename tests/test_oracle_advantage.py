"""The fp64 TreePO advantage oracle against its pins (CPU)."""

import pytest

from tests import advantage_pins as P


@pytest.mark.parametrize("pin", P.ALL, ids=lambda f: f.__name__)
def test_advantage_pin(pin):
    pin()
