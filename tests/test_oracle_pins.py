"""The CPU oracle against its pins (closed forms, library routines, independent
implementations, invariants).  No GPU involved."""
import pytest

import oracle.reusevit as ora

from .pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(ora)
