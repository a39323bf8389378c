"""The CPU oracle against its pins (worked examples, numpy indexing,
library special cases, invariants, error rules)."""
import pytest

import oracle_pins
from oracle import kvx_oracle


@pytest.fixture(scope="module")
def oracle():
    kvx_oracle.build()
    return kvx_oracle.Oracle(kvx_oracle.LIBRARY)


@pytest.mark.parametrize("pin", oracle_pins.PINS, ids=lambda f: f.__name__)
def test_pin(oracle, pin):
    pin(oracle)
