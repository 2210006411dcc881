"""The CPU oracle against its pins (sizes from the paper, library transposes,
round-trip and multiset invariants, brute force).  CPU only."""
import pytest

import oracle
import pins


class OracleImpl:
    pack_layer = staticmethod(oracle.pack_layer)
    unpack_layer = staticmethod(oracle.unpack_layer)


@pytest.mark.parametrize("pin", pins.FULL_PINS, ids=lambda p: p.__name__)
def test_oracle_pin(pin):
    pin(OracleImpl)
