"""The oracle against its pins (CPU only)."""
import pytest


import oracle as O
from oracle_pins import ALL_PINS


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(O)


def test_oracle_rejects_bad_geometry():
    with pytest.raises(ValueError):
        O.layout([1, 2], 256, 100)  # chunk not a multiple of the alignment
    with pytest.raises(ValueError):
        O.layout([1, 2], 12, 24)  # alignment not a multiple of 8
    with pytest.raises(ValueError):
        O.chunk_sums(bytes(504), 8, 512, 256)  # window does not start a chunk
