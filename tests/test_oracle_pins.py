"""The oracle against its pins (CPU only)."""
import pytest

from pins import PINS


@pytest.mark.parametrize("name", sorted(PINS))
def test_pin(name, oracle_lib):
    PINS[name](oracle_lib)
