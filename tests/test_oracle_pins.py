"""The CPU oracle against its pins (hand-derived fixtures, closed forms,
invariants, exact-rational brute force).  CPU only."""

import pytest

import oracle
import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin):
    pin(oracle)


def test_pins_are_independent_of_oracle_source():
    # The pins and the exact helpers must not import the oracle themselves:
    # they only receive it as an argument.
    import inspect

    import exact

    for mod in (oracle_pins, exact):
        src = inspect.getsource(mod)
        assert "import oracle" not in src and "from oracle" not in src
