"""The fp64 oracle checked against library routines, closed forms and
invariants (see pins.py for what each pin fixes)."""
import pytest

import oracle.oracle as orc
import pins


@pytest.fixture(scope="module")
def lib():
    orc.build(force=False)
    return orc.load()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(lib, pin):
    pin(lib)
