"""The CPU oracle against its pins, and the pins against planted mistakes (CPU only)."""
import pytest

import oracle
from oracle_pins import ALL_PINS


@pytest.fixture(scope="module")
def lib():
    return oracle.load()


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_oracle_pin(lib, pin):
    pin(lib)


# Each planted mistake of oracle.c (ORACLE_MUTANT=<id>) must fail at least one pin:
# 1 mask ignored, 2 X transposed, 3 wrong fp16 exponent bias,
# 4 fp16 subnormals flushed, 5 last column of the sum dropped, 6 sign dropped.
@pytest.mark.parametrize("mutant", [1, 2, 3, 4, 5, 6])
def test_pins_catch_planted_mistake(tmp_path, mutant):
    oracle.build(mutant=mutant, out_dir=str(tmp_path))
    mlib = oracle.load(mutant=mutant, out_dir=str(tmp_path))
    caught = []
    for pin in ALL_PINS:
        try:
            pin(mlib)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin caught planted mistake {mutant}"
