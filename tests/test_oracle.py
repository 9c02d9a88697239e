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


# --- fused epilogue (activations) -----------------------------------------

def test_activations_pinned():
    import math

    import numpy as np
    from scipy.special import expit
    x = np.linspace(-12.0, 12.0, 4801)
    relu, gelu, silu = (oracle.activation(x, a) for a in (1, 2, 3))
    # Odd-part identities: f(x) - f(-x) = x for ReLU, both GELU forms and SiLU.
    for f, a in ((relu, 1), (gelu, 2), (silu, 3)):
        assert np.allclose(f - oracle.activation(-x, a), x, rtol=0, atol=1e-12)
    assert np.array_equal(relu, np.where(x > 0, x, 0.0))
    # SiLU = x * logistic(x) (scipy's logistic function).
    assert np.allclose(silu, x * expit(x), rtol=1e-14, atol=1e-300)
    # The tanh form of GELU stays within 1e-3 of the exact GELU x * Phi(x).
    exact = np.array([0.5 * v * (1.0 + math.erf(v / math.sqrt(2.0))) for v in x])
    assert np.max(np.abs(gelu - exact)) < 1e-3
    # Slopes: 1/2 at 0 for GELU and SiLU; never above the bound the tolerance uses.
    h = 1e-6
    for a in (2, 3):
        d0 = (oracle.activation(np.array([h]), a) - oracle.activation(np.array([-h]), a))[0] / (2 * h)
        assert abs(d0 - 0.5) < 1e-6
        slope = np.diff(oracle.activation(x, a)) / np.diff(x)
        assert slope.max() < oracle.ACT_SLOPE_BOUND and slope.max() > 1.05
