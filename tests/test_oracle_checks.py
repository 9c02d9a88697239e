"""Pins of the oracle's acceptance checker and of its fused-epilogue reference (CPU only).

``oracle.check_tolerance`` decides every tolerance-based GPU parity verdict, so
it is pinned by hand-made outputs just inside and just outside each of its
bounds: the elementwise bound |Y - Yref| <= 1e-2 A + 1e-3, the relative
Frobenius bound 1e-3, the all-zero reference (which requires Y == 0 exactly),
and NaN. ``oracle.activation`` and ``oracle.linear_epilogue`` are pinned
against PyTorch's own CPU routines in float64 (``F.linear``, ``F.relu``,
``F.gelu(approximate="tanh")``, ``F.silu``), and the bias path exactly by
carrying the bias as an extra weight column against a row of ones through
``oracle.masked_gemm``. Each function also gets planted mistakes (its source
with one change, compiled here) that at least one pin must reject.
"""
from __future__ import annotations

import inspect
import textwrap

import numpy as np
import pytest

import oracle


# --- check_tolerance ---------------------------------------------------------

def _ref(shape=(4, 6), seed=0):
    rng = np.random.default_rng(seed)
    Yref = rng.normal(size=shape)
    A = np.abs(Yref) + rng.uniform(0.5, 2.0, size=shape)
    return Yref, A


def pin_accepts_exact(check):
    Yref, A = _ref()
    assert check(Yref.copy(), Yref, A)["ok"]


def pin_accepts_just_inside_elementwise(check):
    """One element at 0.999 of its bound, the rest exact: accepted (its Frobenius error stays small)."""
    Yref, A = _ref(shape=(8, 64))
    Yref[0, 0], A[0, 0] = 40.0, 1.0  # bound 0.011, Frobenius share tiny next to |Yref|
    Y = Yref.copy()
    Y[0, 0] += 0.999 * (1e-2 * A[0, 0] + 1e-3)
    r = check(Y, Yref, A)
    assert r["ok"] and r["ok_elem"] and r["ok_frob"], r


def pin_rejects_just_outside_elementwise(check):
    """One element at 1.001 of its bound: rejected, by the elementwise test."""
    Yref, A = _ref(shape=(8, 64))
    Yref[0, 0], A[0, 0] = 40.0, 1.0
    Y = Yref.copy()
    Y[3, 5] -= 1.001 * (1e-2 * A[3, 5] + 1e-3)
    r = check(Y, Yref, A)
    assert not r["ok"] and not r["ok_elem"], r


def pin_rejects_frobenius_only(check):
    """Every element within its bound, yet a relative Frobenius error of 2e-3: rejected."""
    Yref = np.ones((4, 6))
    A = np.full((4, 6), 100.0)  # elementwise bound 1.001
    Y = Yref * (1.0 + 2e-3)
    r = check(Y, Yref, A)
    assert r["ok_elem"] and not r["ok_frob"] and not r["ok"], r
    # and just inside the Frobenius bound: accepted
    r = check(Yref * (1.0 + 0.9e-3), Yref, A)
    assert r["ok"], r


def pin_zero_reference_needs_exact_zero(check):
    """With Yref == 0 (e.g. an all-zero mask), any nonzero Y is rejected, even one inside the bound."""
    Yref = np.zeros((3, 5))
    A = np.zeros((3, 5))
    assert check(np.zeros((3, 5)), Yref, A)["ok"]
    Y = np.zeros((3, 5))
    Y[1, 2] = 1e-4  # below the 1e-3 absolute bound
    r = check(Y, Yref, A)
    assert not r["ok"], r


def pin_rejects_nan(check):
    Yref, A = _ref()
    Y = Yref.copy()
    Y[2, 3] = np.nan
    r = check(Y, Yref, A)
    assert not r["ok"] and not r["ok_elem"], r


def pin_rejects_inf(check):
    Yref, A = _ref()
    Y = Yref.copy()
    Y[1, 1] = np.inf
    assert not check(Y, Yref, A)["ok"]


CHECK_PINS = [pin_accepts_exact, pin_accepts_just_inside_elementwise, pin_rejects_just_outside_elementwise,
              pin_rejects_frobenius_only, pin_zero_reference_needs_exact_zero, pin_rejects_nan, pin_rejects_inf]


def _mutant(fn, old: str, new: str):
    """fn's source with one substring replaced, compiled in the oracle module's namespace."""
    src = textwrap.dedent(inspect.getsource(fn))
    assert src.count(old) >= 1, (fn.__name__, old)
    ns = dict(vars(oracle))
    exec(compile(src.replace(old, new, 1), f"<mutant of {fn.__name__}>", "exec"), ns)
    return ns[fn.__name__]


@pytest.mark.parametrize("pin", CHECK_PINS, ids=[p.__name__ for p in CHECK_PINS])
def test_check_tolerance_pin(pin):
    pin(oracle.check_tolerance)


CHECK_MUTANTS = [
    ("np.all(err <= bound)", "np.any(err <= bound)"),           # any element instead of all
    ("ok=ok_elem and ok_frob", "ok=ok_elem"),                   # Frobenius term dropped
    ("bound = rel * A + abs_", "bound = rel * A + 10 * abs_"),   # absolute term too loose
    ("bound = rel * A + abs_", "bound = 2 * rel * A + abs_"),    # relative term too loose
    ("ok_frob = frob_err == 0.0", "ok_frob = frob_err <= frob"),  # zero reference treated as relative
    ("err = np.abs(Y - Yref)", "err = np.nan_to_num(np.abs(Y - Yref))"),  # NaN passes
]


@pytest.mark.parametrize("old,new", CHECK_MUTANTS)
def test_check_tolerance_pins_catch_planted_mistake(old, new):
    bad = _mutant(oracle.check_tolerance, old, new)
    caught = []
    for pin in CHECK_PINS:
        try:
            pin(bad)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin caught: {old!r} -> {new!r}"


# --- activation and linear_epilogue ------------------------------------------

def _torch_act(torch, v, act):
    F = torch.nn.functional
    return {0: lambda t: t, 1: F.relu, 2: lambda t: F.gelu(t, approximate="tanh"), 3: F.silu}[act](v)


def pin_activations_match_torch(activation, linear_epilogue):
    """Each activation equals PyTorch's float64 CPU routine to 1e-12 relative, 1e-13 absolute
    (the tanh form of GELU cancels to ~|x| 2^-53 far below zero, where the two differ by rounding)."""
    import torch
    x = np.concatenate([np.linspace(-30.0, 30.0, 6001), [0.0, -0.0, 1e-300, -1e-300]])
    for act in (0, 1, 2, 3):
        got = activation(x, act)
        exp = _torch_act(torch, torch.from_numpy(x.copy()), act).numpy()
        assert np.allclose(got, exp, rtol=1e-12, atol=1e-13), act


def _layer(seed=5, M=40, K=300, N=7):
    import workloads as wl
    W, mask, X = wl.make_random(M, K, N, 0.5, seed=seed)
    rng = np.random.default_rng(seed + 1)
    bias = rng.normal(0.0, 0.5, M).astype(np.float16).view(np.uint16)
    res = rng.normal(0.0, 1.0, (N, M)).astype(np.float16).view(np.uint16)
    return W, mask, X, bias, res


def pin_epilogue_matches_torch_linear(activation, linear_epilogue):
    """act(W X + bias) + residual equals F.linear in float64, then PyTorch's activation and add,
    to 1e-12 relative; with a residual whose sign and size make its place (before or after the
    activation) matter."""
    import torch
    W, mask, X, bias, res = _layer()
    Yref, A = oracle.masked_gemm(W, mask, X)
    Wm = torch.from_numpy(oracle.f16_to_f64(oracle.masked_bits(W, mask)))
    Xt = torch.from_numpy(oracle.f16_to_f64(X))
    b = oracle.f16_to_f64(bias)
    r = oracle.f16_to_f64(res)
    lin = torch.nn.functional.linear(Xt, Wm, torch.from_numpy(b))
    for act in (0, 1, 2, 3):
        exp = (_torch_act(torch, lin, act) + torch.from_numpy(r)).numpy()
        got, _ = linear_epilogue(Yref, A, act, bias=b, residual=r)
        scale = np.abs(exp) + 1.0
        assert np.max(np.abs(got - exp) / scale) < 1e-12, act
    # without bias and residual the epilogue is the identity on the product
    got, sc = linear_epilogue(Yref, A, 0)
    assert np.array_equal(got, Yref) and np.array_equal(sc, A)


def pin_bias_is_an_extra_column(activation, linear_epilogue):
    """The bias path exactly: a bias is the product's last term when it is stored as one more
    weight column (kept) and X gets one more feature equal to 1; the oracle then sums it last,
    as the epilogue adds it, so both Y and the error scale agree bit for bit."""
    W, mask, X, bias, _ = _layer(seed=9)
    M, K = W.shape
    N = X.shape[0]
    W2 = np.concatenate([W, bias[:, None]], axis=1)
    m2 = np.concatenate([mask, np.ones((M, 1), np.uint8)], axis=1)
    X2 = np.concatenate([X, np.full((N, 1), 0x3C00, np.uint16)], axis=1)  # 1.0
    Y2, A2 = oracle.masked_gemm(W2, m2, X2)
    Yref, A = oracle.masked_gemm(W, mask, X)
    y, s = linear_epilogue(Yref, A, 0, bias=oracle.f16_to_f64(bias))
    assert np.array_equal(y, Y2) and np.array_equal(s, A2)


def pin_scale_bounds_the_propagated_error(activation, linear_epilogue):
    """The error scale carries a product error e (|e| <= A) through the epilogue: for every
    activation, |act(z + e) + r - (act(z) + r)| <= scale, checked on the extreme errors e = +-A;
    and the slope bound it uses is at least the largest slope of tanh-GELU and SiLU (autograd,
    float64) and within 1% of it."""
    import torch
    W, mask, X, bias, res = _layer(seed=13)
    Yref, A = oracle.masked_gemm(W, mask, X)
    b, r = oracle.f16_to_f64(bias), oracle.f16_to_f64(res)
    for act in (0, 1, 2, 3):
        y, scale = linear_epilogue(Yref, A, act, bias=b, residual=r)
        for sgn in (1.0, -1.0):
            y2, _ = linear_epilogue(Yref + sgn * A, A, act, bias=b, residual=r)
            assert np.all(np.abs(y2 - y) <= scale * (1 + 1e-12)), act
    # where the activations are steepest (tanh-GELU near 1.5, SiLU near 2.4) a product error
    # grows by the slope, so the scale must too
    z = np.array([[1.5, 2.4, -0.5]])
    a = np.full_like(z, 0.01)
    for act in (2, 3):
        y, scale = linear_epilogue(z, a, act)
        y2, _ = linear_epilogue(z + a, a, act)
        assert np.all(np.abs(y2 - y) <= scale), act
    x = torch.linspace(-10.0, 10.0, 200001, dtype=torch.float64, requires_grad=True)
    worst = 0.0
    for act in (2, 3):
        (g,) = torch.autograd.grad(_torch_act(torch, x, act).sum(), x)
        worst = max(worst, float(g.abs().max()))
    assert worst <= oracle.ACT_SLOPE_BOUND < 1.01 * worst, worst


def pin_scale_covers_output_rounding(activation, linear_epilogue):
    """The output is rounded to fp16 once, after the bias, activation and residual; that
    rounding (up to half an fp16 ulp of the output) must fit the acceptance bound 1e-2 scale +
    1e-3 even where the product is zero and the bias or residual carries the whole value."""
    rng = np.random.default_rng(21)
    N, R = 16, 64
    zero = np.zeros((N, R))
    b = rng.normal(0.0, 300.0, R).astype(np.float16).astype(np.float64)
    r = rng.normal(0.0, 300.0, (N, R)).astype(np.float16).astype(np.float64)
    for act in (0, 1, 2, 3):
        for kw in (dict(bias=b), dict(residual=r), dict(bias=b, residual=r)):
            y, scale = linear_epilogue(zero, zero, act, **kw)
            rounded = y.astype(np.float16).astype(np.float64)
            assert np.all(np.abs(rounded - y) <= 1e-2 * scale + 1e-3), (act, sorted(kw))


EPI_PINS = [pin_activations_match_torch, pin_epilogue_matches_torch_linear, pin_bias_is_an_extra_column,
            pin_scale_bounds_the_propagated_error, pin_scale_covers_output_rounding]


@pytest.mark.parametrize("pin", EPI_PINS, ids=[p.__name__ for p in EPI_PINS])
def test_epilogue_pin(pin):
    pin(oracle.activation, oracle.linear_epilogue)


# Planted mistakes: (function, old, new).
EPI_MUTANTS = [
    ("activation", "np.sqrt(2.0 / np.pi)", "0.8"),                          # GELU constant off
    ("activation", "0.044715 * v ** 3", "0.04 * v ** 3"),                   # GELU cubic term off
    ("activation", "v / (1.0 + np.exp(-v))", "v / (1.0 + np.exp(v))"),      # SiLU sign
    ("activation", "np.maximum(v, 0.0)", "np.maximum(v, 0.0) + 0.0 * v + (v < -20) * v"),  # ReLU leaks
    ("linear_epilogue", "y = activation(z, act)", "y = activation(z + (0.0 if residual is None else residual), act)"),  # residual before act
    ("linear_epilogue", "z = Yref + (0.0 if bias is None else bias[None, :])", "z = Yref - (0.0 if bias is None else bias[None, :])"),  # bias sign
    ("linear_epilogue", "scale = ACT_SLOPE_BOUND * scale", "scale = 1.0 * scale"),  # slope ignored
    ("linear_epilogue", "scale = scale + np.abs(residual)", "scale = scale"),        # residual not in scale
    ("linear_epilogue", "scale = A + (0.0 if bias is None else np.abs(bias)[None, :])", "scale = A"),  # bias not in scale
]


@pytest.mark.parametrize("fname,old,new", EPI_MUTANTS)
def test_epilogue_pins_catch_planted_mistake(fname, old, new):
    act, epi = oracle.activation, oracle.linear_epilogue
    if fname == "activation":
        act = _mutant(oracle.activation, old, new)
        # the epilogue must use the mutated activation too
        src = textwrap.dedent(inspect.getsource(oracle.linear_epilogue))
        ns = dict(vars(oracle))
        ns["activation"] = act
        exec(compile(src, "<epilogue over mutant activation>", "exec"), ns)
        epi = ns["linear_epilogue"]
    else:
        epi = _mutant(oracle.linear_epilogue, old, new)
    caught = []
    for pin in EPI_PINS:
        try:
            pin(act, epi)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin caught {fname}: {old!r} -> {new!r}"
