"""Pins of the parity measure itself, oracle.rel_err = max|got - ref| /
max|ref| with an exact match required against an all-zero reference, on
hand-computed cases, and planted mistakes in a copy of it that the pins
must reject (a dropped absolute value on either side, a mean instead of a
maximum, a zero-reference rule that lets errors pass, a relative error
taken element by element)."""
import inspect
import math

import numpy as np
import pytest

import oracle.oracle as orc


def check_rel_err(fn):
    """Raises AssertionError when fn disagrees with a hand-computed value."""
    # largest difference over largest reference magnitude: |3 - 4| / 4
    assert fn([1.0, 2.0, 3.0], [1.0, 2.0, 4.0]) == 0.25
    # the reference's largest magnitude is a negative entry: 0.5 / |-4|
    assert fn([-4.0, 1.5], [-4.0, 1.0]) == 0.125
    # the difference is negative everywhere: |(-2) - 0| / 2 over ref [0, 2]
    assert fn([-2.0, 0.0], [0.0, 2.0]) == 1.0
    # sign error: got = -ref gives 2 max|ref| / max|ref|
    assert fn([-3.0, 0.0, 1.0], [3.0, 0.0, -1.0]) == 2.0
    # one outlier among many exact values dominates (a maximum, not a mean)
    ref = np.ones(1000)
    got = ref.copy()
    got[617] += 0.01
    assert abs(fn(got, ref) - 0.01) < 1e-15
    # an error relative to a tiny reference entry is measured against the
    # largest one: |1e-6 - 2e-6| / 1, not 0.5
    assert abs(fn([1.0, 1e-6], [1.0, 2e-6]) - 1e-6) < 1e-18
    # all-zero reference: exact zeros pass, anything else fails
    assert fn(np.zeros(5), np.zeros(5)) == 0.0
    assert fn([0.0, 1e-300, 0.0], [0.0, 0.0, 0.0]) == math.inf
    assert fn([0.0, -1e-300], [0.0, -0.0]) == math.inf
    # shapes are compared element by element after broadcasting as arrays
    assert fn(np.array([[1.0, 2.0], [3.0, 5.0]]), np.array([[1.0, 2.0], [3.0, 4.0]])) == 0.25
    # empty arrays: nothing to compare
    assert fn(np.zeros(0), np.zeros(0)) == 0.0


def test_rel_err_pins():
    check_rel_err(orc.rel_err)


PLANTS = [
    ("no abs on the difference", "np.abs(got - ref)", "(got - ref)"),
    ("no abs on the reference", "np.max(np.abs(ref))", "np.max(ref)"),
    ("mean difference", "float(np.max(np.abs(got - ref)))", "float(np.mean(np.abs(got - ref)))"),
    ("zero reference accepts anything", 'return 0.0 if d == 0.0 else float("inf")', "return 0.0"),
    ("elementwise relative error",
     "return d / m", "return float(np.max(np.abs(got - ref) / np.maximum(np.abs(ref), 1e-300)))"),
]


@pytest.mark.parametrize("name,find,repl", PLANTS, ids=[p[0] for p in PLANTS])
def test_rel_err_plants_are_caught(name, find, repl):
    src = inspect.getsource(orc.rel_err)
    assert find in src, name
    ns = {"np": np}
    exec(src.replace(find, repl), ns)
    with pytest.raises(AssertionError):
        check_rel_err(ns["rel_err"])
