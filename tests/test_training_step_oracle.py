"""Pins of the training-step oracle (dynamic loss scaling of Sec. 3.3,
Listing 6; the fp32 momentum-SGD update) against facts fixed independently of
its code: counts worked out by hand from the listing's order of operations,
closed forms, and invariants."""
import numpy as np
import pytest

from oracle.training_step import LossScaler, sgd_update


def test_first_growth_on_step_2002_then_every_2001():
    """Listing 6 with factor 2, interval 2000, counter starting at 0: after
    k clean steps the counter is k, so the test `counter > 2000` first holds
    at the start of clean step 2002; afterwards the counter restarts at 0
    and is incremented to 1 in the same step, so the test next holds 2001
    steps later."""
    s = LossScaler(scale=8.0)
    growth_steps = []
    for step in range(1, 2002 + 2001 * 2 + 1):
        before = s.scale
        assert s.step(False)
        if s.scale != before:
            growth_steps.append(step)
    assert growth_steps == [2002, 4003, 6004]
    assert s.scale == 64.0


def test_overflow_halves_resets_and_skips():
    s = LossScaler(scale=1024.0, interval=3)
    assert s.step(False) and s.counter == 1
    assert s.step(False) and s.counter == 2
    assert not s.step(True)
    assert s.scale == 512.0 and s.counter == 0 and s.skipped == 1
    # growth needs counter > 3 at the test: steps 1..4 build it to 4, step 5 grows
    applied = [s.step(False) for _ in range(5)]
    assert all(applied)
    assert s.scale == 1024.0 and s.counter == 1


def test_alternating_overflow_never_grows():
    """interval 1: a clean step only raises the counter to 1 (growth needs
    counter > 1 at the test), and every overflow halves and resets."""
    s = LossScaler(scale=2.0 ** 20, interval=1)
    for _ in range(50):
        s.step(False)
        s.step(True)
    assert s.scale == 2.0 ** -30
    assert s.skipped == 50 and s.counter == 0


class _IncrementFirst(LossScaler):
    def step(self, overflow):
        if overflow:
            return super().step(True)
        self.counter += 1
        if self.counter > self.interval:
            self.scale *= self.factor
            self.counter = 0
        return True


class _NoResetOnOverflow(LossScaler):
    def step(self, overflow):
        if overflow:
            self.scale /= self.factor
            self.skipped += 1
            return False
        return super().step(False)


class _GreaterEqual(LossScaler):
    def step(self, overflow):
        if overflow:
            return super().step(True)
        if self.counter >= self.interval:
            self.scale *= self.factor
            self.counter = 0
        self.counter += 1
        return True


@pytest.mark.parametrize("bad", [_IncrementFirst, _NoResetOnOverflow, _GreaterEqual])
def test_pins_catch_plausible_mistakes(bad, monkeypatch):
    """Each plausible misreading of the listing fails at least one pin."""
    import tests.test_training_step_oracle as me
    monkeypatch.setattr(me, "LossScaler", bad)
    failed = 0
    for pin in (me.test_first_growth_on_step_2002_then_every_2001,
                me.test_overflow_halves_resets_and_skips,
                me.test_alternating_overflow_never_grows):
        try:
            pin()
        except AssertionError:
            failed += 1
    assert failed >= 1


def test_sgd_constant_gradient_closed_form():
    """With a constant gradient g and no weight decay, v_t = g (1 - mu^t) /
    (1 - mu) and w_t = w_0 - lr g sum_{i=1..t} (1 - mu^i) / (1 - mu)."""
    rng = np.random.default_rng(0)
    w0 = rng.standard_normal(17)
    g = rng.standard_normal(17)
    lr, mu, t = 0.1, 0.9, 12
    w, v = w0.copy(), np.zeros(17)
    for _ in range(t):
        w, v = sgd_update(w, v, g * 4.0, 4.0, lr, mu, 0.0)
    vt = g * (1 - mu ** t) / (1 - mu)
    wt = w0 - lr * g * sum((1 - mu ** i) / (1 - mu) for i in range(1, t + 1))
    np.testing.assert_allclose(v, vt, rtol=1e-12)
    np.testing.assert_allclose(w, wt, rtol=1e-12, atol=1e-12)


def test_sgd_weight_decay_only_shrinks_geometrically():
    """Zero gradient, zero momentum: w_t = w_0 (1 - lr * wd)^t."""
    w0 = np.linspace(-2, 3, 11)
    w, v = w0.copy(), np.zeros(11)
    for _ in range(5):
        w, v = sgd_update(w, v, np.zeros(11), 1.0, 0.5, 0.0, 0.1)
    np.testing.assert_allclose(w, w0 * (1 - 0.05) ** 5, rtol=1e-13)


@pytest.mark.parametrize("scale", [1.0, 1024.0, 2.0 ** -3])
def test_sgd_unscale_is_division_by_scale(scale):
    rng = np.random.default_rng(1)
    w0, v0, g = rng.standard_normal((3, 9))
    a = sgd_update(w0, v0, g * scale, scale, 0.01, 0.9, 1e-4)
    b = sgd_update(w0, v0, g, 1.0, 0.01, 0.9, 1e-4)
    np.testing.assert_allclose(a[0], b[0], rtol=1e-14)
    np.testing.assert_allclose(a[1], b[1], rtol=1e-14)
