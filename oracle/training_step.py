"""Oracle for the two training-step pieces that follow the convolution passes:
dynamic loss scaling and the fp32 master-weight update.

TEST INFRASTRUCTURE ONLY.  Only the test-suite imports this module.  It
never imports the GPU package and the GPU package never imports it.

Dynamic loss scaling (Sec. 3.3, Listing 6).  Per training step, after the
backward pass: when the gradients hold an inf or a NaN, the loss scale is
divided by the scaling factor, the step counter goes back to zero and the
update is skipped.  Otherwise the gradients are divided by the loss scale,
the solver updates the weights, and then -- in this order -- the scale is
multiplied by the factor if the counter has passed the interval (the
counter then restarts at zero), and finally the counter grows by one.  With
factor 2 and interval 2000 the first growth therefore happens on the
2002nd consecutive clean step and each later one 2001 clean steps after the
previous.

Master-weight update (Sec. 3.3: half-precision storage, fp32 update of fp32
master weights that also exist as a half-precision copy).  The paper does
not name the solver; this file uses momentum SGD with L2 weight decay,
written as
    g = grad / scale + weight_decay * w
    v = momentum * v + g
    w = w - lr * v
    w16 = round_to_nearest_even(w)
everything in float64 here (the GPU computes in fp32).
"""
from __future__ import annotations

import dataclasses

import numpy as np


@dataclasses.dataclass
class LossScaler:
    scale: float
    factor: float = 2.0
    interval: int = 2000
    counter: int = 0
    skipped: int = 0

    def step(self, overflow: bool) -> bool:
        """Advance one training step; returns True when the update is
        applied (no inf/NaN in the gradients).

        Written as the transition the rule defines, not in the listing's
        statement order: a clean step grows the scale exactly when more than
        `interval` clean steps were counted before it; the counter then holds
        the clean steps since the last growth or overflow, this one
        included."""
        ovf = bool(overflow)
        grow = (not ovf) and self.counter > self.interval
        # an overflow divides by the factor (not a multiply by its
        # reciprocal, which rounds differently for other than powers of two)
        self.scale = self.scale / self.factor if ovf else \
            self.scale * (self.factor if grow else 1.0)
        self.counter = 0 if ovf else (1 if grow else self.counter + 1)
        self.skipped += int(ovf)
        return not ovf


def sgd_update(master, momentum, grad, scale, lr, mu, weight_decay):
    """One momentum-SGD step on float64 copies; returns (master, momentum)."""
    w = np.asarray(master, np.float64)
    v = np.asarray(momentum, np.float64)
    g = np.asarray(grad, np.float64) / scale + weight_decay * w
    v = mu * v + g
    w = w - lr * v
    return w, v
