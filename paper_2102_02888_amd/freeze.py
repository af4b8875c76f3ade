"""When to end the Adam warm-up (Section 7.1, warm-up auto-tuning).

The paper freezes the variance once it has become stable, and gives a rule
to find that point: the warm-up lasts at least as long as the learning-rate
warm-up, and ends at the first step t whose variance l1 norm has stopped
shrinking, ||v_t||_1 / ||v_{t-Delta}||_1 >= 0.96 with Delta = 1/(1-beta2).
This is host-side bookkeeping over one fp64 norm per step, which the GPU
computes with onebit_l1_norm.
"""
from collections import deque


class VarianceFreezeDetector:
    def __init__(self, beta2, threshold=0.96, min_steps=0):
        self.delta = int(round(1.0 / (1.0 - float(beta2))))
        self.threshold = float(threshold)
        self.min_steps = int(min_steps)
        self._norms = deque(maxlen=self.delta + 1)
        self._last_t = 0
        self.frozen_at = None

    def update(self, t, norm):
        """Records ||v_t||_1 of warm-up step t (1-based, consecutive) and
        returns True if the warm-up should end after step t."""
        if t != self._last_t + 1:
            raise ValueError("steps must be consecutive (got %d after %d)" % (t, self._last_t))
        self._last_t = t
        self._norms.append(float(norm))
        if self.frozen_at is not None:
            return True
        if t < self.min_steps or len(self._norms) <= self.delta:
            return False
        past = self._norms[0]  # the norm at step t - delta
        if past > 0.0 and self._norms[-1] >= self.threshold * past:
            self.frozen_at = t
            return True
        return False
