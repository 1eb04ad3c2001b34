"""The plateau schedule of the learning rate and perturbation radius -- test
infrastructure (only the tests use it).

Paper, Section 4 and Table experimental-setup: lr and eps start at 1e-3 and
are decayed together on expert validation plateaus, halved after 1,000
updates without an improvement of 1e-8, with a floor of 1e-5.  Readings:
an improvement is a validation loss below best - threshold (compared in
fp64; best starts at +inf); `since` counts updates since the last
improvement or decay, and a decay happens when it reaches `patience`, after
which it restarts at 0; a decay never raises a rate that is already below
the floor.  Rates are fp32 values (they cross the library boundary as fp32),
so products are fp32 products.
"""
import math

import numpy as np

f32 = np.float32


class Plateau:
    def __init__(self, n, lr0, eps0, factor=0.5, patience=1000, threshold=1e-8, floor=1e-5):
        self.n = int(n)
        self.lr = [f32(lr0)] * self.n
        self.eps = [f32(eps0)] * self.n
        self.best = [f32(math.inf)] * self.n
        self.since = [0] * self.n
        self.factor, self.patience = f32(factor), int(patience)
        self.threshold, self.floor = f32(threshold), f32(floor)

    def _decay(self, x):
        return min(x, max(f32(x * self.factor), self.floor))

    def observe(self, val_loss, updates=1):
        for e in range(self.n):
            v = f32(val_loss[e])
            if float(v) < float(self.best[e]) - float(self.threshold):
                self.best[e] = v
                self.since[e] = 0
            else:
                self.since[e] += int(updates)
            if self.since[e] >= self.patience:
                self.lr[e] = self._decay(self.lr[e])
                self.eps[e] = self._decay(self.eps[e])
                self.since[e] = 0

    def state(self):
        return (np.array(self.lr, np.float32), np.array(self.eps, np.float32),
                np.array(self.best, np.float32), np.array(self.since, np.int32))
