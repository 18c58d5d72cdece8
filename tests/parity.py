"""Comparison helpers for the GPU-vs-oracle parity tests.

Two metrics per tensor and per step (b: the oracle's value):
    rel(a, b)      = ||a - b||_2 / ||b||_2             relative 2-norm error
    normwise(a, b) = max_i |a_i - b_i| / max_i |b_i|   max-abs normwise error
The bound applies to the maximum over steps: 1e-4 for float32 stages and 2e-2
for bf16 stages. The stepwise tests gate both (check2); the free-running
trajectory tests gate the 2-norm (check).

The weight change W_t - W_0 gets one more term: W is stored in float32 on both
sides, so a value computed on opposite sides of a float32 rounding boundary is
stored one float32 step apart, at most 2^-23 |W| per element. The bound on the
weight change is therefore tol + 2^-23 ||W_t|| / ||W_t - W_0|| in the 2-norm
and tol + 2^-23 max|W_t| / max|W_t - W_0| in the max-abs norm, which matters
only in the first steps of float32 stages (one step of the float32 MLP moves W
by ~1e-3 of its norm).
"""
import numpy as np

import synth
from oracle import trajectory

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def rel(a, b):
    a = np.asarray(a, np.float64).reshape(-1)
    b = np.asarray(b, np.float64).reshape(-1)
    if b.size == 0:
        return 0.0
    return float(np.linalg.norm(a - b) / max(float(np.linalg.norm(b)), 1e-300))


def normwise(a, b):
    a = np.asarray(a, np.float64).reshape(-1)
    b = np.asarray(b, np.float64).reshape(-1)
    if b.size == 0:
        return 0.0
    return float(np.max(np.abs(a - b)) / max(float(np.max(np.abs(b))), 1e-300))


def dw_bound(tol, W_t, W0):
    dW = np.linalg.norm(np.asarray(W_t, np.float64) - np.asarray(W0, np.float64))
    return tol + 2.0 ** -23 * float(np.linalg.norm(W_t)) / max(float(dW), 1e-300)


class Worst:
    """Running maxima of both metrics per quantity, with the bound checked."""

    def __init__(self, name):
        self.name = name
        self.rel = {}
        self.nw = {}

    def check(self, key, a, b, bound, where=""):
        r, n = rel(a, b), normwise(a, b)
        self.rel[key] = max(self.rel.get(key, 0.0), r)
        self.nw[key] = max(self.nw.get(key, 0.0), n)
        assert r <= bound, (self.name, key, where, r, bound)

    def check2(self, key, a, b, bound, where=""):
        """Both metrics within the bound."""
        r, n = rel(a, b), normwise(a, b)
        self.rel[key] = max(self.rel.get(key, 0.0), r)
        self.nw[key] = max(self.nw.get(key, 0.0), n)
        assert r <= bound and n <= bound, (self.name, key, where, r, n, bound)

    def check_dw(self, a, b, W_t, tol, where=""):
        """The step's weight change in both metrics, with the float32 storage
        floor of the weights added to each bound."""
        W_t = np.asarray(W_t, np.float64).reshape(-1)
        r, n = rel(a, b), normwise(a, b)
        db = np.asarray(b, np.float64).reshape(-1)
        br = tol + 2.0 ** -23 * float(np.linalg.norm(W_t)) / max(float(np.linalg.norm(db)), 1e-300)
        bn = tol + 2.0 ** -23 * float(np.max(np.abs(W_t))) / max(float(np.max(np.abs(db))), 1e-300)
        self.rel["step dW"] = max(self.rel.get("step dW", 0.0), r)
        self.nw["step dW"] = max(self.nw.get("step dW", 0.0), n)
        assert r <= br and n <= bn, (self.name, "step dW", where, r, br, n, bn)

    def note(self, key, a, b):
        """Record both metrics without a bound (diagnostic only)."""
        self.rel[key] = max(self.rel.get(key, 0.0), rel(a, b))
        self.nw[key] = max(self.nw.get(key, 0.0), normwise(a, b))

    def report(self):
        return ", ".join(f"{k}: rel {self.rel[k]:.2e} maxabs {self.nw[k]:.2e}" for k in self.rel)


def synthetic_inputs(spec, m):
    x = synth.stage_input(spec, m)
    dy = synth.upstream_grad(spec, m) if spec.head == "none" else None
    lab = synth.labels(spec, m) if spec.head == "ce" else None
    return x, dy, lab


def oracle_trajectory(wl, steps=None, keep_io=True):
    states = {}
    r = trajectory.run(wl, steps=steps, keep_io=keep_io,
                       on_update=lambda k, u, W, v: states.__setitem__((k, u), (W.copy(), v.copy())))
    return r, states
