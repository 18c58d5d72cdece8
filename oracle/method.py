"""SpecTrain's weight prediction and momentum update (test infrastructure only).

Section 3.2 of the paper:
  Eq. 1   v_t = gamma * v_{t-1} + (1 - gamma) * g_t       (smoothed gradient)
  Eq. 2   W_{t+1} = W_t - eta * g_t                       (plain SGD)
  Eq. 3   W^_{t+1} = W_t - eta * v_{t-1}                  (one-step prediction)
  Eq. 4   W^_{t+s} = W_t - s * eta * v_{t-1}              (s-step prediction)
  Eq. 5   s = floor(k/2) + N - k - 1                      (forward pass at GPU k)
  Eq. 6   s = floor(k/2)                                  (backward pass at GPU k)

Reading: the momentum weight update is not printed. Eq. 3 obtains the
prediction by substituting v for g in Eq. 2, so the update the prediction
anticipates is W_{t+1} = W_t - eta * v_t with v_t from Eq. 1. W and v are
held in float32 (the master format of every workload).
"""
import numpy as np

from .numerics import to_f32


def version_difference(k: int, N: int, forward: bool) -> int:
    """Eq. 5 (forward) / Eq. 6 (backward); k is the 0-based stage index, N the
    number of pipeline stages."""
    if not (0 <= k < N):
        raise ValueError(f"stage index {k} outside [0, {N})")
    if forward:
        return k // 2 + N - k - 1
    return k // 2


def staleness_versions(policy: str, k: int, N: int):
    """Version differences (before a forward, before a backward) under the three
    ways Section 4.2 compares a pipeline stage treating weight staleness:
    SpecTrain predicts (Eq. 5, Eq. 6); Vanilla model parallelism and PipeDream's
    weight stashing start every forward from the latest weights (no prediction,
    s = 0). Under stashing the backward reuses the forward's weights, which the
    caller keeps; under Vanilla it takes the latest weights at its own time."""
    if policy == "spectrain":
        return version_difference(k, N, True), version_difference(k, N, False)
    if policy in ("vanilla", "stash"):
        return 0, 0
    raise ValueError(f"unknown policy {policy!r}")


def predict(W, v, s: int, lr: float):
    """Eq. 4: W^_{t+s} = W_t - s * eta * v_{t-1}, from the current stored pair
    (W_t, v_{t-1}); the result is held as float32 like the master weights."""
    if s < 0:
        raise ValueError("version difference must be >= 0")
    return to_f32(np.asarray(W, np.float64) - s * float(lr) * np.asarray(v, np.float64))


def smoothed_gradient(v, g, gamma: float):
    """Eq. 1: v_t = gamma * v_{t-1} + (1 - gamma) * g_t, stored as float32."""
    gamma = float(gamma)
    return to_f32(gamma * np.asarray(v, np.float64) + (1.0 - gamma) * np.asarray(g, np.float64))


def weight_update(W, v_new, lr: float):
    """Momentum form of Eq. 2 with g replaced by the fresh smoothed gradient:
    W_{t+1} = W_t - eta * v_t, stored as float32."""
    return to_f32(np.asarray(W, np.float64) - float(lr) * np.asarray(v_new, np.float64))


def momentum_sgd_step(W, v, g, lr: float, gamma: float):
    """One weight update after a backward pass: Eq. 1, then the update."""
    v_new = smoothed_gradient(v, to_f32(g), gamma)
    return weight_update(W, v_new, lr), v_new
