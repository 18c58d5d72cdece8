"""Run a workload's stages through the pipeline order (test infrastructure only).

At every task the stage predicts its weights from its current (W, v) with the
version difference of Eq. 5 (forward) or Eq. 6 (backward) and Eq. 4, rounds
them to the operand format, and runs the pass; each backward is followed by
the momentum update of Eq. 1 and W <- W - eta v (Section 3.2). Initial v is
zero, so every prediction before the first update returns W0. A stage whose
spec names the "vanilla" or "stash" policy (the comparison of Section 4.2)
uses s = 0 instead; under "stash" the backward of a mini-batch reuses the
weights its forward used.

A workload either simulates all N stages of a pipeline (mini-batch m enters
stage 0 with its synthetic input; each stage's output feeds the next; the last
stage's loss head starts the backward) or a single stage k of N (its input and
upstream gradient, or labels, are the synthetic draws for that stage).
"""
from typing import Callable, Dict, List, Optional

import numpy as np

import synth

from . import method, schedule, stages


class StageState:
    def __init__(self, spec, W0):
        self.spec = spec
        self.W = np.asarray(W0, np.float64).copy()
        self.v = np.zeros_like(self.W)
        self.updates = 0
        self.stash: Dict[int, dict] = {}
        # eta and gamma cross the library boundary as float32
        self.lr = float(np.float32(spec.lr))
        self.gamma = float(np.float32(spec.momentum))

    def predicted(self, forward: bool):
        s_f, s_b = method.staleness_versions(getattr(self.spec, "policy", "spectrain"),
                                             self.spec.stage_index, self.spec.num_stages)
        What = method.predict(self.W, self.v, s_f if forward else s_b, self.lr)
        return stages.unpack(self.spec, stages.weight_rounder(self.spec)(What))


def run(workload, steps: Optional[int] = None, exact: bool = False,
        W0: Optional[List[np.ndarray]] = None,
        v0: Optional[List[np.ndarray]] = None,
        inputs: Optional[Callable] = None,
        on_update: Optional[Callable] = None,
        keep_io: bool = False) -> dict:
    """Simulate `steps` mini-batches (default workload.steps).

    on_update(stage_index, update_count, W, v) is called after every update.
    inputs(spec, m) may override the synthetic (x, dy, labels) draws.
    Returns {"loss": {m: loss}, "y": {(k, m): y}, "dx": {(k, m): dx}} (y and dx
    only with keep_io) plus the final states {"W": [...], "v": [...]}.
    """
    specs = workload.stages
    M = workload.steps if steps is None else steps
    N = specs[0].num_stages
    full = len(specs) == N
    st = {}
    for i, spec in enumerate(specs):
        w0 = synth.initial_params(spec) if W0 is None else W0[i]
        st[spec.stage_index] = StageState(spec, w0)
        if v0 is not None:
            st[spec.stage_index].v = np.asarray(v0[i], np.float64).copy()

    def draw(spec, m):
        if inputs is not None:
            return inputs(spec, m)
        x = synth.stage_input(spec, m)
        dy = synth.upstream_grad(spec, m) if spec.head == "none" else None
        lab = synth.labels(spec, m) if spec.head == "ce" else None
        return x, dy, lab

    if full:
        tasks = schedule.pipeline_tasks(N, M)
    else:
        k = specs[0].stage_index
        tasks = [(k, kind, m) for kind, m in schedule.stage_tasks(k, N, M)]

    out = {"loss": {}, "y": {}, "dx": {}}
    handoff_y: Dict[tuple, np.ndarray] = {}
    handoff_dx: Dict[tuple, np.ndarray] = {}
    for k, kind, m in tasks:
        S = st[k]
        spec = S.spec
        if kind == "F":
            x, dy, lab = draw(spec, m)
            if full and k > 0:
                x = handoff_y.pop((k - 1, m))
            P = S.predicted(forward=True)
            y, loss, stash = stages.forward(spec, P, x, lab, exact=exact)
            stash["dy"] = dy
            if getattr(spec, "policy", "spectrain") == "stash":
                stash["weights"] = P         # the backward of m reuses these (weight stashing)
            S.stash[m] = stash
            if loss is not None:
                out["loss"][m] = loss
            if full and k < N - 1:
                handoff_y[(k, m)] = y
            if keep_io:
                out["y"][(k, m)] = y
        else:
            stash = S.stash.pop(m)
            dy = stash["dy"]
            if full and k < N - 1:
                dy = handoff_dx.pop((k + 1, m))
            P = stash["weights"] if "weights" in stash else S.predicted(forward=False)
            dx, grads = stages.backward(spec, P, stash, dy, exact=exact)
            g = stages.pack(spec, grads)
            S.W, S.v = method.momentum_sgd_step(S.W, S.v, g, S.lr, S.gamma)
            S.updates += 1
            if full and k > 0:
                handoff_dx[(k, m)] = dx
            if keep_io:
                out["dx"][(k, m)] = dx
            if on_update is not None:
                on_update(k, S.updates, S.W, S.v)
    out["W"] = [st[s.stage_index].W for s in specs]
    out["v"] = [st[s.stage_index].v for s in specs]
    return out
