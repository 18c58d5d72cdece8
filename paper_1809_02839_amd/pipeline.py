"""One-forward-one-backward pipeline driver on one GPU.

Runs the stages of a K-stage pipeline (or a single stage k of N) through the
task order of pipelined model parallelism (Section 3.1 of the paper: forward
and backward tasks issued round-robin, several mini-batches in flight, one
weight update per backward). Each stage sees exactly the weight versions it
would see on its own GPU: before its forward it uses weights predicted with the
forward version difference (Eq. 5) and before its backward the ones predicted
with the backward difference (Eq. 6); the fused update after every backward
refreshes W and v and re-predicts both (Eq. 1, Eq. 4). A stage whose spec
names the Vanilla or stashing policy uses s = 0 instead (Section 4.2), the
latter with the library's weight stash for its backward passes.

Device memory and streams come from torch; every step of the stage runs in
libspectrain.so through the C ABI.
"""
from typing import Callable, Dict, List, Optional, Tuple

import numpy as np
import torch

from . import native


def stage_task_order(k: int, N: int, M: int) -> List[Tuple[str, int]]:
    """Stage k of N: N - k warm-up forwards, then alternate one backward and
    one forward while forwards remain, then drain the backwards."""
    warm = min(N - k, M)
    order = [("F", m) for m in range(warm)]
    nf, nb = warm, 0
    while nb < M:
        order.append(("B", nb))
        nb += 1
        if nf < M:
            order.append(("F", nf))
            nf += 1
    return order


def pipeline_task_order(N: int, M: int) -> List[Tuple[int, str, int]]:
    """Interleave the stage orders: in each round every stage whose next task
    has its inputs (the previous stage's forward, the next stage's backward,
    or its own forward at the last stage) runs it."""
    orders = [stage_task_order(k, N, M) for k in range(N)]
    pos = [0] * N
    done = set()
    seq = []
    while any(pos[k] < len(orders[k]) for k in range(N)):
        ready = []
        for k in range(N):
            if pos[k] >= len(orders[k]):
                continue
            kind, m = orders[k][pos[k]]
            if kind == "F":
                ok = k == 0 or (k - 1, "F", m) in done
            else:
                ok = (k + 1, "B", m) in done if k < N - 1 else (k, "F", m) in done
            if ok:
                ready.append((k, kind, m))
        if not ready:
            raise RuntimeError("pipeline order deadlocked")
        for t in ready:
            seq.append(t)
            done.add(t)
            pos[t[0]] += 1
    return seq


def torch_dtype(spec):
    return torch.bfloat16 if spec.dtype == "bf16" else torch.float32


def to_device(a, spec, device, integer=False):
    if a is None or isinstance(a, torch.Tensor):
        return a
    t = torch.from_numpy(np.ascontiguousarray(a))
    if integer:
        return t.to(device=device, dtype=torch.int32)
    return t.to(device=device).to(torch_dtype(spec))


class Pipeline:
    """The simulated stages of one workload.

    inputs(spec, m) returns (x, dy, labels) for mini-batch m at a stage; x is
    used at the first simulated stage (or a single stage), dy at a single stage
    without a loss head, labels at a stage with a CE head; entries that are not
    used may be None. NumPy arrays are uploaded, torch tensors used as given.
    """

    def __init__(self, specs, W0s: List[np.ndarray], device="cuda", stream: Optional[torch.cuda.Stream] = None,
                 v0s: Optional[List[np.ndarray]] = None):
        self.specs = list(specs)
        self.N = self.specs[0].num_stages
        self.full = len(self.specs) == self.N
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.stages: Dict[int, native.Stage] = {}
        self.spec_of: Dict[int, object] = {}
        for spec, W0 in zip(self.specs, W0s):
            st = native.Stage(native.desc_from_spec(spec), W0, self.stream)
            self.stages[spec.stage_index] = st
            self.spec_of[spec.stage_index] = spec
        if v0s is not None:
            for spec, W0, v0 in zip(self.specs, W0s, v0s):
                self.stages[spec.stage_index].set_state(W0, v0)
        versions = {k: native.policy_versions(getattr(self.spec_of[k], "policy", "spectrain"), k, self.N)
                    for k in self.stages}
        self.s_f = {k: versions[k][0] for k in self.stages}
        self.s_b = {k: versions[k][1] for k in self.stages}
        # the first tasks see predictions from the initial (W, v) (Eq. 4)
        for k, st in self.stages.items():
            st.predict(self.s_f[k], 0)
            st.predict(self.s_b[k], 1)

    def tasks(self, M: int):
        if self.full:
            return pipeline_task_order(self.N, M)
        k = self.specs[0].stage_index
        return [(k, kind, m) for kind, m in stage_task_order(k, self.N, M)]

    def run(self, M: int, inputs: Callable, on_update: Optional[Callable] = None, keep_io: bool = False,
            s_override: Optional[Tuple[int, int]] = None, on_forward: Optional[Callable] = None):
        """Run M mini-batches. on_update(k, count, stage) is called after each
        update, on_forward(k, m, stage) after each forward (synchronise inside
        them if device state is read). Returns
        {"loss": {m: device scalar}, "y": {(k, m): tensor}, "dx": {(k, m): tensor}}."""
        held_x: Dict[Tuple[int, int], torch.Tensor] = {}
        held_y: Dict[Tuple[int, int], torch.Tensor] = {}
        held_dy: Dict[Tuple[int, int], torch.Tensor] = {}
        dx_out: Dict[Tuple[int, int], torch.Tensor] = {}
        labels: Dict[Tuple[int, int], torch.Tensor] = {}
        out = {"loss": {}, "y": {}, "dx": {}}
        counts = {k: 0 for k in self.stages}
        with torch.cuda.stream(self.stream):
            for k, kind, m in self.tasks(M):
                spec = self.spec_of[k]
                st = self.stages[k]
                if kind == "F":
                    x, dy, lab = inputs(spec, m)
                    if self.full and k > 0:
                        x = held_y[(k - 1, m)]      # the previous stage's output
                    else:
                        x = to_device(x, spec, self.device)
                    if self.full and k < self.N - 1:
                        dy = None                   # comes from the next stage's backward
                    dy = to_device(dy, spec, self.device)
                    lab = to_device(lab, spec, self.device, integer=True)
                    held_x[(k, m)] = x
                    if spec.head == "ce":
                        loss = torch.empty(1, dtype=torch.float32, device=self.device)
                        labels[(k, m)] = lab
                        st.forward(m, x, None, lab, loss)
                        out["loss"][m] = loss
                    else:
                        y = torch.empty(spec.output_shape(), dtype=torch_dtype(spec), device=self.device)
                        st.forward(m, x, y)
                        held_y[(k, m)] = y
                        if keep_io:
                            out["y"][(k, m)] = y
                    if dy is not None:
                        held_dy[(k, m)] = dy
                    if on_forward is not None:
                        on_forward(k, m, st)
                else:
                    if self.full and k < self.N - 1:
                        dy = dx_out.pop((k + 1, m))
                    else:
                        dy = held_dy.pop((k, m), None)
                    need_dx = not (self.full and k == 0) or keep_io
                    dx = torch.empty(spec.input_shape(), dtype=torch_dtype(spec), device=self.device) if need_dx else None
                    st.backward(m, dy, dx)
                    sf, sb = (self.s_f[k], self.s_b[k]) if s_override is None else s_override
                    st.update(sf, sb)
                    counts[k] += 1
                    if dx is not None:
                        if self.full and k > 0:
                            dx_out[(k, m)] = dx
                        if keep_io:
                            out["dx"][(k, m)] = dx
                    labels.pop((k, m), None)
                    # the stage no longer references its stash for m; upstream
                    # (k+1) has already run its backward, so y and x can go
                    held_x.pop((k, m), None)
                    held_y.pop((k, m), None)
                    if on_update is not None:
                        on_update(k, counts[k], st)
        return out

    def destroy(self):
        for st in self.stages.values():
            st.destroy()
        self.stages = {}
