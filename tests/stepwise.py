"""Re-synchronised per-task parity of the HIP pipeline against the oracle.

The GPU runs the workload's one-forward-one-backward order through the C ABI,
recording its (W, v) after every update, every stage output y and every input
gradient dX. The oracle then recomputes each task from the GPU's own state at
that moment: a forward from the state before it (predicting with Eq. 5's
difference), a backward plus update from the state before that backward
(Eq. 6's difference) and the oracle's own stash of the same mini-batch; in a
full pipeline a stage's input and upstream gradient are the GPU's neighbouring
outputs. Every task is thus compared against an exact recomputation of the
same step, with no divergence carried from earlier steps. Under the Vanilla
and stashing policies the differences are 0 and a stashing backward reuses
the weights the oracle's forward of the same mini-batch used.

With derived=True (every bf16 run) the gradient quantities (v, the step's
weight change, dX) pass when they are within tol of the oracle's bf16
emulation, or else when the GPU is as accurate as that emulation: they are
also recomputed without any bf16 rounding and
    rel(gpu, exact) <= max(tol, 1.5 * rel(oracle_bf16, exact)).
Over many layers the two bf16 computations take different ReLU decisions on
activations within bf16 noise of zero, and each such decision moves a whole
row of a weight gradient, so two correct bf16 implementations differ from
each other about as much as each differs from the exact result (measured
before any GPU run: 5.7 % on the 4-layer VGG stage, 5.4 % on the transformer
stage and 14 % on the 8-block bottleneck stage). Forward outputs, losses and
the weights themselves stay under the plain bound.
"""
import numpy as np

import synth
from oracle import method, stages
from parity import TOL, Worst, dw_bound, rel, synthetic_inputs


def run_stepwise(wl, steps, torch, derived=False):
    from paper_1809_02839_amd.pipeline import Pipeline, stage_task_order

    specs = wl.stages
    N = specs[0].num_stages
    full = len(specs) == N
    W0s = {s.stage_index: synth.initial_params(s) for s in specs}
    pipe = Pipeline(specs, [W0s[s.stage_index] for s in specs])
    states = {}
    out = pipe.run(steps, synthetic_inputs, keep_io=True,
                   on_update=lambda k, u, st: states.__setitem__((k, u), st.get_state()))
    torch.cuda.synchronize()
    y_gpu = {key: t.float().cpu().numpy() for key, t in out["y"].items()}
    dx_gpu = {key: t.float().cpu().numpy() for key, t in out["dx"].items()}
    loss_gpu = {m: t.item() for m, t in out["loss"].items()}
    pipe.destroy()

    worst = Worst(wl.name)
    tol = TOL[specs[0].dtype]
    for spec in specs:
        k = spec.stage_index
        lr = float(np.float32(spec.lr))
        gamma = float(np.float32(spec.momentum))
        policy = getattr(spec, "policy", "spectrain")
        sf, sb = method.staleness_versions(policy, k, N)
        W = W0s[k].astype(np.float64)
        v = np.zeros_like(W)
        u = 0
        stash = {}
        rnd = stages.weight_rounder(spec)
        for kind, m in stage_task_order(k, N, steps):
            x, dy, lab = synthetic_inputs(spec, m)
            if full and k > 0:
                x = y_gpu[(k - 1, m)]
            if kind == "F":
                P = stages.unpack(spec, rnd(method.predict(W, v, sf, lr)))
                y, loss, st = stages.forward(spec, P, x, lab)
                stash[m] = st
                if policy == "stash":
                    stash[("weights", m)] = P   # the backward reuses the forward's weights
                if derived:
                    stash[("exact", m)] = stages.forward(spec, P, x, lab, exact=True)[2]
                if spec.head == "ce":
                    worst.check("loss", [loss_gpu[m]], [loss], tol, f"k{k} m{m}")
                else:
                    worst.check("y", y_gpu[(k, m)], y, tol, f"k{k} m{m}")
            else:
                if full and k < N - 1:
                    dy = dx_gpu[(k + 1, m)]
                if policy == "stash":
                    P = stash.pop(("weights", m))
                else:
                    P = stages.unpack(spec, rnd(method.predict(W, v, sb, lr)))
                dx, grads = stages.backward(spec, P, stash.pop(m), dy)
                W1, v1 = method.momentum_sgd_step(W, v, stages.pack(spec, grads), lr, gamma)
                u += 1
                Wg, vg = states[(k, u)]
                worst.check("W", Wg, W1, tol, f"k{k} u{u}")
                if derived:
                    dxe, ge = stages.backward(spec, P, stash.pop(("exact", m)), dy, exact=True)
                    W1e, v1e = method.momentum_sgd_step(W, v, stages.pack(spec, ge), lr, gamma)
                    pairs = [("v", vg, v1, v1e), ("step dW", Wg.astype(np.float64) - W, W1 - W, W1e - W)]
                    if (k, m) in dx_gpu:
                        pairs.append(("dx", dx_gpu[(k, m)], dx, dxe))
                    for key, a, b, e in pairs:
                        worst.note(key, a, b)
                        if rel(a, b) <= tol:
                            worst.note(key + " vs exact", a, e)
                            continue
                        bound = max(tol, 1.5 * rel(b, e))
                        worst.check(key + " vs exact", a, e, bound, f"k{k} u{u} (oracle bf16 vs exact {rel(b, e):.2e})")
                else:
                    worst.check("v", vg, v1, tol, f"k{k} u{u}")
                    worst.check("step dW", Wg.astype(np.float64) - W, W1 - W, dw_bound(tol, W1, W), f"k{k} u{u}")
                    if (k, m) in dx_gpu:
                        worst.check("dx", dx_gpu[(k, m)], dx, tol, f"k{k} m{m}")
                # continue from the GPU's state: each step is checked on its own
                W, v = Wg.astype(np.float64), vg.astype(np.float64)
    return worst
