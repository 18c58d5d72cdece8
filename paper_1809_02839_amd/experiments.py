"""Experiments of the paper that run on the stage library (Section 3.2, 4.2).

prediction_rmse
    Prediction accuracy (Section 3.2, Fig. 7): one stage trained with momentum
    SGD and no pipeline staleness (N = 1); after every update t the library
    predicts W_{t+s} from (W_t, v_t) with Eq. 4 for each s, and when step t + s
    arrives the RMSE of that prediction against the actual W_{t+s} is set beside
    the RMSE of the stale weights W_t against W_{t+s}.

policy_losses
    The three treatments of weight staleness the evaluation compares (Section
    4.2: Vanilla pipelining, PipeDream's weight stashing, SpecTrain), each run
    on the same pipeline, initial weights and synthetic mini-batches; returns
    the loss of every mini-batch.

Inputs are synthetic (seeded normal draws with the workload's shapes); the
paper trains on CIFAR-10 / IMDb, so the curves are not the paper's numbers.

Command line:

    python -m paper_1809_02839_amd.experiments rmse [--layers 32 --hidden 2048 --steps 100]
    python -m paper_1809_02839_amd.experiments policies [--workload mlp3 --steps 60]
    python -m paper_1809_02839_amd.experiments policies --workload vgg_conv_pipe --steps 200
"""
import argparse
import dataclasses
import json
import sys
from typing import Callable, Dict, Optional, Sequence

import numpy as np




def _rmse(a: np.ndarray, b: np.ndarray) -> float:
    d = a.astype(np.float64) - b.astype(np.float64)
    return float(np.sqrt(np.mean(d * d)))


def snn_spec(layers: int = 32, hidden: int = 2048, batch: int = 128, inputs: int = 3072, classes: int = 10,
             lr: float = 1e-3, momentum: float = 0.9, dtype: str = "fp32"):
    """A stack of `layers` fully connected layers of `hidden` units with a
    softmax cross-entropy head, as one stage of a one-stage pipeline (the SNN
    shape of Section 4.1: 32 layers of 2048 units, learning rate 1e-3, momentum
    0.9, batch 128; ReLU stands in for the self-normalising activation)."""
    import synth
    return synth.StageSpec("fc", dtype, "ce", 0, 1, batch, layers, (inputs, classes, hidden), lr, momentum)


def prediction_rmse(spec, steps: int, s_values: Sequence[int] = (1, 2, 3), W0: Optional[np.ndarray] = None,
                    v0: Optional[np.ndarray] = None, inputs: Optional[Callable] = None, device: str = "cuda"):
    """Train `spec` (a one-stage pipeline, N = 1) for `steps` updates and return
    {s: {"t": [...], "predicted": [...], "stale": [...]}}: for every t >= s the
    RMSE of the prediction of W_t made s updates earlier, and of W_{t-s}."""
    import torch
    import synth
    from .pipeline import Pipeline

    if spec.num_stages != 1:
        raise ValueError("the prediction-accuracy experiment trains a one-stage pipeline (N = 1)")
    W0 = synth.initial_params(spec) if W0 is None else W0
    draw = inputs
    if draw is None:
        def draw(sp, m):
            x = synth.stage_input(sp, m)
            dy = synth.upstream_grad(sp, m) if sp.head == "none" else None
            lab = synth.labels(sp, m) if sp.head == "ce" else None
            return x, dy, lab
    smax = max(s_values)
    history: Dict[int, np.ndarray] = {}             # W_t for the last smax + 1 updates
    pending: Dict[tuple, np.ndarray] = {}           # (target t, s) -> prediction of W_t
    out = {s: {"t": [], "predicted": [], "stale": []} for s in s_values}

    def on_update(k, t, st):
        if t % 10 == 0:
            print(f"[rmse] update {t} of {steps}", file=sys.stderr, flush=True)
        W, _ = st.get_state()
        history[t] = W
        history.pop(t - smax - 1, None)
        for s in s_values:
            if (t, s) in pending:
                out[s]["t"].append(t)
                out[s]["predicted"].append(_rmse(pending.pop((t, s)), W))
                out[s]["stale"].append(_rmse(history[t - s], W))
        # Eq. 4 in the library: slot 0 holds W_t - s eta v_t; restore s = 0 for the next forward
        for s in s_values:
            if t + s <= steps:
                st.predict(s, 0)
                pending[(t + s, s)] = st.get_predicted(0)
        st.predict(0, 0)

    pipe = Pipeline([spec], [W0], device=device, v0s=None if v0 is None else [v0])
    history[0] = np.asarray(W0, np.float32).copy()
    if v0 is not None:
        st0 = pipe.stages[0]
        for s in s_values:
            st0.predict(s, 0)
            pending[(s, s)] = st0.get_predicted(0)
        st0.predict(0, 0)
    pipe.run(steps, draw, on_update=on_update)
    torch.cuda.synchronize()
    pipe.destroy()
    return out


def teacher_labels(workload, seed: int = 4242):
    """A learnable labelling of a workload's synthetic inputs: the class a fixed
    seeded random linear map of the first stage's input scores highest (the
    uniform random labels of the parity tests carry nothing to learn). For
    FC, conv and transformer pipelines (one label per token)."""
    import synth
    first, last = workload.stages[0], workload.stages[-1]
    classes = last.num_classes() if hasattr(last, "num_classes") else last.dims[1]
    rng = np.random.default_rng(seed)
    # conv models end in a global average pool, so their teacher reads the
    # input averaged over positions (a function the pooled head can express);
    # a transformer labels every token from that token's input embedding
    # (its targets come from the first 1024 tokens of the vocabulary; the head
    # still scores all of them). Labels are cached per mini-batch.
    pooled = first.kind in ("conv3x3", "bottleneck")
    per_token = last.kind == "transformer"
    if pooled or per_token:
        width = first.input_shape()[-1]
    else:
        width = int(np.prod(first.input_shape()[1:]))
    used = min(classes, 1024) if per_token else classes
    T = rng.standard_normal((width, used)).astype(np.float32)
    cache = {}

    def labels(sp, m):
        if m not in cache:
            x = synth.stage_input(first, m)
            if per_token:
                cache[m] = np.argmax(x.reshape(-1, width) @ T, axis=1).astype(np.int32).reshape(sp.label_shape())
            else:
                x = x.astype(np.float64)
                x = x.mean(axis=(1, 2)) if pooled else x.reshape(first.batch, -1)
                cache[m] = np.argmax(x @ T, axis=1).astype(np.int32)
        return cache[m]
    return labels


def policy_losses(workload, steps: int, policies: Sequence[str] = ("spectrain", "vanilla", "stash"),
                  device: str = "cuda", labels: Optional[Callable] = None):
    """{policy: [loss of mini-batch m for m < steps]} for a workload whose last
    stage has a cross-entropy head, every policy from the same W0 and inputs.
    labels(spec, m) overrides the synthetic labels."""
    import torch
    import synth
    from .pipeline import Pipeline

    if workload.stages[-1].head != "ce":
        raise ValueError("policy_losses needs a workload whose last stage has a loss head")
    losses = {}
    for policy in policies:
        specs = [dataclasses.replace(s, policy=policy) for s in workload.stages]
        pipe = Pipeline(specs, [synth.initial_params(s) for s in workload.stages], device=device)

        full = len(specs) == specs[0].num_stages

        def draw(sp, m):
            # in a whole pipeline only stage 0 reads its input (the others take
            # the previous stage's output)
            x = synth.stage_input(sp, m) if (not full or sp.stage_index == 0) else None
            if sp.head != "ce":
                return x, None, None
            return x, None, (labels or synth.labels)(sp, m)
        def progress(k, count, st):
            if k == 0 and count % 50 == 0:
                print(f"[policies] {policy}: {count} of {steps} updates at stage 0", file=sys.stderr, flush=True)
        out = pipe.run(steps, draw, on_update=progress)
        torch.cuda.synchronize()
        losses[policy] = [out["loss"][m].item() for m in range(steps)]
        print(f"[policies] {policy}: {steps} mini-batches", file=sys.stderr, flush=True)
        pipe.destroy()
    return losses


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("rmse", help="prediction accuracy of Eq. 4 (Fig. 7)")
    a.add_argument("--layers", type=int, default=32)
    a.add_argument("--hidden", type=int, default=2048)
    a.add_argument("--batch", type=int, default=128)
    a.add_argument("--steps", type=int, default=100)
    a.add_argument("--dtype", default="fp32", choices=["fp32", "bf16"])
    b = sub.add_parser("policies", help="losses under SpecTrain, Vanilla and weight stashing")
    b.add_argument("--workload", default="mlp3")
    b.add_argument("--steps", type=int, default=60)
    b.add_argument("--random-labels", action="store_true",
                   help="uniform random labels instead of the linear-teacher labels")
    b.add_argument("--lr", type=float, default=None, help="learning rate for every stage instead of the workload's")
    args = ap.parse_args(argv)
    if args.cmd == "rmse":
        spec = snn_spec(args.layers, args.hidden, args.batch, dtype=args.dtype)
        r = prediction_rmse(spec, args.steps)
        summary = {str(s): {"mean_predicted_rmse": float(np.mean(v["predicted"])),
                            "mean_stale_rmse": float(np.mean(v["stale"])),
                            "steps_predicted_better": int(np.sum(np.array(v["predicted"]) < np.array(v["stale"]))),
                            "steps": len(v["t"])} for s, v in r.items()}
        print(json.dumps({"experiment": "prediction_rmse", "layers": args.layers, "hidden": args.hidden,
                          "batch": args.batch, "steps": args.steps, "dtype": args.dtype, "by_s": summary,
                          "curves": {str(s): v for s, v in r.items()}}))
    else:
        import synth
        wl = synth.ALL_WORKLOADS[args.workload]
        if args.lr is not None:
            wl = synth.Workload(wl.name, tuple(dataclasses.replace(s, lr=args.lr) for s in wl.stages), wl.steps)
        losses = policy_losses(wl, args.steps, labels=None if args.random_labels else teacher_labels(wl))
        tail = max(1, args.steps // 4)
        print(json.dumps({"experiment": "policy_losses", "workload": args.workload, "steps": args.steps,
                          "lr": wl.stages[0].lr,
                          "labels": "random" if args.random_labels else "linear teacher",
                          "mean_loss_last_quarter": {p: float(np.mean(l[-tail:])) for p, l in losses.items()},
                          "losses": losses}))
    return 0


if __name__ == "__main__":
    sys.exit(main())
