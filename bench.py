"""Benchmark of one SpecTrain pipeline stage's steady-state step on one MI355X.

A step is one pass of the whole stage path over one mini-batch: the backward
of the oldest mini-batch in flight (data and weight gradients against the
backward-predicted weights), the fused momentum update that re-predicts both
weight slots (Eq. 1, Eq. 4), and the forward of the next mini-batch (against
the forward-predicted weights, Eq. 5 difference). The stage keeps N - k
mini-batches in flight, as in the one-forward-one-backward schedule.

Default workload: the ResNet-152-style bottleneck stage (8 bottleneck blocks
1x1 1024->256, 3x3 256->256, 1x1 256->1024 with identity skips, 14x14 maps,
batch 64, bf16 operands with float32 master weights, stage 3 of 4), the
stage with the most contraction work per step. Inputs are synthetic (seeded
normal draws, already resident in HBM when the timed region starts; a ring
of eight mini-batches whose second half repeats the first with negated
upstream gradients, so the weights stay bounded over hundreds of steps).

Output: one JSON line on stdout. `value` is samples per second. A separate
pass times every launch with HIP events on the stage's stream; each kernel
family (one kernel instantiation) is set against the roof that bounds it,
MFMA when its algorithmic flops at the MFMA peak take longer than its
algorithmic bytes at the HBM peak, HBM otherwise. `roofline` describes the
family with the largest share of the step time; `kernels` lists the largest
families. `step_roofline_frac` is the step's lower bound (the sum over
families of max(flops / MFMA peak, bytes / HBM peak)) over the measured step.
`predict_update_GBps` counts the fused update's 24 algorithmic bytes per
parameter (28 for float32 stages); `predict_update_GBps_cold` is the same in
a pass that evicts every cache before each update. `cpu_baseline` times the
CPU oracle on a bounded sample of the same workload.
"""
import argparse
import dataclasses
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0    # dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3     # dense fp32 MFMA
PEAK_HBM_GBPS = 8000.0
METRIC = "stage samples/sec (fwd+bwd+predict+update); MFMA util %; predict/update GB/s"

DESCRIPTIONS = {
    "mlp3": "3-stage pipeline of one fully connected layer per stage (784->256->256->10), batch 32, float32, "
            "softmax-CE head on the last stage",
    "vgg_conv": "VGG-16-style conv stage: 4x conv3x3 256->512->512->512->512, 8x8 maps, NHWC, ReLU",
    "resnet_bottleneck": "ResNet-152-style stage: 8 bottlenecks 1024->256->256->1024, 14x14 maps, identity skip",
    "transformer_enc": "Transformer encoder stage: 3 post-LN layers, d=512, 8 heads, FFN 2048, seq 128",
    "reslstm": "Residual LSTM stage: 2 layers, input=hidden=1024, T=35, vocab-10000 softmax-CE head",
    "vgg_conv_pipe": "4-stage pipeline of VGG-16-style conv stages (16 conv3x3 layers, 8x8 maps, 512 channels)",
    "resnet_bottleneck_pipe": "4-stage pipeline of ResNet-152-style stages (32 bottlenecks, 14x14 maps)",
    "transformer_enc_pipe": "4-stage pipeline of transformer encoder stages (12 layers) with a 32000-token "
                            "softmax-CE head on the last stage",
    "reslstm_pipe": "4-stage pipeline of residual LSTM stages (8 layers, hidden 1024, T=35) with a "
                    "10000-token softmax-CE head on the last stage",
    "transformer_enc_last": "Last transformer encoder stage: 3 post-LN layers, d=512, seq 128, with the "
                            "32000-token vocabulary projection and softmax-CE head",
}


# Kernel (rocprofv3 short name prefix) behind each pass family that is not
# named by its kernel (GEMM families are the kernel instantiations).
FAMILY_KERNEL = {
    "fused_update": "fused_update",   # fused_update_kernel, or fused_update_partials_kernel where K-slice
    "attention": "attention_fwd_kernel",   # partials of filter gradients are summed in the update
    "attention_bwd": "attention_bwd_kernel",
    "lstm_step": "lstm_step_fwd_kernel",
    "lstm_step_bwd": "lstm_step_bwd_kernel",
    "layernorm_bwd": "layernorm_bwd",
    "softmax_ce": "softmax_ce",
}


def kernel_prefix(family):
    return family if "<" in family else FAMILY_KERNEL.get(family)


def traffic_per_launch(workload, family):
    """HBM bytes per launch of the family's kernel from the committed counter
    summary of this workload, or None when there is none or the kernel
    sources changed since the counters were taken."""
    from paper_1809_02839_amd import profiling
    digest, table = profiling.read_traffic(os.path.join(ROOT, "profiles", f"stage_kernels_{workload}_hbm_traffic.md"),
                                           with_dispatches=True)
    prefix = kernel_prefix(family)
    if digest is None or prefix is None or digest != profiling.source_digest():
        return None
    hits = [v for k, v in table.items() if k.startswith(prefix)]
    n = sum(d for d, _ in hits)
    return round(sum(d * b for d, b in hits) / n) if n else None


def family_roof(v, peak_mfma):
    """(bound, achieved, peak, unit, roof_ms) of a family's summed launches."""
    t_mfma = v["flops_total"] / (peak_mfma * 1e12) * 1e3
    t_hbm = v["bytes_total"] / (PEAK_HBM_GBPS * 1e9) * 1e3
    if v["flops_total"] > 0 and t_mfma >= t_hbm:
        return "mfma", v["flops_total"] / (v["ms_total"] / 1e3) / 1e12, peak_mfma, "TFLOP/s", t_mfma
    return "hbm", v["bytes_total"] / (v["ms_total"] / 1e3) / 1e9, PEAK_HBM_GBPS, "GB/s", t_hbm


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class StageLoop:
    """Steady-state driver of one stage through the C ABI with a device ring of inputs."""

    def __init__(self, spec, torch, native, stream, ring=8, concurrent=True):
        import numpy as np
        import synth
        self.torch, self.spec, self.stream = torch, spec, stream
        dev = torch.device("cuda")
        dt = torch.bfloat16 if spec.dtype == "bf16" else torch.float32
        self.st = native.Stage(native.desc_from_spec(spec), synth.initial_params(spec), stream)
        k, N = spec.stage_index, spec.num_stages
        self.sf, self.sb = native.policy_versions(spec.policy, k, N)
        self.depth = N - k
        # Each step is a forward, a backward and the update (the stage's
        # one-forward-one-backward order). With two or more mini-batches in
        # flight the forward of mini-batch m + depth - 1 and the backward of
        # m, which read weights of the same version, go through the combined
        # call that runs them concurrently; at the last stage (depth 1) the
        # forward is the one its backward needs, so the calls stay separate.
        self.concurrent = concurrent and self.depth >= 2
        self.ring = ring
        with torch.cuda.stream(stream):
            self.st.predict(self.sf, 0)
            self.st.predict(self.sb, 1)
            # Antithetic ring: entries h and h + ring/2 share x, and their upstream
            # gradients have opposite signs, so hundreds of steps over the ring
            # do not drive the weights of the (unbounded) synthetic objective
            # systematically in one direction.
            half = ring // 2
            self.x = [torch.from_numpy(synth.stage_input(spec, m % half)).to(dev).to(dt) for m in range(ring)]
            if spec.head == "ce":
                self.lab = [torch.from_numpy(synth.labels(spec, m % half)).to(dev) for m in range(ring)]
                self.loss = [torch.zeros(1, device=dev) for _ in range(ring)]
                self.dy = None
                self.y = None
            else:
                self.dy = [torch.from_numpy(synth.upstream_grad(spec, m % half) * (1 if m < half else -1)).to(dev).to(dt)
                           for m in range(ring)]
                self.y = [torch.empty(spec.output_shape(), device=dev, dtype=dt) for _ in range(self.depth + 1)]
            self.dx = torch.empty(spec.input_shape(), device=dev, dtype=dt)
        self.next_b = 0
        for m in range(self.depth - 1 if self.concurrent else self.depth):
            self._forward(m)
        stream.synchronize()
        _ = np

    def _forward(self, m):
        r = m % self.ring
        if self.spec.head == "ce":
            self.st.forward(m, self.x[r], None, self.lab[r], self.loss[r])
        else:
            self.st.forward(m, self.x[r], self.y[m % (self.depth + 1)])

    def graph_period(self):
        """Steps after which every pointer the steps use repeats: the input
        ring, the output ring and the stash slots (the stage reuses the slot
        the backward just freed, so slots repeat every N - k steps)."""
        import math
        return math.lcm(self.ring, self.depth + 1, self.depth)

    def steps(self, n, before_update=None):
        for _ in range(n):
            m = self.next_b
            dy = None if self.dy is None else self.dy[m % self.ring]
            if self.concurrent:
                f = m + self.depth - 1
                r = f % self.ring
                if self.spec.head == "ce":
                    self.st.forward_backward(f, self.x[r], None, m, dy, self.dx, labels=self.lab[r], loss=self.loss[r])
                else:
                    self.st.forward_backward(f, self.x[r], self.y[f % (self.depth + 1)], m, dy, self.dx)
            else:
                self.st.backward(m, dy, self.dx)
            if before_update is not None:
                before_update()
            self.st.update(self.sf, self.sb)
            if not self.concurrent:
                self._forward(m + self.depth)
            self.next_b += 1


class PipeLoop:
    """All N stages of a pipeline workload on one GPU, driven in the
    one-forward-one-backward task order (every stage's forward, backward and
    update of each mini-batch). Stage 0 inputs, last-stage labels or upstream
    gradients, and every stage output and input gradient live in device rings
    sized to the mini-batches a stage can hold in flight."""

    def __init__(self, specs, torch, native, stream, ring=8):
        import synth
        self.torch, self.specs, self.stream = torch, list(specs), stream
        dev = torch.device("cuda")
        dt = torch.bfloat16 if self.specs[0].dtype == "bf16" else torch.float32
        self.N = len(self.specs)
        self.ring = ring
        self.st, self.sf, self.sb = [], [], []
        for spec in self.specs:
            st = native.Stage(native.desc_from_spec(spec), synth.initial_params(spec), stream)
            sf, sb = native.policy_versions(spec.policy, spec.stage_index, spec.num_stages)
            self.st.append(st)
            self.sf.append(sf)
            self.sb.append(sb)
        first, last = self.specs[0], self.specs[-1]
        half = ring // 2
        depth = self.N + 1    # outputs and input gradients kept per stage (more than any stage holds in flight)
        self.depth = depth
        with torch.cuda.stream(stream):
            for k, st in enumerate(self.st):
                st.predict(self.sf[k], 0)
                st.predict(self.sb[k], 1)
            self.x = [torch.from_numpy(synth.stage_input(first, m % half)).to(dev).to(dt) for m in range(ring)]
            if last.head == "ce":
                self.lab = [torch.from_numpy(synth.labels(last, m % half)).to(dev) for m in range(ring)]
                self.loss = [torch.zeros(1, device=dev) for _ in range(ring)]
                self.dy = None
            else:
                self.dy = [torch.from_numpy(synth.upstream_grad(last, m % half) * (1 if m < half else -1)).to(dev)
                           .to(dt) for m in range(ring)]
            self.y = [[torch.empty(sp.output_shape(), device=dev, dtype=dt) for _ in range(depth)]
                      if k < self.N - 1 or sp.head != "ce" else None for k, sp in enumerate(self.specs)]
            self.dx = [[torch.empty(sp.input_shape(), device=dev, dtype=dt) for _ in range(depth)] if k > 0 else None
                       for k, sp in enumerate(self.specs)]
            self.dx0 = torch.empty(first.input_shape(), device=dev, dtype=dt)
        self.m0 = 0
        stream.synchronize()

    def graph_period(self):
        """Any call starts and ends with every stash empty; the input rings
        repeat every `ring` mini-batches."""
        return self.ring

    def steps(self, n, before_update=None):
        """n mini-batches through the whole pipeline (fill and drain included)."""
        from paper_1809_02839_amd.pipeline import pipeline_task_order
        N, d = self.N, self.depth
        for k, kind, i in pipeline_task_order(N, n):
            m = self.m0 + i
            st = self.st[k]
            if kind == "F":
                x = self.x[m % self.ring] if k == 0 else self.y[k - 1][m % d]
                if self.y[k] is None:
                    st.forward(m, x, None, self.lab[m % self.ring], self.loss[m % self.ring])
                else:
                    st.forward(m, x, self.y[k][m % d])
            else:
                if k < N - 1:
                    dy = self.dx[k + 1][m % d]
                else:
                    dy = None if self.dy is None else self.dy[m % self.ring]
                dx = self.dx[k][m % d] if k > 0 else self.dx0
                st.backward(m, dy, dx)
                if before_update is not None:
                    before_update()
                st.update(self.sf[k], self.sb[k])
        self.m0 += n

    def profile(self, on):
        for st in self.st:
            st.profile(on)

    def profile_read(self):
        total = {}
        for st in self.st:
            for k, v in st.profile_read().items():
                t = total.setdefault(k, {"launches": 0, "ms_total": 0.0, "flops_total": 0.0, "bytes_total": 0.0,
                                     "extra_bytes_total": 0.0})
                for f in t:
                    t[f] += v[f]
        return total

    def destroy(self):
        for st in self.st:
            st.destroy()


def host_info():
    """CPU model and the BLAS library (and its threads) NumPy runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        import numpy  # noqa: F401  (loads the BLAS library threadpoolctl reports)
        from threadpoolctl import threadpool_info
        libs = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        if libs:
            blas = f"{libs[0].get('internal_api')} {libs[0].get('version')} ({libs[0].get('num_threads')} threads)"
    except Exception:
        pass
    return {"cpu_model": model, "blas": blas}


def cpu_baseline_pipeline(specs, n_steps):
    """The oracle as it stands on the host: n_steps mini-batches through all
    stages of the pipeline workload (each stage's forward, backward, update)."""
    import numpy as np
    import synth
    from oracle import trajectory
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count()
    wl = synth.Workload("sample", tuple(specs), n_steps)
    t0 = time.perf_counter()
    trajectory.run(wl)
    dt = time.perf_counter() - t0
    per_step = dt / n_steps
    extra = {}
    if specs[0].dtype == "fp32":
        # the small float32 pipeline also on one thread (BLAS threading barely helps at its sizes)
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1):
            t0 = time.perf_counter()
            trajectory.run(wl)
            extra["value_1thread"] = specs[0].batch / ((time.perf_counter() - t0) / n_steps)
    _ = np
    return {"value": specs[0].batch / per_step, "unit": "samples/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{n_steps} full-size mini-batches through all {len(specs)} stages (forward, backward, "
                      f"update each), float64 NumPy, {per_step:.2f} s per mini-batch", **extra, **host_info()}


def cpu_baseline(spec, n_steps, layers=0):
    """The oracle as it stands, timed on the host: n_steps (forward, backward,
    update) of the same stage at full size, median step time. With layers > 0
    the timed stage holds that many of the workload's (identical) layers and
    its step time is scaled by num_layers / layers."""
    import numpy as np
    import synth
    from oracle import method, stages
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count()
    full_layers = spec.num_layers
    if layers and layers < full_layers:
        spec = dataclasses.replace(spec, num_layers=layers)
    scale = full_layers / spec.num_layers
    k, N = spec.stage_index, spec.num_stages
    lr, gamma = float(np.float32(spec.lr)), float(np.float32(spec.momentum))
    W = synth.initial_params(spec).astype(np.float64)
    v = np.zeros_like(W)
    rnd = stages.weight_rounder(spec)
    sf, sb = method.staleness_versions(spec.policy, k, N)
    per = []
    for m in range(n_steps):
        t0 = time.perf_counter()
        x = synth.stage_input(spec, m)
        dy = synth.upstream_grad(spec, m) if spec.head == "none" else None
        lab = synth.labels(spec, m) if spec.head == "ce" else None
        _, _, st = stages.forward(spec, stages.unpack(spec, rnd(method.predict(W, v, sf, lr))), x, lab)
        _, g = stages.backward(spec, stages.unpack(spec, rnd(method.predict(W, v, sb, lr))), st, dy)
        W, v = method.momentum_sgd_step(W, v, stages.pack(spec, g), lr, gamma)
        per.append((time.perf_counter() - t0) * scale)
    per_step = float(np.median(per))
    what = (f"{n_steps} full-size steps (forward, backward, update) of the same stage"
            if scale == 1 else
            f"{n_steps} full-size steps (forward, backward, update) of a stage of {spec.num_layers} of its "
            f"{full_layers} identical layers, step time scaled by {scale:g}")
    return {"value": spec.batch / per_step, "unit": "samples/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{what}; float64 NumPy, median {per_step:.2f} s per stage step", **host_info()}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="resnet_bottleneck", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--profile-steps", type=int, default=50)
    ap.add_argument("--cpu-steps", type=int, default=3,
                    help="oracle steps timed for cpu_baseline (the median step is reported)")
    ap.add_argument("--cpu-layers", type=int, default=0,
                    help="time the oracle on a stage of this many of the workload's layers (identical "
                         "blocks) and scale its step time to the whole stage (0: the whole stage; "
                         "default 1 for the bottleneck stage, whose whole step takes the oracle ~30 s)")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--policy", default="spectrain", choices=["spectrain", "vanilla", "stash"],
                    help="weight staleness treatment (Section 4.2): SpecTrain prediction (default), Vanilla "
                         "pipelining (latest weights) or weight stashing (backward reuses the forward's weights)")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of a HIP graph that captures a period of steps (the period after which "
                         "every buffer the steps use repeats); --steps is rounded up to a whole number of periods")
    ap.add_argument("--median-steps", type=int, default=50,
                    help="steps of a pass with an event between steps, for the median step time of a single-stage "
                         "workload (0: skip)")
    ap.add_argument("--cold-steps", type=int, default=10,
                    help="steps of a second per-launch pass in which a 1 GiB read evicts the caches (MALL "
                         "included) before every update, for the update's cold-cache bandwidth (0: skip)")
    ap.add_argument("--serial", action="store_true",
                    help="issue each step's forward and backward as separate calls (by default a single stage "
                         "with two or more mini-batches in flight runs them concurrently through "
                         "spectrain_stage_forward_backward)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first run one device-to-device copy of this many MiB (a known-size reference "
                         "dispatch for scaling hardware byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs one pipeline stage on one GPU; --gpus above 1 is not supported "
              "(the multi-GPU pipeline is simulated in order on one device)", file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_1809_02839_amd import native

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    wl = synth.ALL_WORKLOADS[args.workload]
    specs = [dataclasses.replace(sp, policy=args.policy) for sp in wl.stages]
    spec = specs[0]
    pipeline = len(specs) > 1
    if args.copy_calibration_mib > 0:
        n = args.copy_calibration_mib << 18   # float32 elements
        src = torch.ones(n, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)   # one elementwise kernel: n*4 bytes read, n*4 written
        torch.cuda.synchronize()
        log(f"[bench] calibration kernel (neg): {n * 4} bytes read, {n * 4} bytes written")
        del src, dst
    stream = torch.cuda.Stream()
    loop = (PipeLoop(specs, torch, native, stream) if pipeline
            else StageLoop(spec, torch, native, stream, concurrent=not args.serial))

    loop.steps(args.warmup)
    torch.cuda.synchronize()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if args.graph:
        period = loop.graph_period()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=stream):
            loop.steps(period)
        reps = -(-args.steps // period)
        args.steps = reps * period
        with torch.cuda.stream(stream):
            graph.replay()   # the captured steps themselves, untimed
        torch.cuda.synchronize()
        start.record(stream)
        with torch.cuda.stream(stream):
            for _ in range(reps):
                graph.replay()
        stop.record(stream)
        torch.cuda.synchronize()
        log(f"[bench] HIP graph of {period} steps, {reps} replays")
    else:
        torch.cuda.synchronize()
        start.record(stream)
        loop.steps(args.steps)
        stop.record(stream)
        torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps
    value = spec.batch / (ms_step / 1e3)
    log(f"[bench] {args.workload}: {ms_step:.3f} ms/step, {value:.0f} samples/s")

    # per-step durations (an event between steps, outside the timed region);
    # single stages only: a pipeline call runs its own fill and drain
    ms_median = None
    if args.median_steps > 0 and not pipeline:
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.median_steps + 1)]
        ev[0].record(stream)
        for i in range(args.median_steps):
            loop.steps(1)
            ev[i + 1].record(stream)
        torch.cuda.synchronize()
        per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(args.median_steps))
        ms_median = per[len(per) // 2]
        log(f"[bench] per-step median {ms_median:.3f} ms, min {per[0]:.3f}, max {per[-1]:.3f} "
            f"over {args.median_steps} steps")

    # per-kernel pass (events around every launch, separate from the timed
    # region). A single stage issues every launch on its stage stream, one at
    # a time, with the kernels and launch shapes of the timed steps: each
    # event-to-event duration is then the launch's own (under concurrency it
    # would include the time the launch shares the GPU with the other streams,
    # and a profiler's kernel trace, which also reduces that sharing, would
    # not see the same durations).
    if pipeline:
        loop.profile(True)
        loop.steps(args.profile_steps)
        prof = loop.profile_read()
        loop.profile(False)
    else:
        loop.st.profile(True, serial=True)
        loop.steps(args.profile_steps)
        prof = loop.st.profile_read()
        loop.st.profile(False)
    torch.cuda.synchronize()
    upd_cold_gbps = None
    if args.cold_steps > 0:
        # the same per-launch pass with the caches evicted before every update:
        # W, v and g then come from HBM, as they would after a long backward.
        # The eviction reads (a sum over 1 GiB, four times the MALL), so it
        # leaves no dirty lines whose write-back would land in the update.
        evict = torch.zeros(1 << 28, device="cuda")
        sink = []

        def flush():
            with torch.cuda.stream(stream):
                sink.append(evict.sum())
        if pipeline:
            loop.profile(True)
        else:
            loop.st.profile(True, serial=True)
        loop.steps(args.cold_steps, before_update=flush)
        cold = loop.profile_read() if pipeline else loop.st.profile_read()
        if pipeline:
            loop.profile(False)
        else:
            loop.st.profile(False)
        torch.cuda.synchronize()
        del evict, sink
        u = cold.get("fused_update")
        if u and u["ms_total"] > 0:
            upd_cold_gbps = u["bytes_total"] / (u["ms_total"] / 1e3) / 1e9
            log(f"[bench]   fused_update cold     {u['ms_total'] / u['launches'] * 1e3:9.1f} us/launch  "
                f"{upd_cold_gbps:.0f} GB/s (caches evicted before each update)")
    fam_ms = {k: v["ms_total"] / args.profile_steps for k, v in prof.items()}
    peak_mfma = PEAK_BF16_TFLOPS if spec.dtype == "bf16" else PEAK_FP32_TFLOPS
    roofs = {k: family_roof(v, peak_mfma) for k, v in prof.items()}
    for k, v in sorted(prof.items(), key=lambda kv: -kv[1]["ms_total"]):
        bound, ach, peak, unit, _ = roofs[k]
        log(f"[bench]   {k:40s} {v['launches'] / args.profile_steps:5.1f}/step "
            f"{v['ms_total'] / v['launches'] * 1e3:8.1f} us/launch {fam_ms[k] * 1e3:8.1f} us/step  "
            f"{bound} {ach:8.1f} {unit} ({ach / peak:.3f})")
    dom = max(prof, key=lambda k: prof[k]["ms_total"])
    d = prof[dom]
    bound, ach, peak, unit, _ = roofs[dom]
    roof = {"bound": bound, "achieved": round(ach, 2), "peak": peak, "unit": unit, "frac": round(ach / peak, 4),
            "traffic": traffic_per_launch(args.workload, dom), "kernel": dom,
            "launches_per_step": d["launches"] / args.profile_steps,
            "us_per_launch": round(d["ms_total"] / d["launches"] * 1e3, 2),
            "algorithmic_bytes_per_launch": round(d["bytes_total"] / d["launches"]),
            "algorithmic_flops_per_launch": round(d["flops_total"] / d["launches"])}
    kernels = []
    for k in sorted(prof, key=lambda k: -prof[k]["ms_total"])[:12]:
        v = prof[k]
        b, a, pk, u, _ = roofs[k]
        kernels.append({"kernel": k, "launches_per_step": v["launches"] / args.profile_steps,
                        "us_per_launch": round(v["ms_total"] / v["launches"] * 1e3, 2), "bound": b,
                        "achieved": round(a, 1), "unit": u, "frac": round(a / pk, 4)})
    gemm_flops = sum(v["flops_total"] for v in prof.values())
    gemm_ms = sum(v["ms_total"] for k, v in prof.items() if v["flops_total"] > 0)
    upd = prof.get("fused_update")
    upd_gbps = upd["bytes_total"] / (upd["ms_total"] / 1e3) / 1e9 if upd else None
    upd_extra = upd["extra_bytes_total"] / upd["launches"] if upd else None
    # Lower bound of the step: every family at its roof (flops at the MFMA
    # peak or algorithmic bytes at the HBM peak, whichever takes longer)
    bound_us = sum(r[4] for r in roofs.values()) / args.profile_steps * 1e3

    cpu = None
    if not args.no_cpu:
        log(f"[bench] timing the CPU oracle on {args.cpu_steps} steps ...")
        # whole pipelines: a quarter of the steps (each is N stage steps); the
        # small float32 pipeline: its full 20 mini-batches (well under a second)
        n_pipe = wl.steps if spec.dtype == "fp32" else max(1, args.cpu_steps // 4)
        layers = args.cpu_layers or (1 if args.workload == "resnet_bottleneck" else 0)
        cpu = cpu_baseline_pipeline(specs, n_pipe) if pipeline else cpu_baseline(spec, args.cpu_steps, layers)
        log(f"[bench] oracle: {cpu['value']:.2f} samples/s on {cpu['cores']} threads")

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_median": round(ms_median, 4) if ms_median else None,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": spec.dtype,
        "data": "synthetic",
        "hip_graph": bool(args.graph),
        "concurrent_forward_backward": bool(getattr(loop, "concurrent", False)),
        "config": {"workload": f"{args.workload}: {DESCRIPTIONS[args.workload]}", "policy": args.policy,
                   "batch": spec.batch,
                   "stage_index": None if pipeline else spec.stage_index, "num_stages": spec.num_stages,
                   "s_forward": loop.sf, "s_backward": loop.sb,
                   "params": sum(synth.num_params(sp) for sp in specs)},
        "mfma_util_pct": round(100.0 * gemm_flops / (gemm_ms / 1e3) / 1e12 / peak_mfma, 2) if gemm_ms else None,
        "mfma_util_pct_of_step": round(100.0 * gemm_flops / args.profile_steps / (ms_step / 1e3) / 1e12 / peak_mfma, 2),
        "predict_update_GBps": round(upd_gbps, 1) if upd_gbps else None,
        "predict_update_frac_hbm": round(upd_gbps / PEAK_HBM_GBPS, 4) if upd_gbps else None,
        "predict_update_GBps_cold": round(upd_cold_gbps, 1) if upd_cold_gbps else None,
        "predict_update_us": round(upd["ms_total"] / upd["launches"] * 1e3, 2) if upd else None,
        "predict_update_extra_bytes_per_launch": round(upd_extra) if upd else None,
        "step_bound_us": round(bound_us, 2),
        "step_roofline_frac": round(bound_us / (ms_step * 1e3), 4),
        "roofline": roof,
        "kernels": kernels,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    if pipeline:
        loop.destroy()
    else:
        loop.st.destroy()


if __name__ == "__main__":
    main()
