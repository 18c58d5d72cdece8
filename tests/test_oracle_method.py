"""Pins of the oracle's method core: version differences, pipeline order,
prediction and momentum update (Section 3.1, 3.2, Eq. 1-6)."""
import dataclasses

import numpy as np
import pytest
import torch

import synth
from oracle import method, schedule, stages, trajectory


# ------------------------------------------------ version differences ----

def test_worked_example_section_3_2():
    # Section 3.2 example: N=3 GPUs, first stage (k=0), forward pass: s=2, so the
    # 4th mini-batch predicts W_6 from W_4 (and v_3).
    assert method.version_difference(0, 3, forward=True) == 2
    W4 = np.array([1.0, -2.0, 0.5])
    v3 = np.array([0.25, 0.5, -1.0])
    eta = 0.125
    assert np.array_equal(method.predict(W4, v3, 2, eta), W4 - (6 - 4) * eta * v3)


@pytest.mark.parametrize("N", range(1, 9))
def test_update_count_between_forward_and_backward(N):
    """Brute force over the simulated pipeline: the number of weight updates
    stage k performs between F_k(m) and B_k(m) equals s_f - s_b, and the last
    stage's forward and backward see the same weight version."""
    M = 3 * N + 4
    for k in range(N):
        tasks = schedule.stage_tasks(k, N, M)
        pos = {t: i for i, t in enumerate(tasks)}
        sf = method.version_difference(k, N, True)
        sb = method.version_difference(k, N, False)
        for m in range(M):
            between = sum(1 for kind, _ in tasks[pos[("F", m)] + 1:pos[("B", m)]] if kind == "B")
            # in steady state the count is the pipeline depth below stage k
            if m >= N:
                assert between == sf - sb == N - 1 - k
        if k == N - 1:
            assert sf == sb


@pytest.mark.parametrize("N", range(1, 9))
def test_version_difference_counts_updates_until_round_trip_completes(N):
    """Section 3.2 defines s as the number of time units between the current
    pass at stage k and the moment the mini-batch completes its round trip
    (its backward at stage 0). Counted on the oracle's half-unit grid: the
    updates stage k makes, from other mini-batches' backwards, after the pass
    and no later than B_0(m) must equal Eq. 5 for F_k(m) and Eq. 6 for B_k(m).
    The count is taken by enumeration of the task times, not by the formula,
    so a ceil(k/2) or an off-by-one in either equation fails at some (k, N)."""
    M = 4 * N + 6
    for k in range(N):
        upd_times = {m2: schedule.backward_time(k, N, m2) for m2 in range(M)}
        for m in range(N, M - N):
            done = schedule.backward_time(0, N, m)          # round trip completes
            for forward in (True, False):
                t = schedule.forward_time(k, N, m) if forward else schedule.backward_time(k, N, m)
                count = sum(1 for m2, tb in upd_times.items() if m2 != m and t < tb <= done)
                assert count == method.version_difference(k, N, forward), (N, k, m, forward, count)


@pytest.mark.parametrize("N", range(1, 9))
def test_pipeline_dependencies(N):
    """Every forward at stage k>0 runs after the same mini-batch's forward at
    k-1, every backward after the loss (last forward) and after the backward at
    k+1; each stage holds at most N-k mini-batches in flight."""
    M = 2 * N + 3
    order = schedule.pipeline_tasks(N, M)
    pos = {t: i for i, t in enumerate(order)}
    for m in range(M):
        for k in range(N):
            if k > 0:
                assert pos[(k - 1, "F", m)] < pos[(k, "F", m)]
            if k < N - 1:
                assert pos[(k + 1, "B", m)] < pos[(k, "B", m)]
            assert pos[(N - 1, "F", m)] <= pos[(k, "B", m)] or k == N - 1
    for k in range(N):
        live = 0
        for kind, _ in schedule.stage_tasks(k, N, M):
            live += 1 if kind == "F" else -1
            assert 0 <= live <= N - k


def test_single_gpu_is_staleness_free():
    # N=1: F(m), B(m) alternate and both use the current weights (s=0).
    assert schedule.stage_tasks(0, 1, 3) == [("F", 0), ("B", 0), ("F", 1), ("B", 1), ("F", 2), ("B", 2)]
    assert method.version_difference(0, 1, True) == 0 == method.version_difference(0, 1, False)


def test_version_difference_rejects_bad_stage():
    with pytest.raises(ValueError):
        method.version_difference(3, 3, True)
    with pytest.raises(ValueError):
        method.version_difference(-1, 3, False)


# ------------------------------------------------------- update rule ----

def test_momentum_update_matches_torch_sgd_with_zero_buffer():
    """Eq. 1 plus W <- W - eta v is torch's SGD with dampening = momentum and
    a momentum buffer that starts at zero."""
    rng = np.random.default_rng(0)
    n, eta, gamma = 257, 0.03125, 0.875
    W = rng.standard_normal(n).astype(np.float32).astype(np.float64)
    v = np.zeros(n)
    p = torch.tensor(W.copy(), dtype=torch.float64, requires_grad=True)
    opt = torch.optim.SGD([p], lr=eta, momentum=gamma, dampening=gamma)
    opt.state[p]["momentum_buffer"] = torch.zeros(n, dtype=torch.float64)
    for _ in range(6):
        g = rng.standard_normal(n).astype(np.float32).astype(np.float64)
        W, v = method.momentum_sgd_step(W, v, g, eta, gamma)
        p.grad = torch.tensor(g)
        opt.step()
        np.testing.assert_allclose(W, p.detach().numpy(), rtol=1e-6, atol=1e-7)
        np.testing.assert_allclose(v, opt.state[p]["momentum_buffer"].numpy(), rtol=1e-6, atol=1e-7)


def test_gamma_one_freezes_weights():
    # 0 < gamma <= 1 (Eq. 1); at gamma = 1 the smoothed gradient never leaves 0.
    w = synth.SMALL_WORKLOADS["mlp3_small"]
    w1 = dataclasses.replace(w, stages=tuple(dataclasses.replace(s, momentum=1.0) for s in w.stages), steps=6)
    r = trajectory.run(w1)
    for spec, W, v in zip(w1.stages, r["W"], r["v"]):
        assert np.array_equal(W, synth.initial_params(spec).astype(np.float64))
        assert not np.any(v)


def _fc_closed_form_setup(k, N, batch=6, fin=5, fout=4):
    """FC stage with a large positive bias (ReLU never clips) and dyadic data, so
    the gradient is the same exact dyadic value at every step."""
    spec = synth.StageSpec("fc", "fp32", "none", k, N, batch, 1, (fin, fout, fout), 2.0 ** -7, 0.875)
    rng = np.random.default_rng(7)
    X = rng.integers(-1, 2, size=(batch, fin)) * 2.0 ** -3
    dY = rng.integers(-1, 2, size=(batch, fout)) * 2.0 ** -5
    W0 = np.concatenate([rng.integers(-64, 65, size=fout * fin) * 2.0 ** -12, np.full(fout, 4.0)])
    g = np.concatenate([(dY.T @ X).reshape(-1), dY.sum(axis=0)])
    return spec, X, dY, W0, g


@pytest.mark.parametrize("k,N", [(0, 3), (1, 3), (2, 3), (0, 4), (1, 4), (2, 4), (3, 4)])
def test_closed_form_constant_gradient(k, N):
    """With g constant and v0 = g, v stays g, W_t = W0 - t eta g exactly, and the
    weights a pass predicts with difference s are exactly W_{t+s}: every
    forward output must equal the one computed from the closed form."""
    spec, X, dY, W0, g = _fc_closed_form_setup(k, N)
    wl = synth.Workload("closed_form", (spec,), steps=12)
    eta = spec.lr
    states = []
    r = trajectory.run(wl, W0=[W0], v0=[g], inputs=lambda s, m: (X, dY, None), keep_io=True,
                       on_update=lambda kk, u, W, v: states.append((u, W.copy(), v.copy())))
    for u, W, v in states:
        assert np.array_equal(v, g)
        assert np.array_equal(W, W0 - u * eta * g)
    sf = method.version_difference(k, N, True)
    sb = method.version_difference(k, N, False)
    tasks = schedule.stage_tasks(k, N, wl.steps)
    done = 0
    for kind, m in tasks:
        if kind == "B":
            # the backward's dX uses the weights predicted with Eq. 6's difference
            Wt = stages.unpack(spec, W0 - (done + sb) * eta * g)
            assert np.array_equal(r["dx"][(k, m)], dY @ Wt["fc0.weight"])
            done += 1
            continue
        Wt = W0 - (done + sf) * eta * g
        P = stages.unpack(spec, Wt)
        y = np.maximum(X @ P["fc0.weight"].T + P["fc0.bias"], 0)
        assert np.array_equal(r["y"][(k, m)], y)


def test_s0_pipeline_equals_sequential_momentum_sgd_torch():
    """N=1 (s=0 for both passes): the oracle's trajectory is plain sequential
    momentum SGD; compared with torch autograd + SGD(dampening=momentum) on CPU."""
    base = synth.SMALL_WORKLOADS["mlp3_small"]
    spec = synth.StageSpec("fc", "fp32", "ce", 0, 1, 7, 3, (37, 10, 50), 0.05, 0.9)
    wl = synth.Workload("seq", (spec,), steps=8)
    W0 = synth.initial_params(spec)
    r = trajectory.run(wl, exact=True, W0=[W0], keep_io=True)

    P = stages.unpack(spec, W0)
    params = [torch.tensor(P[n].copy(), requires_grad=True) for n, _, _ in synth.param_layout(spec)]
    opt = torch.optim.SGD(params, lr=float(np.float32(spec.lr)), momentum=float(np.float32(0.9)),
                          dampening=float(np.float32(0.9)))
    for p in params:
        opt.state[p]["momentum_buffer"] = torch.zeros_like(p)
    for m in range(wl.steps):
        x = torch.tensor(synth.stage_input(spec, m), dtype=torch.float64)
        lab = torch.tensor(synth.labels(spec, m), dtype=torch.long)
        h = x
        for l in range(3):
            h = h @ params[2 * l].T + params[2 * l + 1]
            if l < 2:
                h = torch.relu(h)
        loss = torch.nn.functional.cross_entropy(h, lab)
        assert abs(loss.item() - r["loss"][m]) < 1e-5 * max(1.0, abs(loss.item()))
        opt.zero_grad()
        loss.backward()
        opt.step()
    flat = np.concatenate([p.detach().numpy().reshape(-1) for p in params])
    np.testing.assert_allclose(r["W"][0], flat, rtol=2e-6, atol=2e-7)


def test_pipeline_handoff_equals_composed_network():
    """Section 3.1: a mini-batch's forward output at stage k is the input of
    stage k+1, and its input gradient at stage k+1 is the upstream gradient of
    stage k. With gamma = 1 (v stays 0, so every pass uses W0) the whole
    3-stage pipeline must reproduce, for every mini-batch, the composed
    network's loss, every stage's output and every stage's input gradient, as
    torch CPU autograd computes them on the three stages chained."""
    base = synth.SMALL_WORKLOADS["mlp3_small"]
    wl = dataclasses.replace(base, stages=tuple(dataclasses.replace(s, momentum=1.0) for s in base.stages),
                             steps=9)
    r = trajectory.run(wl, exact=True, keep_io=True)
    Ps = [stages.unpack(s, synth.initial_params(s)) for s in wl.stages]
    for m in range(wl.steps):
        x = torch.tensor(synth.stage_input(wl.stages[0], m), dtype=torch.float64, requires_grad=True)
        lab = torch.tensor(synth.labels(wl.stages[2], m), dtype=torch.long)
        hs = [x]
        for k, P in enumerate(Ps):
            z = hs[-1] @ torch.tensor(P["fc0.weight"]).T + torch.tensor(P["fc0.bias"])
            if k < 2:
                z = torch.relu(z)
                z.retain_grad()
            hs.append(z)
        loss = torch.nn.functional.cross_entropy(hs[-1], lab)
        loss.backward()
        assert abs(loss.item() - r["loss"][m]) <= 1e-12 * max(1.0, abs(loss.item()))
        for k in range(2):
            np.testing.assert_allclose(r["y"][(k, m)], hs[k + 1].detach().numpy(), rtol=1e-12, atol=1e-14)
            # the input gradient of stage k+1 is the gradient of stage k's output
            np.testing.assert_allclose(r["dx"][(k + 1, m)], hs[k + 1].grad.numpy(), rtol=1e-10, atol=1e-14)
        np.testing.assert_allclose(r["dx"][(0, m)], x.grad.numpy(), rtol=1e-10, atol=1e-14)


# ------------------------------------------- staleness policies (Section 4.2) ----

@pytest.mark.parametrize("policy", ["vanilla", "stash"])
@pytest.mark.parametrize("k,N", [(0, 3), (1, 3), (2, 3), (0, 4), (1, 4), (3, 4)])
def test_closed_form_constant_gradient_policies(policy, k, N):
    """Same dyadic closed form as above (W_t = W0 - t eta g exactly). Vanilla
    model parallelism runs every pass on the weights current at that pass;
    weight stashing runs the forward on the current weights and the backward on
    the forward's weights (Section 3.2, the PipeDream example). The forward
    outputs and backward dX must match those weight versions exactly."""
    spec, X, dY, W0, g = _fc_closed_form_setup(k, N)
    spec = dataclasses.replace(spec, policy=policy)
    wl = synth.Workload("closed_form", (spec,), steps=12)
    eta = spec.lr
    r = trajectory.run(wl, W0=[W0], v0=[g], inputs=lambda s, m: (X, dY, None), keep_io=True)
    done, at_forward = 0, {}
    for kind, m in schedule.stage_tasks(k, N, wl.steps):
        if kind == "F":
            at_forward[m] = done
            P = stages.unpack(spec, W0 - done * eta * g)
            assert np.array_equal(r["y"][(k, m)], np.maximum(X @ P["fc0.weight"].T + P["fc0.bias"], 0))
        else:
            version = at_forward[m] if policy == "stash" else done
            Wt = stages.unpack(spec, W0 - version * eta * g)
            assert np.array_equal(r["dx"][(k, m)], dY @ Wt["fc0.weight"])
            done += 1


def test_policies_coincide_without_staleness():
    """With one stage (N = 1) nothing is stale: F(m) and B(m) are adjacent and
    Eq. 5 / Eq. 6 give s = 0, so SpecTrain, Vanilla and weight stashing produce
    the same trajectory bit for bit."""
    base = synth.StageSpec("fc", "fp32", "ce", 0, 1, 7, 3, (37, 10, 50), 0.05, 0.9)
    runs = {}
    for policy in ("spectrain", "vanilla", "stash"):
        spec = dataclasses.replace(base, policy=policy)
        runs[policy] = trajectory.run(synth.Workload("p", (spec,), steps=6), W0=[synth.initial_params(base)])
    for policy in ("vanilla", "stash"):
        assert np.array_equal(runs[policy]["W"][0], runs["spectrain"]["W"][0])
        assert all(runs[policy]["loss"][m] == runs["spectrain"]["loss"][m] for m in range(6))


@pytest.mark.parametrize("N", [2, 3, 4])
def test_stash_staleness_is_updates_between_passes(N):
    """Brute force over the stage order: under weight stashing the backward of
    mini-batch m at stage k runs on weights that are as many updates old as
    the stage performed between F_k(m) and B_k(m) (N - 1 - k in steady state),
    while SpecTrain's backward prediction aims s_b updates ahead of the current
    weights (Eq. 6)."""
    M = 3 * N
    for k in range(N):
        tasks = schedule.stage_tasks(k, N, M)
        pos = {t: i for i, t in enumerate(tasks)}
        for m in range(N, M - N):
            between = sum(1 for kind, _ in tasks[pos[("F", m)] + 1:pos[("B", m)]] if kind == "B")
            assert between == N - 1 - k
        assert method.staleness_versions("stash", k, N) == (0, 0)
        assert method.staleness_versions("vanilla", k, N) == (0, 0)
        assert method.staleness_versions("spectrain", k, N) == (method.version_difference(k, N, True),
                                                                method.version_difference(k, N, False))
