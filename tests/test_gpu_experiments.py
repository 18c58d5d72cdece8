"""GPU checks of the experiments module: the prediction-accuracy experiment
(Section 3.2, Fig. 7) against the constant-gradient closed form, and the
three-policy loss comparison (Section 4.2) against the oracle."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import trajectory
from parity import TOL, rel

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def test_prediction_rmse_closed_form():
    """Dyadic FC stage whose gradient is the same exact value g at every step,
    started with v = g: W_t = W0 - t eta g exactly, so the library's prediction
    of W_{t+s} is exact (RMSE 0) and the stale weights W_t miss by s eta g
    (RMSE s eta sqrt(mean(g^2)))."""
    from paper_1809_02839_amd import experiments
    batch, fin, fout = 8, 16, 8
    spec = synth.StageSpec("fc", "fp32", "none", 0, 1, batch, 1, (fin, fout, fout), 2.0 ** -7, 0.875)
    rng = np.random.default_rng(7)
    X = (rng.integers(-1, 2, size=(batch, fin)) * 2.0 ** -3).astype(np.float32)
    dY = (rng.integers(-1, 2, size=(batch, fout)) * 2.0 ** -5).astype(np.float32)
    W0 = np.concatenate([rng.integers(-64, 65, size=fout * fin) * 2.0 ** -12, np.full(fout, 4.0)]).astype(np.float32)
    g = np.concatenate([(dY.T.astype(np.float64) @ X).reshape(-1), dY.sum(axis=0)]).astype(np.float32)
    steps = 12
    r = experiments.prediction_rmse(spec, steps, (1, 2, 3), W0=W0, v0=g, inputs=lambda sp, m: (X, dY, None))
    g_rms = float(np.sqrt(np.mean(g.astype(np.float64) ** 2)))
    for s in (1, 2, 3):
        assert r[s]["t"] == list(range(s, steps + 1))
        assert all(p == 0.0 for p in r[s]["predicted"])
        np.testing.assert_allclose(r[s]["stale"], s * 2.0 ** -7 * g_rms, rtol=1e-12)


def test_prediction_rmse_small_stack():
    """A 4-layer stack for 16 steps: one RMSE pair per reachable (t, s), finite."""
    from paper_1809_02839_amd import experiments
    spec = experiments.snn_spec(layers=4, hidden=64, batch=16, inputs=48, lr=1e-2)
    r = experiments.prediction_rmse(spec, 16)
    for s in (1, 2, 3):
        assert r[s]["t"] == list(range(s + 1, 17))
        assert np.all(np.isfinite(r[s]["predicted"])) and np.all(np.isfinite(r[s]["stale"]))
        assert min(r[s]["stale"]) > 0.0


@pytest.mark.parametrize("name", ["mlp3_small", "vgg_conv_small_pipe"])
def test_policy_losses_match_oracle(name):
    """Loss of every mini-batch of a reduced pipeline (the 3-stage MLP, the
    4-stage VGG with its classifier) under each staleness policy, against
    the oracle run with the same policy."""
    from paper_1809_02839_amd import experiments
    wl = synth.ALL_WORKLOADS[name]
    steps = 12
    got = experiments.policy_losses(wl, steps)
    tol = TOL[wl.stages[0].dtype]
    for policy, losses in got.items():
        ref_wl = synth.Workload(wl.name, tuple(dataclasses.replace(s, policy=policy) for s in wl.stages), steps)
        ref = trajectory.run(ref_wl)
        want = [ref["loss"][m] for m in range(steps)]
        assert rel(np.array(losses), np.array(want)) <= tol, (policy, losses, want)
    # the three policies see different weight versions in a 3-stage pipeline
    assert got["spectrain"] != got["vanilla"] and got["vanilla"] != got["stash"]
