"""GPU stepwise parity: every forward, backward and update of the HIP path
against the oracle's recomputation of the same task from the GPU's state, for
every stage kind at reduced sizes (20 mini-batches, several GEMM tiles and
ragged tails) and at the full benchmark sizes (enough mini-batches to reach a
forward that uses a non-trivial prediction; bf16 gradient quantities there
are held to the accuracy of the oracle's own bf16 emulation, see
stepwise.run_stepwise)."""
import pytest

import synth
from stepwise import run_stepwise

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.mark.parametrize("name", ["mlp3_small", "vgg_conv_small", "vgg_conv_mid", "resnet_bottleneck_small",
                                  "transformer_enc_small", "transformer_enc_mid", "reslstm_small", "reslstm_mid"])
def test_stepwise_small(name):
    wl = synth.ALL_WORKLOADS[name]
    print(f"[stepwise] {name}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch, derived=wl.stages[0].dtype == "bf16")
    print(f"[stepwise] {name}: {worst.report()}", flush=True)


# steps: the stage's N - k warm-up forwards, one backward + update, then a
# forward against a prediction from a non-zero smoothed gradient
FULL = {"mlp3": 20, "vgg_conv": 4, "resnet_bottleneck": 3, "transformer_enc": 4, "reslstm": 2}


@pytest.mark.parametrize("name", list(FULL))
def test_stepwise_full_size(name):
    wl = synth.WORKLOADS[name]
    print(f"[stepwise-full] {name} steps={FULL[name]}", flush=True)
    worst = run_stepwise(wl, FULL[name], torch, derived=wl.stages[0].dtype == "bf16")
    print(f"[stepwise-full] {name}: {worst.report()}", flush=True)


def _with_policy(wl, policy):
    import dataclasses
    return synth.Workload(f"{wl.name}/{policy}", tuple(dataclasses.replace(s, policy=policy) for s in wl.stages),
                          wl.steps)


@pytest.mark.parametrize("policy", ["vanilla", "stash"])
@pytest.mark.parametrize("name", ["mlp3_small", "vgg_conv_small", "vgg_conv_mid", "resnet_bottleneck_small",
                                  "transformer_enc_small", "reslstm_small"])
def test_stepwise_small_policies(name, policy):
    """The Vanilla and weight-stashing pipelines of Section 4.2 on the same
    stage kinds: every task against the oracle's recomputation of it."""
    wl = _with_policy(synth.ALL_WORKLOADS[name], policy)
    print(f"[stepwise] {wl.name}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch, derived=wl.stages[0].dtype == "bf16")
    print(f"[stepwise] {wl.name}: {worst.report()}", flush=True)


@pytest.mark.parametrize("policy", ["vanilla", "stash"])
def test_stepwise_full_size_vgg_policies(policy):
    wl = _with_policy(synth.WORKLOADS["vgg_conv"], policy)
    print(f"[stepwise-full] {wl.name} steps=4", flush=True)
    worst = run_stepwise(wl, 4, torch, derived=True)
    print(f"[stepwise-full] {wl.name}: {worst.report()}", flush=True)


# Whole 4-stage pipelines of each bf16 model (every stage simulated, the
# last stage's loss head or synthetic upstream gradient starting each
# backward): every task of every stage against the oracle.
@pytest.mark.parametrize("name", ["vgg_conv_small_pipe", "resnet_bottleneck_small_pipe", "transformer_enc_small_pipe",
                                  "transformer_enc_mid_pipe", "reslstm_small_pipe", "reslstm_mid_pipe"])
def test_stepwise_pipeline(name):
    wl = synth.ALL_WORKLOADS[name]
    print(f"[stepwise-pipe] {name}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch, derived=True)
    print(f"[stepwise-pipe] {name}: {worst.report()}", flush=True)


def test_stepwise_transformer_vocab_head_full_size():
    """The transformer's last stage at full size: 3 layers and the
    32000-token projection with the mean token cross-entropy."""
    wl = synth.ALL_WORKLOADS["transformer_enc_last"]
    print("[stepwise-full] transformer_enc_last steps=2", flush=True)
    worst = run_stepwise(wl, 2, torch, derived=True)
    print(f"[stepwise-full] transformer_enc_last: {worst.report()}", flush=True)
