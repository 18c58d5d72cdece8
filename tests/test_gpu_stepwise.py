"""GPU stepwise parity: every forward, backward and update of the HIP path
against the oracle's recomputation of the same task from the GPU's state, for
every stage kind at reduced sizes (20 mini-batches, several GEMM tiles and
ragged tails), at the full benchmark sizes (20 mini-batches) and for single
layers of every full-size shape. bf16 backward passes are recomputed from
the GPU's own stashed activations (see stepwise.run_stepwise); every tensor
is held to the stated bound in both the 2-norm and the max-abs normwise
metric."""
import dataclasses

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
    worst = run_stepwise(wl, wl.steps, torch)
    print(f"[stepwise] {name}: {worst.report()}", flush=True)


# 20 mini-batches of every full-size stage: its N - k warm-up forwards, then
# backward, update and forward alternating (forwards against predictions
# from a non-zero smoothed gradient from the first update on). The oracle
# recomputes every task of the float32 and VGG stages; for the deeper stages
# (a full-size oracle step takes it 20-45 s) the forward and backward of a
# sample of mini-batches: the first (weights W0), the first forward after
# the first update, one from the middle and the last.
FULL = {"mlp3": None, "vgg_conv": None, "resnet_bottleneck": {0, 2, 10, 19}, "transformer_enc": {0, 3, 10, 19},
        "reslstm": {0, 1, 10, 19}}


@pytest.mark.parametrize("name", list(FULL))
def test_stepwise_full_size(name):
    wl = synth.WORKLOADS[name]
    print(f"[stepwise-full] {name} steps=20 checked={sorted(FULL[name]) if FULL[name] else 'all'}", flush=True)
    worst = run_stepwise(wl, 20, torch, check=FULL[name])
    print(f"[stepwise-full] {name}: {worst.report()}", flush=True)


def _one_layer(name, check=None, **change):
    spec = dataclasses.replace(synth.WORKLOADS[name].stages[0], num_layers=1, **change)
    return synth.Workload(f"{name}/1", (spec,), 20), check


# one layer of each full-size shape: the VGG stage's first (256 -> 512) and
# later (512 -> 512) convolutions, one bottleneck block (1024/256 at 14x14,
# batch 64), one encoder layer (d = 512, S = 128, batch 64) and one LSTM
# layer (H = 1024, T = 35, batch 64) with the 10000-token head
SINGLE = {
    "vgg_conv_first": lambda: _one_layer("vgg_conv"),
    "vgg_conv_later": lambda: _one_layer("vgg_conv", dims=(512, 512, 8, 8)),
    "resnet_bottleneck_block": lambda: _one_layer("resnet_bottleneck", {0, 2, 5, 10, 15, 19}),
    "transformer_enc_layer": lambda: _one_layer("transformer_enc", {0, 3, 10, 19}),
    "reslstm_layer": lambda: _one_layer("reslstm", {0, 1, 5, 10, 19}),
}


@pytest.mark.parametrize("name", list(SINGLE))
def test_stepwise_full_shape_single_layer(name):
    wl, check = SINGLE[name]()
    print(f"[stepwise-layer] {name} steps={wl.steps} checked={sorted(check) if check else 'all'}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch, check=check)
    print(f"[stepwise-layer] {name}: {worst.report()}", flush=True)


def _with_policy(wl, policy):
    return synth.Workload(f"{wl.name}/{policy}", tuple(dataclasses.replace(s, policy=policy) for s in wl.stages),
                          wl.steps)


# reslstm_small's stage is the last of its pipeline (forward and backward of
# a mini-batch adjacent, every policy giving the same weights): the policy
# runs take the same stage at k = 1 of 4
POLICY_WORKLOADS = ["mlp3_small", "vgg_conv_small", "vgg_conv_mid", "resnet_bottleneck_small",
                    "transformer_enc_small", "reslstm_small_k1"]


@pytest.mark.parametrize("policy", ["vanilla", "stash"])
@pytest.mark.parametrize("name", POLICY_WORKLOADS)
def test_stepwise_small_policies(name, policy):
    """The Vanilla and weight-stashing pipelines of Section 4.2 on the same
    stage kinds: every task against the oracle's recomputation of it."""
    wl = _with_policy(synth.ALL_WORKLOADS[name], policy)
    print(f"[stepwise] {wl.name}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch)
    print(f"[stepwise] {wl.name}: {worst.report()}", flush=True)


@pytest.mark.parametrize("policy", ["vanilla", "stash"])
def test_stepwise_full_size_vgg_policies(policy):
    wl = _with_policy(synth.WORKLOADS["vgg_conv"], policy)
    print(f"[stepwise-full] {wl.name} steps=8", flush=True)
    worst = run_stepwise(wl, 8, torch)
    print(f"[stepwise-full] {wl.name}: {worst.report()}", flush=True)


# Whole 4-stage pipelines of each bf16 model (every stage simulated, the
# last stage's loss head or synthetic upstream gradient starting each
# backward): every task of every stage against the oracle.
@pytest.mark.parametrize("name", ["vgg_conv_small_pipe", "resnet_bottleneck_small_pipe", "transformer_enc_small_pipe",
                                  "transformer_enc_mid_pipe", "reslstm_small_pipe", "reslstm_mid_pipe"])
def test_stepwise_pipeline(name):
    wl = synth.ALL_WORKLOADS[name]
    print(f"[stepwise-pipe] {name}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch)
    print(f"[stepwise-pipe] {name}: {worst.report()}", flush=True)


def test_stepwise_transformer_vocab_head_full_size():
    """The transformer's last stage at full size: 3 layers and the
    32000-token projection with the mean token cross-entropy."""
    wl = synth.ALL_WORKLOADS["transformer_enc_last"]
    print("[stepwise-full] transformer_enc_last steps=6", flush=True)
    worst = run_stepwise(wl, 6, torch)
    print(f"[stepwise-full] transformer_enc_last: {worst.report()}", flush=True)
