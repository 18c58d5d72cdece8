"""Host checks of the teacher-forced stepwise harness (no GPU): the oracle's
own stash of every stage kind, written out in the buffer order and formats
the header lists for spectrain_stage_read_stash, is read back by
stepwise.oracle_stash_from_gpu into a stash the oracle's backward accepts,
giving the same gradients and dX."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import stages
from parity import rel
from stepwise import forward_buffers, oracle_stash_from_gpu, stash_count


def _bf16_bytes(a):
    return (synth.bf16_bits(np.asarray(a, np.float32))).view(np.uint8).reshape(-1)


def _f32_bytes(a):
    return np.ascontiguousarray(a, np.float32).view(np.uint8).reshape(-1)


def _to_gpu_layout(spec, st):
    """Stash buffers as the library lays them out (bytes by id)."""
    bf = spec.dtype == "bf16"
    act = _bf16_bytes if bf else _f32_bytes
    L, ce = spec.num_layers, spec.head == "ce"
    b = {i: np.empty(0, np.uint8) for i in range(stash_count(spec))}
    if spec.kind == "fc":
        for l in range(1, L):
            b[l - 1] = act(st["acts"][l])
        if ce:
            b[L - 1] = act(st["dlogits"])
    elif spec.kind == "conv3x3":
        for l in range(1, L):
            b[l - 1] = act(st["acts"][l])
        if ce:
            b[L - 1], b[L], b[L + 1] = act(st["acts"][L]), act(st["pooled"]), act(st["dlogits"])
    elif spec.kind == "bottleneck":
        for l, blk in enumerate(st["blocks"]):
            b[3 * l], b[3 * l + 1] = act(blk["t1"]), act(blk["t2"])
            if l < L - 1 or ce:
                b[3 * l + 2] = act(blk["y"])
        if ce:
            b[3 * L], b[3 * L + 1] = act(st["pooled"]), act(st["dlogits"])
    elif spec.kind == "transformer":
        for l, c in enumerate(st["layers"]):
            q = 13 * l
            b[q], b[q + 3], b[q + 4], b[q + 7], b[q + 8], b[q + 9] = (act(c[k]) for k in
                                                                      ("qkv", "ctx", "r1", "h", "f1", "r2"))
            if l > 0:
                b[13 * (l - 1) + 12] = act(c["a"])
        if ce:
            b[13 * (L - 1) + 12] = act(st["out"])
            b[13 * L] = act(st["dlogits"])
    elif spec.kind == "reslstm":
        for l, c in enumerate(st["layers"]):
            b[4 * l], b[4 * l + 1], b[4 * l + 2] = _f32_bytes(c["gates"]), _f32_bytes(c["c"]), act(c["h"])
            if l > 0:
                b[4 * (l - 1) + 3] = act(c["u"])
        if ce:
            b[4 * (L - 1) + 3] = act(st["out"])
            b[4 * L] = act(st["dlogits"])
    return b


CASES = ["mlp3_small", "vgg_conv_small", "resnet_bottleneck_small", "transformer_enc_small", "reslstm_small",
         "vgg_conv_small_pipe", "resnet_bottleneck_small_pipe", "transformer_enc_small_pipe"]


@pytest.mark.parametrize("name", CASES)
def test_stash_layout_round_trip(name):
    wl = synth.ALL_WORKLOADS[name]
    for spec in wl.stages:
        if spec.dtype == "fp32":
            spec = dataclasses.replace(spec, dtype="bf16") if spec.kind != "fc" else spec
        P = stages.unpack(spec, stages.weight_rounder(spec)(synth.initial_params(spec)))
        x = synth.stage_input(spec, 0)
        dy = synth.upstream_grad(spec, 0) if spec.head == "none" else None
        lab = synth.labels(spec, 0) if spec.head == "ce" else None
        y, _, st = stages.forward(spec, P, x, lab)
        got = oracle_stash_from_gpu(spec, _to_gpu_layout(spec, st), x, None if spec.head == "ce" else y)
        names = [n for n, _ in forward_buffers(spec, st)]
        assert names == [n for n, _ in forward_buffers(spec, got)] and names
        for (n, a), (_, b) in zip(forward_buffers(spec, got), forward_buffers(spec, st)):
            assert a.shape == b.shape, n
            # bf16 activations round-trip bit for bit; float32 ones (float32
            # stages, the LSTM's gates and cell state) to float32
            np.testing.assert_allclose(a.reshape(-1), np.asarray(b, np.float64).reshape(-1), rtol=2.0 ** -23, atol=0)
        dx1, g1 = stages.backward(spec, P, st, dy)
        dx2, g2 = stages.backward(spec, P, got, dy)
        # float32 storage of those activations may move a bf16 rounding inside
        # the backward by one step: the 2-norm difference stays far below it
        assert rel(stages.pack(spec, g2), stages.pack(spec, g1)) < 1e-3
        if dx1 is not None:
            assert rel(dx2, dx1) < 1e-3
