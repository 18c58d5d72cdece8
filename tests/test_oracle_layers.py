"""Pins of the oracle's stage forward/backward: central finite differences in
float64 on tiny stages of every kind, and special cases that reduce to torch
CPU library routines (conv2d, LSTM, TransformerEncoderLayer, layer_norm,
cross_entropy) and to the bf16 format definition."""
import numpy as np
import pytest
import torch

import synth
from oracle import layers as Lr
from oracle import numerics, stages

TINY = {
    "fc": synth.StageSpec("fc", "fp32", "none", 0, 2, 3, 2, (5, 4, 6), 0.01, 0.9),
    "fc_ce": synth.StageSpec("fc", "fp32", "ce", 1, 2, 4, 2, (5, 3, 6), 0.01, 0.9),
    "conv3x3": synth.StageSpec("conv3x3", "bf16", "none", 1, 4, 2, 2, (2, 3, 4, 3), 0.01, 0.9),
    "bottleneck": synth.StageSpec("bottleneck", "bf16", "none", 1, 4, 2, 2, (4, 2, 3, 4), 0.01, 0.9),
    "conv3x3_ce": synth.StageSpec("conv3x3", "bf16", "ce", 3, 4, 3, 2, (2, 3, 4, 3, 5), 0.01, 0.9),
    "bottleneck_ce": synth.StageSpec("bottleneck", "bf16", "ce", 3, 4, 3, 2, (4, 2, 3, 4, 5), 0.01, 0.9),
    "transformer": synth.StageSpec("transformer", "bf16", "none", 1, 4, 2, 2, (8, 2, 6, 4), 0.01, 0.9),
    "transformer_ce": synth.StageSpec("transformer", "bf16", "ce", 3, 4, 2, 2, (8, 2, 6, 4, 7), 0.01, 0.9),
    "reslstm": synth.StageSpec("reslstm", "bf16", "none", 1, 4, 2, 2, (3, 3, 4, 7), 0.01, 0.9),
    "reslstm_ce": synth.StageSpec("reslstm", "bf16", "ce", 3, 4, 2, 2, (3, 3, 4, 7), 0.01, 0.9),
}


def _random_params(spec, rng):
    flat = []
    for _, shape, init in synth.param_layout(spec):
        n = int(np.prod(shape))
        base = 1.0 if init == "ones" else 0.0
        flat.append(base + rng.standard_normal(n) * (0.6 if init == "he" else 0.2))
    return np.concatenate(flat)


def _scalar_loss(spec, flat, x, lab, R):
    P = stages.unpack(spec, flat)
    y, loss, _ = stages.forward(spec, P, x, lab, exact=True)
    return loss if spec.head == "ce" else float(np.sum(y * R))


@pytest.mark.parametrize("name", list(TINY))
def test_stage_gradients_central_differences(name):
    spec = TINY[name]
    rng = np.random.default_rng(11)
    flat = _random_params(spec, rng)
    x = rng.standard_normal(spec.input_shape())
    lab = rng.integers(0, spec.num_classes(), size=spec.label_shape()) if spec.head == "ce" else None
    R = None if spec.head == "ce" else rng.standard_normal(spec.output_shape())
    P = stages.unpack(spec, flat)
    y, loss, stash = stages.forward(spec, P, x, lab, exact=True)
    dx, grads = stages.backward(spec, P, stash, R, exact=True)
    g = stages.pack(spec, grads)
    eps = 1e-6
    idx = rng.choice(flat.size, size=min(flat.size, 60), replace=False)
    for i in idx:
        e = np.zeros_like(flat)
        e[i] = eps
        fd = (_scalar_loss(spec, flat + e, x, lab, R) - _scalar_loss(spec, flat - e, x, lab, R)) / (2 * eps)
        assert abs(fd - g[i]) <= 1e-6 * max(1.0, abs(fd)), (name, i, fd, g[i])
    xi = rng.choice(x.size, size=min(x.size, 30), replace=False)
    for i in xi:
        e = np.zeros(x.size)
        e[i] = eps
        e = e.reshape(x.shape)
        fd = (_scalar_loss(spec, flat, x + e, lab, R) - _scalar_loss(spec, flat, x - e, lab, R)) / (2 * eps)
        assert abs(fd - dx.reshape(-1)[i]) <= 1e-6 * max(1.0, abs(fd)), (name, "dx", i)


def test_bf16_rounding_matches_torch_and_format():
    rng = np.random.default_rng(3)
    v = np.concatenate([rng.standard_normal(5000) * 10.0 ** rng.integers(-30, 30, 5000),
                        [0.0, -0.0, 1.0, 1.00390625, 1.01171875, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8,
                         3.0e38, 1e-40, -1e-39, 2.0 ** -133 * 1.5]])
    ref = torch.tensor(v.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    got = numerics.to_bf16(v)
    assert np.array_equal(got, ref)
    # ties go to even: 1 + 2^-8 sits halfway between 1 and 1 + 2^-7
    assert numerics.to_bf16(np.array([1.0 + 2 ** -8]))[0] == 1.0
    assert numerics.to_bf16(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6


def test_conv3x3_matches_torch_conv2d():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 5, 4, 3))
    Wf = rng.standard_normal((6, 3, 3, 3))
    y = Lr.conv3x3_forward(x, Wf)
    xt = torch.tensor(x).permute(0, 3, 1, 2)
    wt = torch.tensor(Wf).permute(0, 3, 1, 2)
    ref = torch.nn.functional.conv2d(xt, wt, padding=1).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_conv_stage_backward_matches_torch_autograd():
    spec = TINY["bottleneck"]
    rng = np.random.default_rng(8)
    flat = _random_params(spec, rng)
    x = rng.standard_normal(spec.input_shape())
    R = rng.standard_normal(spec.output_shape())
    P = stages.unpack(spec, flat)
    y, _, st = stages.forward(spec, P, x, exact=True)
    dx, grads = stages.backward(spec, P, st, R, exact=True)
    T = {k: torch.tensor(v, requires_grad=True) for k, v in P.items()}
    a = torch.tensor(x, requires_grad=True)
    h = a.permute(0, 3, 1, 2)
    conv = lambda t, w, pad: torch.nn.functional.conv2d(t, w.permute(0, 3, 1, 2), padding=pad)
    for l in range(spec.num_layers):
        p = f"block{l}."
        t1 = torch.relu(conv(h, T[p + "conv1.weight"], 0))
        t2 = torch.relu(conv(t1, T[p + "conv2.weight"], 1))
        h = torch.relu(h + conv(t2, T[p + "conv3.weight"], 0))
    out = h.permute(0, 2, 3, 1)
    np.testing.assert_allclose(y, out.detach().numpy(), rtol=1e-10, atol=1e-12)
    (out * torch.tensor(R)).sum().backward()
    np.testing.assert_allclose(dx, a.grad.numpy(), rtol=1e-9, atol=1e-12)
    for k in T:
        np.testing.assert_allclose(grads[k], T[k].grad.numpy(), rtol=1e-9, atol=1e-12)


def test_conv_classifier_head_matches_torch_autograd():
    """conv3x3 stage with the classifier head: torch conv2d, ReLU,
    adaptive_avg_pool2d, linear and cross_entropy give the same loss, logits
    and gradients."""
    spec = TINY["conv3x3_ce"]
    rng = np.random.default_rng(9)
    flat = _random_params(spec, rng)
    x = rng.standard_normal(spec.input_shape())
    lab = rng.integers(0, spec.num_classes(), size=spec.label_shape())
    P = stages.unpack(spec, flat)
    logits, loss, st = stages.forward(spec, P, x, lab, exact=True)
    dx, grads = stages.backward(spec, P, st, None, exact=True)
    T = {k: torch.tensor(v, requires_grad=True) for k, v in P.items()}
    a = torch.tensor(x, requires_grad=True)
    h = a.permute(0, 3, 1, 2)
    for l in range(spec.num_layers):
        h = torch.relu(torch.nn.functional.conv2d(h, T[f"conv{l}.weight"].permute(0, 3, 1, 2), padding=1))
    pooled = torch.nn.functional.adaptive_avg_pool2d(h, 1).flatten(1)
    z = torch.nn.functional.linear(pooled, T["head.weight"], T["head.bias"])
    ref = torch.nn.functional.cross_entropy(z, torch.tensor(lab))
    np.testing.assert_allclose(logits, z.detach().numpy(), rtol=1e-10, atol=1e-12)
    assert abs(loss - ref.item()) < 1e-12
    ref.backward()
    np.testing.assert_allclose(dx, a.grad.numpy(), rtol=1e-9, atol=1e-13)
    for k in T:
        np.testing.assert_allclose(grads[k], T[k].grad.numpy(), rtol=1e-9, atol=1e-13, err_msg=k)


def test_lstm_stage_matches_torch_lstm():
    spec = TINY["reslstm"]
    rng = np.random.default_rng(9)
    flat = _random_params(spec, rng)
    x = rng.standard_normal(spec.input_shape())
    R = rng.standard_normal(spec.output_shape())
    P = stages.unpack(spec, flat)
    y, _, st = stages.forward(spec, P, x, exact=True)
    dx, grads = stages.backward(spec, P, st, R, exact=True)
    I, H = spec.dims[0], spec.dims[1]
    a = torch.tensor(x, requires_grad=True)
    u = a
    mods = []
    for l in range(spec.num_layers):
        m = torch.nn.LSTM(I if l == 0 else H, H).double()
        with torch.no_grad():
            m.weight_ih_l0.copy_(torch.tensor(P[f"lstm{l}.weight_x"]))
            m.weight_hh_l0.copy_(torch.tensor(P[f"lstm{l}.weight_h"]))
            m.bias_ih_l0.copy_(torch.tensor(P[f"lstm{l}.bias"]))
            m.bias_hh_l0.zero_()
        mods.append(m)
        hseq, _ = m(u)
        u = u + hseq
    np.testing.assert_allclose(y, u.detach().numpy(), rtol=1e-10, atol=1e-12)
    (u * torch.tensor(R)).sum().backward()
    np.testing.assert_allclose(dx, a.grad.numpy(), rtol=1e-9, atol=1e-12)
    for l, m in enumerate(mods):
        np.testing.assert_allclose(grads[f"lstm{l}.weight_x"], m.weight_ih_l0.grad.numpy(), rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose(grads[f"lstm{l}.weight_h"], m.weight_hh_l0.grad.numpy(), rtol=1e-9, atol=1e-12)
        np.testing.assert_allclose(grads[f"lstm{l}.bias"], m.bias_ih_l0.grad.numpy(), rtol=1e-9, atol=1e-12)


def test_transformer_stage_matches_torch_encoder_layer():
    spec = TINY["transformer"]
    dm, H, F, S = spec.dims
    rng = np.random.default_rng(10)
    flat = _random_params(spec, rng)
    x = rng.standard_normal(spec.input_shape())
    R = rng.standard_normal(spec.output_shape())
    P = stages.unpack(spec, flat)
    y, _, st = stages.forward(spec, P, x, exact=True)
    dx, grads = stages.backward(spec, P, st, R, exact=True)
    a = torch.tensor(x, requires_grad=True)
    h = a
    mods = []
    for l in range(spec.num_layers):
        p = f"layer{l}."
        m = torch.nn.TransformerEncoderLayer(dm, H, F, dropout=0.0, activation="relu",
                                             batch_first=True, norm_first=False, layer_norm_eps=1e-5).double()
        with torch.no_grad():
            m.self_attn.in_proj_weight.copy_(torch.tensor(P[p + "attn.qkv.weight"]))
            m.self_attn.in_proj_bias.copy_(torch.tensor(P[p + "attn.qkv.bias"]))
            m.self_attn.out_proj.weight.copy_(torch.tensor(P[p + "attn.out.weight"]))
            m.self_attn.out_proj.bias.copy_(torch.tensor(P[p + "attn.out.bias"]))
            m.linear1.weight.copy_(torch.tensor(P[p + "ffn1.weight"]))
            m.linear1.bias.copy_(torch.tensor(P[p + "ffn1.bias"]))
            m.linear2.weight.copy_(torch.tensor(P[p + "ffn2.weight"]))
            m.linear2.bias.copy_(torch.tensor(P[p + "ffn2.bias"]))
            m.norm1.weight.copy_(torch.tensor(P[p + "ln1.weight"]))
            m.norm1.bias.copy_(torch.tensor(P[p + "ln1.bias"]))
            m.norm2.weight.copy_(torch.tensor(P[p + "ln2.weight"]))
            m.norm2.bias.copy_(torch.tensor(P[p + "ln2.bias"]))
        m.train()
        mods.append(m)
        h = m(h)
    np.testing.assert_allclose(y, h.detach().numpy(), rtol=1e-9, atol=1e-11)
    (h * torch.tensor(R)).sum().backward()
    np.testing.assert_allclose(dx, a.grad.numpy(), rtol=1e-8, atol=1e-11)
    for l, m in enumerate(mods):
        p = f"layer{l}."
        pairs = [("attn.qkv.weight", m.self_attn.in_proj_weight), ("attn.qkv.bias", m.self_attn.in_proj_bias),
                 ("attn.out.weight", m.self_attn.out_proj.weight), ("attn.out.bias", m.self_attn.out_proj.bias),
                 ("ffn1.weight", m.linear1.weight), ("ffn1.bias", m.linear1.bias),
                 ("ffn2.weight", m.linear2.weight), ("ffn2.bias", m.linear2.bias),
                 ("ln1.weight", m.norm1.weight), ("ln1.bias", m.norm1.bias),
                 ("ln2.weight", m.norm2.weight), ("ln2.bias", m.norm2.bias)]
        for name, t in pairs:
            np.testing.assert_allclose(grads[p + name], t.grad.numpy(), rtol=1e-8, atol=1e-11, err_msg=name)


def test_cross_entropy_zero_logits_and_torch():
    C, n = 10000, 6
    lab = np.arange(n) * 7 % C
    loss, d = Lr.softmax_cross_entropy(np.zeros((n, C)), lab)
    assert abs(loss - np.log(C)) < 1e-12
    expect = np.full((n, C), 1.0 / C)
    expect[np.arange(n), lab] -= 1.0
    np.testing.assert_allclose(d, expect / n, rtol=1e-12, atol=1e-18)
    rng = np.random.default_rng(1)
    z = rng.standard_normal((n, 13)) * 5
    lab = rng.integers(0, 13, n)
    loss, d = Lr.softmax_cross_entropy(z, lab)
    zt = torch.tensor(z, requires_grad=True)
    ref = torch.nn.functional.cross_entropy(zt, torch.tensor(lab))
    ref.backward()
    assert abs(loss - ref.item()) < 1e-12
    np.testing.assert_allclose(d, zt.grad.numpy(), rtol=1e-10, atol=1e-15)


@pytest.mark.parametrize("name", ["reslstm_ce", "transformer_ce", "conv3x3_ce", "bottleneck_ce"])
def test_zero_head_weights_give_ln_classes(name):
    """CE head with zero vocabulary weights and bias: loss = ln C exactly and
    the head gradient is (1/C - onehot)/count, with one target per token."""
    spec = TINY[name]
    rng = np.random.default_rng(2)
    flat = _random_params(spec, rng)
    P = stages.unpack(spec, flat)
    head = "head" if spec.kind in ("conv3x3", "bottleneck") else "vocab"
    P[head + ".weight"][:] = 0
    P[head + ".bias"][:] = 0
    x = rng.standard_normal(spec.input_shape())
    C = spec.num_classes()
    lab = rng.integers(0, C, size=spec.label_shape())
    _, loss, st = stages.forward(spec, P, x, lab, exact=True)
    assert abs(loss - np.log(C)) < 1e-12
    n = int(np.prod(spec.label_shape()))
    expect = np.full((n, C), 1.0 / C)
    expect[np.arange(n), lab.reshape(-1)] -= 1
    np.testing.assert_allclose(st["dlogits"], expect / n, rtol=1e-12)
