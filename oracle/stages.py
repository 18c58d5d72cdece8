"""Forward and backward of one pipeline stage, per workload kind
(test infrastructure only).

A stage is the group of layers one GPU owns (Section 2.2, model parallelism).
Its forward runs against the forward-predicted weights and stashes what the
backward needs; its backward runs against the backward-predicted weights
(every weight-dependent term of dX) and the stashed activations (dW), and
returns dX and the gradient g (Section 3.2: the version differences of Eq. 5
and Eq. 6 are separate for the two passes).

Rounding points (`q` is bf16 rounding for bf16 stages and the identity for
float32 stages and for the exact gradient checks): every tensor a stage stores
as a GEMM operand or stage output (activations, post-activation outputs,
gradients flowing between layers) is rounded with q; sums, normalisation
statistics, LSTM cell state, softmax probabilities inside attention before
they are used as an operand, and the weight gradient g are not.
"""
from typing import Dict, List, Tuple

import numpy as np

import synth

from . import layers as Lr
from .numerics import identity, to_bf16

LN_EPS = 1e-5


def rounder(spec, exact: bool = False):
    return identity if (exact or spec.dtype == "fp32") else to_bf16


def weight_rounder(spec):
    """Operand format of predicted weights: bf16 for bf16 stages, else float32
    (the prediction is already float32)."""
    return to_bf16 if spec.dtype == "bf16" else identity


def unpack(spec, flat) -> Dict[str, np.ndarray]:
    out, off = {}, 0
    flat = np.asarray(flat, dtype=np.float64)
    for name, shape, _ in synth.param_layout(spec):
        n = int(np.prod(shape))
        out[name] = flat[off:off + n].reshape(shape)
        off += n
    if off != flat.size:
        raise ValueError(f"flat parameter vector has {flat.size} values, layout needs {off}")
    return out


def pack(spec, tensors: Dict[str, np.ndarray]) -> np.ndarray:
    return np.concatenate([np.asarray(tensors[name], np.float64).reshape(-1)
                           for name, _, _ in synth.param_layout(spec)])


# ============================================================== forward ====

def forward(spec, P, x, labels=None, exact=False):
    """Returns (y, loss, stash). y is the stage output (logits for a CE head),
    loss is the mean cross-entropy for a CE head and None otherwise."""
    q = rounder(spec, exact)
    fn = {"fc": _fc_fwd, "conv3x3": _conv_fwd, "bottleneck": _bneck_fwd,
          "transformer": _tfm_fwd, "reslstm": _lstm_fwd}[spec.kind]
    return fn(spec, P, np.asarray(x, np.float64), labels, q)


def backward(spec, P, stash, dy=None, exact=False):
    """Returns (dx, grads) with grads keyed like the parameter layout.
    For a CE head dy is ignored (the head's dlogits is in the stash)."""
    q = rounder(spec, exact)
    fn = {"fc": _fc_bwd, "conv3x3": _conv_bwd, "bottleneck": _bneck_bwd,
          "transformer": _tfm_bwd, "reslstm": _lstm_bwd}[spec.kind]
    return fn(spec, P, stash, None if dy is None else np.asarray(dy, np.float64), q)


# ------------------------------------------------------------------ fc ----

def _fc_fwd(spec, P, x, labels, q):
    acts = [x]
    L = spec.num_layers
    loss = None
    for l in range(L):
        z = Lr.linear(acts[-1], P[f"fc{l}.weight"], P[f"fc{l}.bias"])
        if l == L - 1 and spec.head == "ce":
            loss, dlogits = Lr.softmax_cross_entropy(z, labels)
            return z, loss, {"acts": acts, "dlogits": q(dlogits)}
        acts.append(q(Lr.relu(z)))
    return acts[-1], loss, {"acts": acts}


def _fc_bwd(spec, P, st, dy, q):
    acts = st["acts"]
    L = spec.num_layers
    grads = {}
    if spec.head == "ce":
        dz = st["dlogits"]
    else:
        dz = dy * Lr.relu_mask(acts[L])
    dx = None
    for l in range(L - 1, -1, -1):
        grads[f"fc{l}.weight"] = dz.T @ acts[l]
        grads[f"fc{l}.bias"] = dz.sum(axis=0)
        da = q(dz @ P[f"fc{l}.weight"])
        if l > 0:
            dz = da * Lr.relu_mask(acts[l])
        else:
            dx = da
    return dx, grads


# ---------------------------------------------- classifier of conv stages ----

def _pool_head_fwd(P, y, labels, q, st):
    """Global average pool of the NHWC output over H x W, a linear layer to
    the classes and the mean softmax cross-entropy over the batch."""
    pooled = q(y.mean(axis=(1, 2)))
    logits = Lr.linear(pooled, P["head.weight"], P["head.bias"])
    loss, dlogits = Lr.softmax_cross_entropy(logits, np.asarray(labels).reshape(-1))
    st["pooled"] = pooled
    st["dlogits"] = q(dlogits)
    return logits, loss, st


def _pool_head_bwd(P, st, y_shape, q, grads):
    """Head gradients and dL/dY: the pooled gradient spread evenly over H x W."""
    dl = st["dlogits"]
    grads["head.weight"] = dl.T @ st["pooled"]
    grads["head.bias"] = dl.sum(axis=0)
    dpool = q(dl @ P["head.weight"])
    B, H, W, C = y_shape
    return np.broadcast_to(q(dpool / (H * W))[:, None, None, :], y_shape)


# ------------------------------------------------------------- conv3x3 ----

def _conv_fwd(spec, P, x, labels, q):
    acts = [x]
    for l in range(spec.num_layers):
        acts.append(q(Lr.relu(Lr.conv3x3_forward(acts[-1], P[f"conv{l}.weight"]))))
    if spec.head == "ce":
        return _pool_head_fwd(P, acts[-1], labels, q, {"acts": acts})
    return acts[-1], None, {"acts": acts}


def _conv_bwd(spec, P, st, dy, q):
    acts = st["acts"]
    L = spec.num_layers
    grads = {}
    if spec.head == "ce":
        dy = _pool_head_bwd(P, st, acts[L].shape, q, grads)
    dz = dy * Lr.relu_mask(acts[L])
    dx = None
    for l in range(L - 1, -1, -1):
        Wf = P[f"conv{l}.weight"]
        grads[f"conv{l}.weight"] = Lr.conv3x3_wgrad(dz, acts[l])
        da = q(Lr.conv3x3_dgrad(dz, Wf, acts[l].shape))
        if l > 0:
            dz = da * Lr.relu_mask(acts[l])
        else:
            dx = da
    return dx, grads


# ---------------------------------------------------------- bottleneck ----

def _bneck_fwd(spec, P, x, labels, q):
    """Block: y = relu(x + conv1x1_c(relu(conv3x3_b(relu(conv1x1_a(x)))))),
    identity skip, no bias, no normalisation."""
    blocks = []
    a = x
    for l in range(spec.num_layers):
        p = f"block{l}."
        t1 = q(Lr.relu(Lr.conv1x1_forward(a, P[p + "conv1.weight"])))
        t2 = q(Lr.relu(Lr.conv3x3_forward(t1, P[p + "conv2.weight"])))
        y = q(Lr.relu(a + Lr.conv1x1_forward(t2, P[p + "conv3.weight"])))
        blocks.append({"x": a, "t1": t1, "t2": t2, "y": y})
        a = y
    if spec.head == "ce":
        return _pool_head_fwd(P, a, labels, q, {"blocks": blocks})
    return a, None, {"blocks": blocks}


def _bneck_bwd(spec, P, st, dy, q):
    grads = {}
    blocks = st["blocks"]
    if spec.head == "ce":
        dy = _pool_head_bwd(P, st, blocks[-1]["y"].shape, q, grads)
    g = dy   # gradient w.r.t. the current block's output y
    for l in range(spec.num_layers - 1, -1, -1):
        p = f"block{l}."
        b = blocks[l]
        dr = g * Lr.relu_mask(b["y"])                    # through the output ReLU
        grads[p + "conv3.weight"] = Lr.conv1x1_wgrad(dr, b["t2"])
        dt2 = q(Lr.conv1x1_dgrad(dr, P[p + "conv3.weight"])) * Lr.relu_mask(b["t2"])
        grads[p + "conv2.weight"] = Lr.conv3x3_wgrad(dt2, b["t1"])
        dt1 = q(Lr.conv3x3_dgrad(dt2, P[p + "conv2.weight"], b["t1"].shape)) * Lr.relu_mask(b["t1"])
        grads[p + "conv1.weight"] = Lr.conv1x1_wgrad(dt1, b["x"])
        g = q(Lr.conv1x1_dgrad(dt1, P[p + "conv1.weight"]) + dr)   # main path + skip
    return g, grads


# ----------------------------------------------------------- transformer ----

def _tfm_fwd(spec, P, x, labels, q):
    """Post-LN encoder layer: h = LN1(x + W_o MHA(x) + b_o),
    y = LN2(h + W_2 relu(W_1 h + b_1) + b_2); softmax scale 1/sqrt(d_head),
    no mask, no dropout. A CE head projects every token to the vocabulary and
    averages the per-token loss (the target-token head of the last stage)."""
    dm, H, _, S = spec.dims[:4]
    B = spec.batch
    a = x.reshape(B * S, dm)
    layers = []
    for l in range(spec.num_layers):
        p = f"layer{l}."
        qkv = q(Lr.linear(a, P[p + "attn.qkv.weight"], P[p + "attn.qkv.bias"]))
        Q = Lr.split_heads(qkv[:, :dm], B, S, H)
        K = Lr.split_heads(qkv[:, dm:2 * dm], B, S, H)
        V = Lr.split_heads(qkv[:, 2 * dm:], B, S, H)
        Pr = q(Lr.attention_probs(Q, K))
        ctx = q(Lr.merge_heads(Pr @ V))
        r1 = q(a + Lr.linear(ctx, P[p + "attn.out.weight"], P[p + "attn.out.bias"]))
        h, _, _ = Lr.layernorm_forward(r1, P[p + "ln1.weight"], P[p + "ln1.bias"], LN_EPS)
        h = q(h)
        f1 = q(Lr.relu(Lr.linear(h, P[p + "ffn1.weight"], P[p + "ffn1.bias"])))
        r2 = q(h + Lr.linear(f1, P[p + "ffn2.weight"], P[p + "ffn2.bias"]))
        y, _, _ = Lr.layernorm_forward(r2, P[p + "ln2.weight"], P[p + "ln2.bias"], LN_EPS)
        layers.append({"a": a, "qkv": qkv, "ctx": ctx, "r1": r1, "h": h, "f1": f1, "r2": r2})
        a = q(y)
    st = {"layers": layers}
    if spec.head == "ce":
        # vocabulary projection of every token and the mean token cross-entropy
        logits = Lr.linear(a, P["vocab.weight"], P["vocab.bias"])
        loss, dlogits = Lr.softmax_cross_entropy(logits, np.asarray(labels).reshape(B * S))
        st["out"] = a
        st["dlogits"] = q(dlogits)
        return logits, loss, st
    return a.reshape(B, S, dm), None, st


def _attention_backward(dctx, qkv, B, S, H, q):
    dm = qkv.shape[1] // 3
    Q = Lr.split_heads(qkv[:, :dm], B, S, H)
    K = Lr.split_heads(qkv[:, dm:2 * dm], B, S, H)
    V = Lr.split_heads(qkv[:, 2 * dm:], B, S, H)
    scale = 1.0 / np.sqrt(Q.shape[-1])
    Pr = Lr.attention_probs(Q, K)                    # recomputed, unrounded
    dO = Lr.split_heads(dctx, B, S, H)
    dV = q(q(Pr).transpose(0, 1, 3, 2) @ dO)
    dP = dO @ V.transpose(0, 1, 3, 2)
    dS = q(Pr * (dP - (Pr * dP).sum(axis=-1, keepdims=True)))   # softmax backward
    dQ = q(dS @ K * scale)
    dK = q(dS.transpose(0, 1, 3, 2) @ Q * scale)
    return np.concatenate([Lr.merge_heads(dQ), Lr.merge_heads(dK), Lr.merge_heads(dV)], axis=1)


def _tfm_bwd(spec, P, st, dy, q):
    dm, H, _, S = spec.dims[:4]
    B = spec.batch
    grads = {}
    if spec.head == "ce":
        dl = st["dlogits"]
        grads["vocab.weight"] = dl.T @ st["out"]
        grads["vocab.bias"] = dl.sum(axis=0)
        g = q(dl @ P["vocab.weight"])
    else:
        g = dy.reshape(B * S, dm)
    for l in range(spec.num_layers - 1, -1, -1):
        p = f"layer{l}."
        c = st["layers"][l]
        _, xh2, rs2 = Lr.layernorm_forward(c["r2"], P[p + "ln2.weight"], P[p + "ln2.bias"], LN_EPS)
        dr2, grads[p + "ln2.weight"], grads[p + "ln2.bias"] = Lr.layernorm_backward(g, xh2, rs2, P[p + "ln2.weight"])
        dr2 = q(dr2)
        grads[p + "ffn2.weight"] = dr2.T @ c["f1"]
        grads[p + "ffn2.bias"] = dr2.sum(axis=0)
        df1 = q(dr2 @ P[p + "ffn2.weight"]) * Lr.relu_mask(c["f1"])
        grads[p + "ffn1.weight"] = df1.T @ c["h"]
        grads[p + "ffn1.bias"] = df1.sum(axis=0)
        dh = q(df1 @ P[p + "ffn1.weight"] + dr2)
        _, xh1, rs1 = Lr.layernorm_forward(c["r1"], P[p + "ln1.weight"], P[p + "ln1.bias"], LN_EPS)
        dr1, grads[p + "ln1.weight"], grads[p + "ln1.bias"] = Lr.layernorm_backward(dh, xh1, rs1, P[p + "ln1.weight"])
        dr1 = q(dr1)
        grads[p + "attn.out.weight"] = dr1.T @ c["ctx"]
        grads[p + "attn.out.bias"] = dr1.sum(axis=0)
        dctx = q(dr1 @ P[p + "attn.out.weight"])
        dqkv = _attention_backward(dctx, c["qkv"], B, S, H, q)
        grads[p + "attn.qkv.weight"] = dqkv.T @ c["a"]
        grads[p + "attn.qkv.bias"] = dqkv.sum(axis=0)
        g = q(dqkv @ P[p + "attn.qkv.weight"] + dr1)
    return g.reshape(B, S, dm), grads


# -------------------------------------------------------- residual LSTM ----

def _lstm_fwd(spec, P, x, labels, q):
    """Each layer: z_t = x_t W_x^T + h_{t-1} W_h^T + b, gates (i, f, g, o),
    c_t = f c_{t-1} + i g, h_t = o tanh(c_t), h_{-1} = c_{-1} = 0; the layer
    output is its input plus h (residual). A CE head projects to the vocabulary
    and averages the per-token loss."""
    T, B, _ = x.shape
    Hd = spec.dims[1]
    u = x
    layers = []
    for l in range(spec.num_layers):
        p = f"lstm{l}."
        zx = Lr.linear(u.reshape(T * B, -1), P[p + "weight_x"], P[p + "bias"]).reshape(T, B, 4 * Hd)
        Wh = P[p + "weight_h"]
        h_prev = np.zeros((B, Hd))
        c_prev = np.zeros((B, Hd))
        gates = np.empty((T, B, 4 * Hd))
        cs = np.empty((T, B, Hd))
        hs = np.empty((T, B, Hd))
        for t in range(T):
            z = zx[t] + h_prev @ Wh.T
            i = Lr.sigmoid(z[:, :Hd])
            f = Lr.sigmoid(z[:, Hd:2 * Hd])
            gg = np.tanh(z[:, 2 * Hd:3 * Hd])
            o = Lr.sigmoid(z[:, 3 * Hd:])
            c = f * c_prev + i * gg
            h = q(o * np.tanh(c))
            gates[t] = np.concatenate([i, f, gg, o], axis=1)
            cs[t], hs[t] = c, h
            h_prev, c_prev = h, c
        layers.append({"u": u, "gates": gates, "c": cs, "h": hs})
        u = q(u + hs)
    st = {"layers": layers, "out": u}
    if spec.head == "ce":
        logits = Lr.linear(u.reshape(T * B, Hd), P["vocab.weight"], P["vocab.bias"])
        loss, dlogits = Lr.softmax_cross_entropy(logits, np.asarray(labels).reshape(T * B))
        st["dlogits"] = q(dlogits)
        return logits, loss, st
    return u, None, st


def _lstm_bwd(spec, P, st, dy, q):
    Hd = spec.dims[1]
    T, B = spec.dims[2], spec.batch
    grads = {}
    if spec.head == "ce":
        dl = st["dlogits"]
        uL = st["out"].reshape(T * B, Hd)
        grads["vocab.weight"] = dl.T @ uL
        grads["vocab.bias"] = dl.sum(axis=0)
        du = q(dl @ P["vocab.weight"]).reshape(T, B, Hd)
    else:
        du = dy
    for l in range(spec.num_layers - 1, -1, -1):
        p = f"lstm{l}."
        c = st["layers"][l]
        Wh = P[p + "weight_h"]
        dz = np.empty((T, B, 4 * Hd))
        dh_rec = np.zeros((B, Hd))
        dc_next = np.zeros((B, Hd))
        for t in range(T - 1, -1, -1):
            gt = c["gates"][t]
            i, f, gg, o = gt[:, :Hd], gt[:, Hd:2 * Hd], gt[:, 2 * Hd:3 * Hd], gt[:, 3 * Hd:]
            tc = np.tanh(c["c"][t])
            c_prev = c["c"][t - 1] if t > 0 else np.zeros((B, Hd))
            dh = du[t] + dh_rec
            do = dh * tc
            dc = dc_next + dh * o * (1.0 - tc * tc)
            di, dg, df = dc * gg, dc * i, dc * c_prev
            dc_next = dc * f
            dz[t] = q(np.concatenate([di * i * (1 - i), df * f * (1 - f),
                                      dg * (1 - gg * gg), do * o * (1 - o)], axis=1))
            dh_rec = dz[t] @ Wh
        u2 = c["u"].reshape(T * B, -1)
        dz2 = dz.reshape(T * B, 4 * Hd)
        grads[p + "weight_x"] = dz2.T @ u2
        h_shift = np.concatenate([np.zeros((1, B, Hd)), c["h"][:-1]], axis=0).reshape(T * B, Hd)
        grads[p + "weight_h"] = dz2.T @ h_shift
        grads[p + "bias"] = dz2.sum(axis=0)
        du = q((dz2 @ P[p + "weight_x"]).reshape(T, B, -1) + du)
    return du, grads
