"""Seeded synthetic inputs and the workload table for SpecTrain stage steps.

This module is shared by the CPU oracle and the HIP path. It holds no step of
the method: only the description of each workload (shapes, learning rate,
momentum, pipeline position), the flat parameter layout both sides agree on,
and seeded random draws of initial weights, stage inputs, upstream gradients
and labels.

Inputs stand in for the paper's datasets (CIFAR-10 images, IMDb reviews;
Section 4.1), which are not used: every array here is drawn from a seeded
normal or uniform generator with the shape of the corresponding workload.

bf16 workloads receive their floating inputs already rounded once to bf16
(round-to-nearest-even) and stored as the float32 value of that bf16 number,
so both sides see identical input bits.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np

KINDS = ("fc", "conv3x3", "bottleneck", "transformer", "reslstm")
INIT_SEED = 1809
DATA_SEED = 2839


@dataclasses.dataclass(frozen=True)
class StageSpec:
    """One pipeline stage: what it computes and where it sits.

    dims meaning per kind:
      fc:          (in_features, out_features, hidden)   widths in, hidden*(L-1), out
      conv3x3:     (C_in, C_out, H, W[, classes])         L layers, first C_in->C_out
      bottleneck:  (C, C_mid, H, W[, classes])            L blocks
                   (a CE head on a conv stage: global average pool, linear to classes)
      transformer: (d_model, heads, ffn, seq[, vocab])    L encoder layers, vocab used by a CE head
      reslstm:     (input, hidden, T, vocab)              L layers, vocab used by a CE head
    """

    kind: str
    dtype: str              # "fp32" or "bf16": the compute dtype of operands
    head: str               # "none" (dY supplied) or "ce" (labels supplied)
    stage_index: int        # k, 0-based
    num_stages: int         # N
    batch: int
    num_layers: int
    dims: Tuple[int, ...]
    lr: float
    momentum: float
    # how a pass treats weight staleness: "spectrain" (predicted weights),
    # "vanilla" (the latest weights at every pass) or "stash" (the backward
    # reuses the weights of its own forward)
    policy: str = "spectrain"
    # bottleneck: start every block's last convolution at zero, so each block
    # is the identity at initialisation (whole stacks without normalisation)
    zero_residual: bool = False

    # ----- shapes -------------------------------------------------------
    def fc_widths(self) -> List[int]:
        fin, fout, hid = self.dims[0], self.dims[1], self.dims[2]
        return [fin] + [hid] * (self.num_layers - 1) + [fout]

    def input_shape(self) -> Tuple[int, ...]:
        d = self.dims
        if self.kind == "fc":
            return (self.batch, d[0])
        if self.kind == "conv3x3":
            return (self.batch, d[2], d[3], d[0])          # NHWC
        if self.kind == "bottleneck":
            return (self.batch, d[2], d[3], d[0])          # NHWC
        if self.kind == "transformer":
            return (self.batch, d[3], d[0])                # [B, S, d]
        if self.kind == "reslstm":
            return (d[2], self.batch, d[0])                # time-major [T, B, I]
        raise ValueError(self.kind)

    def output_shape(self) -> Tuple[int, ...]:
        """Shape of Y for a stage without a loss head (the tensor dY matches)."""
        d = self.dims
        if self.kind == "fc":
            return (self.batch, d[1])
        if self.kind == "conv3x3":
            return (self.batch, d[2], d[3], d[1])
        if self.kind == "bottleneck":
            return (self.batch, d[2], d[3], d[0])
        if self.kind == "transformer":
            return (self.batch, d[3], d[0])
        if self.kind == "reslstm":
            return (d[2], self.batch, d[1])
        raise ValueError(self.kind)

    def label_shape(self) -> Tuple[int, ...]:
        if self.kind in ("fc", "conv3x3", "bottleneck"):
            return (self.batch,)
        if self.kind == "transformer":
            return (self.batch, self.dims[3])              # one target per token
        if self.kind == "reslstm":
            return (self.dims[2], self.batch)
        raise ValueError(f"{self.kind} has no loss head")

    def num_classes(self) -> int:
        if self.kind == "fc":
            return self.dims[1]
        if self.kind in ("conv3x3", "bottleneck", "transformer"):
            return self.dims[4]
        if self.kind == "reslstm":
            return self.dims[3]
        raise ValueError(self.kind)

    def grad_count(self) -> int:
        """Samples (or tokens) the synthetic upstream gradient is averaged over."""
        if self.kind == "transformer":
            return self.batch * self.dims[3]
        if self.kind == "reslstm":
            return self.batch * self.dims[2]
        return self.batch


def param_layout(spec: StageSpec) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Ordered (name, shape, init) list: the flat parameter order of a stage.

    init is "he" (normal, variance 2/fan_in with fan_in the product of all but
    the first dimension), "zeros" or "ones". Linear weights are [out, in]
    row-major, conv filters [C_out, kh, kw, C_in], LSTM gate blocks (i, f, g, o).
    """
    d, L = spec.dims, spec.num_layers
    out: List[Tuple[str, Tuple[int, ...], str]] = []
    if spec.kind == "fc":
        w = spec.fc_widths()
        for l in range(L):
            out.append((f"fc{l}.weight", (w[l + 1], w[l]), "he"))
            out.append((f"fc{l}.bias", (w[l + 1],), "zeros"))
    elif spec.kind == "conv3x3":
        cin, cout = d[0], d[1]
        for l in range(L):
            out.append((f"conv{l}.weight", (cout, 3, 3, cin if l == 0 else cout), "he"))
        if spec.head == "ce":
            out.append(("head.weight", (d[4], cout), "he"))
            out.append(("head.bias", (d[4],), "zeros"))
    elif spec.kind == "bottleneck":
        c, cm = d[0], d[1]
        for l in range(L):
            out.append((f"block{l}.conv1.weight", (cm, 1, 1, c), "he"))
            out.append((f"block{l}.conv2.weight", (cm, 3, 3, cm), "he"))
            out.append((f"block{l}.conv3.weight", (c, 1, 1, cm), "zeros" if spec.zero_residual else "he"))
        if spec.head == "ce":
            out.append(("head.weight", (d[4], c), "he"))
            out.append(("head.bias", (d[4],), "zeros"))
    elif spec.kind == "transformer":
        dm, ffn = d[0], d[2]
        for l in range(L):
            p = f"layer{l}."
            out += [
                (p + "attn.qkv.weight", (3 * dm, dm), "he"),
                (p + "attn.qkv.bias", (3 * dm,), "zeros"),
                (p + "attn.out.weight", (dm, dm), "he"),
                (p + "attn.out.bias", (dm,), "zeros"),
                (p + "ln1.weight", (dm,), "ones"),
                (p + "ln1.bias", (dm,), "zeros"),
                (p + "ffn1.weight", (ffn, dm), "he"),
                (p + "ffn1.bias", (ffn,), "zeros"),
                (p + "ffn2.weight", (dm, ffn), "he"),
                (p + "ffn2.bias", (dm,), "zeros"),
                (p + "ln2.weight", (dm,), "ones"),
                (p + "ln2.bias", (dm,), "zeros"),
            ]
        if spec.head == "ce":
            out.append(("vocab.weight", (d[4], dm), "he"))
            out.append(("vocab.bias", (d[4],), "zeros"))
    elif spec.kind == "reslstm":
        inp, hid, _, vocab = d
        for l in range(L):
            out.append((f"lstm{l}.weight_x", (4 * hid, inp if l == 0 else hid), "he"))
            out.append((f"lstm{l}.weight_h", (4 * hid, hid), "he"))
            out.append((f"lstm{l}.bias", (4 * hid,), "zeros"))
        if spec.head == "ce":
            out.append(("vocab.weight", (vocab, hid), "he"))
            out.append(("vocab.bias", (vocab,), "zeros"))
    else:
        raise ValueError(spec.kind)
    return out


def num_params(spec: StageSpec) -> int:
    return int(sum(int(np.prod(s)) for _, s, _ in param_layout(spec)))


# ----------------------------------------------------------------------------
# Workload table
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    stages: Tuple[StageSpec, ...]   # all simulated stages (one, or a whole pipeline)
    steps: int = 20                 # mini-batches per trajectory (one update each)


def _mlp3(batch=32, widths=(784, 256, 256, 10), lr=0.01, steps=20) -> Workload:
    n = len(widths) - 1
    stages = []
    for k in range(n):
        last = k == n - 1
        stages.append(StageSpec("fc", "fp32", "ce" if last else "none", k, n, batch, 1,
                                (widths[k], widths[k + 1], widths[k + 1]), lr, 0.9))
    return Workload("mlp3", tuple(stages), steps)


def _single(name, kind, dtype, head, k, N, batch, L, dims, lr, steps=20) -> Workload:
    return Workload(name, (StageSpec(kind, dtype, head, k, N, batch, L, tuple(dims), lr, 0.9),), steps)


def _pipeline(name, kind, N, batch, L, dims, lr, first_dims=None, last_head="none", last_dims=None,
              steps=20, zero_residual=False) -> Workload:
    """All N stages of one model, each a stage of the same kind and shape
    (stage 0 may differ in its input width, the last stage may carry the loss
    head); a last stage without a head takes the synthetic upstream gradient."""
    specs = []
    for k in range(N):
        d = first_dims if (k == 0 and first_dims) else dims
        head = "none"
        if k == N - 1:
            head = last_head
            d = last_dims or d
        specs.append(StageSpec(kind, "bf16", head, k, N, batch, L, tuple(d), lr, 0.9, zero_residual=zero_residual))
    return Workload(name, tuple(specs), steps)


# Full-size workloads: the five stage configurations of the benchmark.
# Learning rates follow Section 4.1 for VGG16 (2e-3), the Transformer (5e-5)
# and the residual LSTM (5e-3); momentum 0.9 for all. The bottleneck stage
# has no batch normalisation (only its convolutions are specified), and with
# ResNet-152's 2e-2 its first update moves W by 1.2x its norm and the second
# by 1e13x; 1e-5 moves it by 6e-4 of its norm per step, like the VGG stage.
WORKLOADS: Dict[str, Workload] = {
    "mlp3": _mlp3(),
    "vgg_conv": _single("vgg_conv", "conv3x3", "bf16", "none", 1, 4, 128, 4, (256, 512, 8, 8), 2e-3),
    "resnet_bottleneck": _single("resnet_bottleneck", "bottleneck", "bf16", "none", 2, 4, 64, 8,
                                 (1024, 256, 14, 14), 1e-5),
    "transformer_enc": _single("transformer_enc", "transformer", "bf16", "none", 1, 4, 64, 3,
                               (512, 8, 2048, 128), 5e-5),
    "reslstm": _single("reslstm", "reslstm", "bf16", "ce", 3, 4, 64, 2, (1024, 1024, 35, 10000), 5e-3),
}

# Reduced workloads of the same structure for parity runs the oracle finishes
# in seconds; sizes are chosen to cover several GEMM tiles plus ragged tails.
SMALL_WORKLOADS: Dict[str, Workload] = {
    "mlp3_small": _mlp3(batch=7, widths=(37, 50, 21, 10), lr=0.05),
    "vgg_conv_small": _single("vgg_conv_small", "conv3x3", "bf16", "none", 1, 4, 3, 3, (24, 40, 7, 9), 1e-3),
    # batch 32 at 7x9: K = 2016 positions, so the filter gradients split K
    "vgg_conv_mid": _single("vgg_conv_mid", "conv3x3", "bf16", "none", 1, 4, 32, 3, (40, 72, 7, 9), 1e-3),
    "resnet_bottleneck_small": _single("resnet_bottleneck_small", "bottleneck", "bf16", "none", 2, 4, 2, 2,
                                       (72, 24, 7, 5), 1e-3),
    "transformer_enc_small": _single("transformer_enc_small", "transformer", "bf16", "none", 1, 4, 3, 2,
                                     (64, 2, 136, 40), 2e-3),
    # sequence 128 and head dimension 64: the fused attention core
    "transformer_enc_mid": _single("transformer_enc_mid", "transformer", "bf16", "none", 1, 4, 2, 2,
                                   (128, 2, 256, 128), 2e-3),
    "reslstm_small": _single("reslstm_small", "reslstm", "bf16", "ce", 3, 4, 5, 2, (48, 48, 6, 104), 5e-2),
    # the same stage at an inner position (k = 1 of 4, three mini-batches in
    # flight): at the last stage a mini-batch's forward and backward are
    # adjacent and every staleness policy gives the same weights
    "reslstm_small_k1": _single("reslstm_small_k1", "reslstm", "bf16", "ce", 1, 4, 5, 2, (48, 48, 6, 104), 5e-2),
    # hidden size a multiple of 32 and batch <= 64: the fused recurrent steps
    "reslstm_mid": _single("reslstm_mid", "reslstm", "bf16", "ce", 3, 4, 24, 2, (96, 96, 7, 136), 5e-2),
}

# Whole 4-stage pipelines of the four bf16 models, every stage simulated in the
# one-forward-one-backward order on one GPU: the benchmark stage shapes
# chained, the last stage with its loss head (the conv models classify the
# average-pooled output into 10 classes, the transformer projects to its
# 32000-token vocabulary, the residual LSTM to 10000; the VGG stage 0 takes
# 256 channels to 512).
PIPELINE_WORKLOADS: Dict[str, Workload] = {
    "vgg_conv_pipe": _pipeline("vgg_conv_pipe", "conv3x3", 4, 128, 4, (512, 512, 8, 8), 2e-3,
                               first_dims=(256, 512, 8, 8), last_head="ce", last_dims=(512, 512, 8, 8, 10)),
    "resnet_bottleneck_pipe": _pipeline("resnet_bottleneck_pipe", "bottleneck", 4, 64, 8, (1024, 256, 14, 14), 1e-5,
                                        zero_residual=True, last_head="ce", last_dims=(1024, 256, 14, 14, 10)),
    "transformer_enc_pipe": _pipeline("transformer_enc_pipe", "transformer", 4, 64, 3, (512, 8, 2048, 128), 5e-5,
                                      last_head="ce", last_dims=(512, 8, 2048, 128, 32000)),
    "reslstm_pipe": _pipeline("reslstm_pipe", "reslstm", 4, 64, 2, (1024, 1024, 35, 10000), 5e-3, last_head="ce"),
}

SMALL_PIPELINE_WORKLOADS: Dict[str, Workload] = {
    "vgg_conv_small_pipe": _pipeline("vgg_conv_small_pipe", "conv3x3", 4, 3, 2, (40, 40, 7, 9), 1e-3,
                                     first_dims=(24, 40, 7, 9), last_head="ce", last_dims=(40, 40, 7, 9, 10)),
    "resnet_bottleneck_small_pipe": _pipeline("resnet_bottleneck_small_pipe", "bottleneck", 4, 2, 2,
                                              (72, 24, 7, 5), 1e-3, zero_residual=True, last_head="ce",
                                              last_dims=(72, 24, 7, 5, 10)),
    "transformer_enc_small_pipe": _pipeline("transformer_enc_small_pipe", "transformer", 4, 3, 2,
                                            (64, 2, 136, 40), 2e-3, last_head="ce",
                                            last_dims=(64, 2, 136, 40, 104)),
    "reslstm_small_pipe": _pipeline("reslstm_small_pipe", "reslstm", 4, 5, 2, (48, 48, 6, 104), 5e-2,
                                    last_head="ce"),
    # sequence 128, head dimension 64 (fused attention) and hidden 96, batch 24 (fused recurrent steps)
    "transformer_enc_mid_pipe": _pipeline("transformer_enc_mid_pipe", "transformer", 4, 2, 1, (128, 2, 256, 128),
                                          2e-3, last_head="ce", last_dims=(128, 2, 256, 128, 136)),
    "reslstm_mid_pipe": _pipeline("reslstm_mid_pipe", "reslstm", 4, 24, 1, (96, 96, 7, 136), 5e-2,
                                  last_head="ce"),
}

# The last transformer stage of the pipeline at full size: 3 encoder layers
# and the 32000-token projection with the mean token cross-entropy.
HEAD_WORKLOADS: Dict[str, Workload] = {
    "transformer_enc_last": _single("transformer_enc_last", "transformer", "bf16", "ce", 3, 4, 64, 3,
                                    (512, 8, 2048, 128, 32000), 5e-5),
}

ALL_WORKLOADS: Dict[str, Workload] = {**WORKLOADS, **SMALL_WORKLOADS, **PIPELINE_WORKLOADS,
                                      **SMALL_PIPELINE_WORKLOADS, **HEAD_WORKLOADS}


# ----------------------------------------------------------------------------
# Seeded draws
# ----------------------------------------------------------------------------

def to_bf16_values(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return them as float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def bf16_bits(x32: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bf16 numbers."""
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    if np.any(u & 0xFFFF):
        raise ValueError("values are not bf16-representable")
    return (u >> 16).astype(np.uint16)


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng([int(k) for k in key])


def initial_params(spec: StageSpec, seed: int = INIT_SEED) -> np.ndarray:
    """Flat float32 initial parameters W0 in the order of param_layout."""
    parts = []
    for i, (_, shape, init) in enumerate(param_layout(spec)):
        n = int(np.prod(shape))
        if init == "he":
            fan_in = int(np.prod(shape[1:]))
            r = _rng(seed, spec.stage_index, i)
            parts.append((r.standard_normal(n) * np.sqrt(2.0 / fan_in)).astype(np.float32))
        elif init == "zeros":
            parts.append(np.zeros(n, np.float32))
        elif init == "ones":
            parts.append(np.ones(n, np.float32))
        else:
            raise ValueError(init)
    return np.concatenate(parts).astype(np.float32)


def _input_scale(spec: StageSpec) -> float:
    return 0.02 if spec.kind == "transformer" else 1.0


def stage_input(spec: StageSpec, mb: int, seed: int = DATA_SEED) -> np.ndarray:
    """X for mini-batch mb at this stage (float32; bf16 values for bf16 stages)."""
    r = _rng(seed, spec.stage_index, mb, 0)
    x = (r.standard_normal(spec.input_shape()) * _input_scale(spec)).astype(np.float32)
    return to_bf16_values(x) if spec.dtype == "bf16" else x


def upstream_grad(spec: StageSpec, mb: int, seed: int = DATA_SEED) -> np.ndarray:
    """dL/dY for a stage without a loss head: N(0,1)/count, in the stage dtype."""
    r = _rng(seed, spec.stage_index, mb, 1)
    g = (r.standard_normal(spec.output_shape()) / spec.grad_count()).astype(np.float32)
    return to_bf16_values(g) if spec.dtype == "bf16" else g


def labels(spec: StageSpec, mb: int, seed: int = DATA_SEED) -> np.ndarray:
    """Integer targets, uniform in [0, classes), for a stage with a CE head."""
    r = _rng(seed, spec.stage_index, mb, 2)
    return r.integers(0, spec.num_classes(), size=spec.label_shape(), dtype=np.int64).astype(np.int32)
