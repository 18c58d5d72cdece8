"""spectrain_stage_forward_backward against the separate calls.

In the one-forward-one-backward order of Section 3.1 every steady-state
step of stage k is a forward, then a backward, then the update; the
forward and the backward read weights of the same version. Two stages with
the same initial weights run the same task sequence, one through
spectrain_stage_forward + spectrain_stage_backward, one through the
combined call whose two passes run concurrently; every stage output, input
gradient, loss and the (W, v) after every update must be bitwise equal.
Also the refusals of the combined call (nothing enqueued, the stage still
usable).
"""
import dataclasses

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

CASES = {
    "mlp3_small.k0": synth.SMALL_WORKLOADS["mlp3_small"].stages[0],
    "mlp3_small.k1": synth.SMALL_WORKLOADS["mlp3_small"].stages[1],
    "vgg_conv_small": synth.SMALL_WORKLOADS["vgg_conv_small"].stages[0],
    "vgg_conv_mid": synth.SMALL_WORKLOADS["vgg_conv_mid"].stages[0],
    "resnet_bottleneck_small": synth.SMALL_WORKLOADS["resnet_bottleneck_small"].stages[0],
    "transformer_enc_small": synth.SMALL_WORKLOADS["transformer_enc_small"].stages[0],
    "transformer_enc_mid": synth.SMALL_WORKLOADS["transformer_enc_mid"].stages[0],
    "reslstm_small_k1": synth.SMALL_WORKLOADS["reslstm_small_k1"].stages[0],
    "reslstm_mid_k1": dataclasses.replace(synth.SMALL_WORKLOADS["reslstm_mid"].stages[0], stage_index=1),
    "resnet_bottleneck_small.stash": dataclasses.replace(
        synth.SMALL_WORKLOADS["resnet_bottleneck_small"].stages[0], policy="stash"),
    "vgg_conv_small.stash": dataclasses.replace(synth.SMALL_WORKLOADS["vgg_conv_small"].stages[0], policy="stash"),
    # the benchmark's bottleneck stage at full size
    "resnet_bottleneck": synth.WORKLOADS["resnet_bottleneck"].stages[0],
}


class _Driver:
    def __init__(self, spec, concurrent):
        from paper_1809_02839_amd import native
        self.spec, self.concurrent = spec, concurrent
        self.native = native
        self.st = native.Stage(native.desc_from_spec(spec), synth.initial_params(spec))
        self.sf, self.sb = native.policy_versions(spec.policy, spec.stage_index, spec.num_stages)
        self.st.predict(self.sf, 0)
        self.st.predict(self.sb, 1)
        self.ce = spec.head == "ce"
        self.keep = {}    # per mini-batch: x, y, labels, loss (alive until its backward)
        self.out = {}

    def _fwd_args(self, m):
        from paper_1809_02839_amd.pipeline import to_device, torch_dtype
        dev = torch.device("cuda")
        spec = self.spec
        x = to_device(synth.stage_input(spec, m), spec, dev)
        y = None if self.ce else torch.empty(spec.output_shape(), dtype=torch_dtype(spec), device=dev)
        lab = to_device(synth.labels(spec, m), spec, dev, integer=True) if self.ce else None
        loss = torch.zeros(1, device=dev) if self.ce else None
        self.keep[m] = (x, y, lab, loss)
        return x, y, lab, loss

    def _bwd_args(self, m):
        from paper_1809_02839_amd.pipeline import to_device, torch_dtype
        dev = torch.device("cuda")
        dy = None if self.ce else to_device(synth.upstream_grad(self.spec, m), self.spec, dev)
        dx = torch.empty(self.spec.input_shape(), dtype=torch_dtype(self.spec), device=dev)
        return dy, dx

    def forward(self, m):
        x, y, lab, loss = self._fwd_args(m)
        self.st.forward(m, x, y, lab, loss)

    def step(self, mf, mb):
        """forward(mf) (None: none) then backward(mb), then the update."""
        dy, dx = self._bwd_args(mb)
        if mf is None:
            self.st.backward(mb, dy, dx)
        else:
            x, y, lab, loss = self._fwd_args(mf)
            if self.concurrent:
                self.st.forward_backward(mf, x, y, mb, dy, dx, labels=lab, loss=loss)
            else:
                self.st.forward(mf, x, y, lab, loss)
                self.st.backward(mb, dy, dx)
        self.st.update(self.sf, self.sb)
        torch.cuda.synchronize()
        _, y, _, loss = self.keep.pop(mb)
        self.out[("dx", mb)] = dx.clone()
        self.out[("y", mb)] = loss.clone() if self.ce else y.clone()
        self.out[("state", mb)] = self.st.get_state()


@pytest.mark.parametrize("name", sorted(CASES))
def test_forward_backward_matches_separate_calls(name):
    spec = CASES[name]
    d = spec.num_stages - spec.stage_index
    assert d >= 2, "a concurrent forward needs a free stash slot"
    steps = 2 if name == "resnet_bottleneck" else 4
    ref, alt = _Driver(spec, False), _Driver(spec, True)
    try:
        for drv in (ref, alt):
            for m in range(d - 1):
                drv.forward(m)
            for m in range(steps):
                drv.step(m + d - 1, m)
        torch.cuda.synchronize()
        for key in ref.out:
            a, b = ref.out[key], alt.out[key]
            if key[0] == "state":
                assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), (name, key)
                assert np.any(a[1] != 0), (name, key)
            else:
                assert torch.equal(a, b), (name, key)
    finally:
        ref.st.destroy()
        alt.st.destroy()


def test_forward_backward_refusals():
    from paper_1809_02839_amd import native
    spec = synth.SMALL_WORKLOADS["resnet_bottleneck_small"].stages[0]     # k = 2 of 4: two slots
    drv = _Driver(spec, True)
    try:
        st = drv.st
        x0, y0, _, _ = drv._fwd_args(0)
        st.forward(0, x0, y0)
        x1, y1, _, _ = drv._fwd_args(1)
        dy, dx = drv._bwd_args(0)
        with pytest.raises(native.SpecTrainError) as e:    # the same mini-batch
            st.forward_backward(0, x1, y1, 0, dy, dx)
        assert e.value.code == native.ESTATE
        with pytest.raises(native.SpecTrainError) as e:    # backward of a mini-batch not in flight
            st.forward_backward(1, x1, y1, 5, dy, dx)
        assert e.value.code == native.ESTATE
        with pytest.raises(native.SpecTrainError) as e:    # forward of a mini-batch already in flight
            st.forward_backward(0, x1, y1, 0, dy, dx)
        assert e.value.code == native.ESTATE
        with pytest.raises(native.SpecTrainError) as e:    # no upstream gradient without a loss head
            st.forward_backward(1, x1, y1, 0, None, dx)
        assert e.value.code == native.EINVAL
        # nothing was enqueued or recorded: the regular order still works
        drv.step(1, 0)                                     # slots: 1
        x2, y2, _, _ = drv._fwd_args(2)
        st.forward_backward(2, x2, y2, 1, *drv._bwd_args(1))   # slots: 2
        x3, y3, _, _ = drv._fwd_args(3)
        with pytest.raises(native.SpecTrainError) as e:    # the gradient still waits for its update
            st.forward_backward(3, x3, y3, 2, *drv._bwd_args(2))
        assert e.value.code == native.ESTATE
        st.update(drv.sf, drv.sb)
        st.forward(3, x3, y3)                              # slots: 2, 3
        x4, y4, _, _ = drv._fwd_args(4)
        with pytest.raises(native.SpecTrainError) as e:    # no free stash slot
            st.forward_backward(4, x4, y4, 2, *drv._bwd_args(2))
        assert e.value.code == native.ESTATE
        drv.step(None, 2)
        drv.step(4, 3)
        torch.cuda.synchronize()
    finally:
        drv.st.destroy()


def test_last_stage_has_no_free_slot():
    from paper_1809_02839_amd import native
    spec = synth.SMALL_WORKLOADS["reslstm_small"].stages[0]     # k = N - 1: one slot
    drv = _Driver(spec, True)
    try:
        drv.forward(0)
        x1, y1, lab, loss = drv._fwd_args(1)
        dy, dx = drv._bwd_args(0)
        with pytest.raises(native.SpecTrainError) as e:
            drv.st.forward_backward(1, x1, y1, 0, dy, dx, labels=lab, loss=loss)
        assert e.value.code == native.ESTATE
        drv.step(None, 0)     # the last stage's own order: forward, backward, update
        torch.cuda.synchronize()
    finally:
        drv.st.destroy()


def test_serial_profile_mode_is_bitwise_and_times_every_launch():
    """Profile mode 2 issues every launch of the combined call on the stage
    stream, one at a time (the durations are the launches' own): results stay
    bitwise equal, every kernel family of both passes is timed, and modes
    other than 0, 1, 2 are refused."""
    from paper_1809_02839_amd import native
    spec = CASES["resnet_bottleneck_small"]
    d = spec.num_stages - spec.stage_index
    ref, alt = _Driver(spec, True), _Driver(spec, True)
    try:
        assert native.lib().spectrain_stage_profile(alt.st.h, 3) == native.EINVAL
        alt.st.profile(True, serial=True)
        for drv in (ref, alt):
            for m in range(d - 1):
                drv.forward(m)
            for m in range(3):
                drv.step(m + d - 1, m)
        prof = alt.st.profile_read()
        alt.st.profile(False)
        for key in ref.out:
            a, b = ref.out[key], alt.out[key]
            if key[0] == "state":
                assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]), key
            else:
                assert torch.equal(a, b), key
        names = " ".join(prof)
        # forward (conv3x3 gather), data gradients, weight gradients, the update
        for fam in ("gemm_bf16_kernel<1, 0,", "gemm_bf16_kernel<0, 3,", "gemm_bf16_kernel<3, 3,", "fused_update"):
            assert fam in names, (fam, sorted(prof))
        assert all(v["launches"] > 0 and v["ms_total"] > 0 for v in prof.values())
    finally:
        ref.st.destroy()
        alt.st.destroy()
