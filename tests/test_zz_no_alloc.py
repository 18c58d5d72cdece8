"""The allocation-free backward (spectrain_stage_backward_noalloc) against
the regular backward: two stages with the same weights run the same
forward, one backward through each entry point, and the same update; dX and
the updated W and v must be bitwise equal. Each stage's weight gradients
split K, so their partial planes go through the per-device scratch array.
Two calls in a row, the second on a smaller input, check that what the
first left in the scratch array does not leak into the second."""
import dataclasses

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

# bf16 stages whose backward GEMMs split K: a two-layer FC stage (weight
# gradients 512 x 256 x batch, 8 slices at batch 6144, 4 at 3072) and a
# small bottleneck stage (weight gradients over 2352 or 1568 pixels, 3 or 2
# slices)
FC_BIG = synth.StageSpec("fc", "bf16", "none", 1, 3, 6144, 2, (256, 256, 512), 0.01, 0.9)
FC_SMALL = dataclasses.replace(FC_BIG, batch=3072)
BNECK_BIG = synth.StageSpec("bottleneck", "bf16", "none", 2, 4, 12, 2, (256, 64, 14, 14), 1e-3, 0.9)
BNECK_SMALL = dataclasses.replace(BNECK_BIG, batch=8)


def _run_pair(spec, steps=3):
    from paper_1809_02839_amd import native
    from paper_1809_02839_amd.pipeline import to_device, torch_dtype
    dev = torch.device("cuda")
    W0 = synth.initial_params(spec)
    desc = native.desc_from_spec(spec)
    ref, alt = native.Stage(desc, W0), native.Stage(desc, W0)
    sf, sb = native.policy_versions("spectrain", spec.stage_index, spec.num_stages)
    try:
        for st in (ref, alt):
            st.predict(sf, 0)
            st.predict(sb, 1)
        for m in range(steps):
            x = to_device(synth.stage_input(spec, m), spec, dev)
            dy = to_device(synth.upstream_grad(spec, m), spec, dev)
            ys = [torch.empty(spec.output_shape(), dtype=torch_dtype(spec), device=dev) for _ in range(2)]
            dxs = [torch.empty(spec.input_shape(), dtype=torch_dtype(spec), device=dev) for _ in range(2)]
            ref.forward(m, x, ys[0])
            alt.forward(m, x, ys[1])
            ref.backward(m, dy, dxs[0])
            alt.backward_noalloc(m, dy, dxs[1])
            ref.update(sf, sb)
            alt.update(sf, sb)
            torch.cuda.synchronize()
            assert torch.equal(dxs[0], dxs[1]), (spec, m, "dx")
            (Wr, vr), (Wa, va) = ref.get_state(), alt.get_state()
            assert np.array_equal(Wr, Wa) and np.array_equal(vr, va), (spec, m, "state")
            assert np.any(vr != 0)
    finally:
        ref.destroy()
        alt.destroy()


@pytest.mark.parametrize("big,small", [(FC_BIG, FC_SMALL), (BNECK_BIG, BNECK_SMALL)], ids=["fc", "bottleneck"])
def test_noalloc_backward_matches_backward(big, small):
    print(f"[noalloc] {big.kind} batch {big.batch} then {small.batch}", flush=True)
    _run_pair(big)
    _run_pair(small)


def test_noalloc_backward_state_rules():
    from paper_1809_02839_amd import native
    spec = FC_SMALL
    st = native.Stage(native.desc_from_spec(spec), synth.initial_params(spec))
    try:
        dy = torch.zeros(spec.output_shape(), dtype=torch.bfloat16, device="cuda")
        with pytest.raises(native.SpecTrainError) as e:
            st.backward_noalloc(5, dy, None)    # no forward of mini-batch 5 in flight
        assert e.value.code == native.ESTATE
    finally:
        st.destroy()
