"""GPU checks of the stage ABI around the method's edges: the call-order
rules (ESTATE / EINVAL on a live stage, which stays usable afterwards), the
degenerate momentum gamma = 1 (v stays 0, so W and both predicted slots stay
W0 bitwise), the non-finite flag of the fused update, and batch-1 stages of
every kind against the oracle."""
import numpy as np
import pytest

import synth
from stepwise import run_stepwise

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _fc_stage(k=1, N=3, batch=4, momentum=0.9, dtype="fp32"):
    from paper_1809_02839_amd import native
    spec = synth.StageSpec("fc", dtype, "none", k, N, batch, 1, (16, 8, 8), 0.01, momentum)
    st = native.Stage(native.desc_from_spec(spec), synth.initial_params(spec), torch.cuda.current_stream())
    dt = torch.float32 if dtype == "fp32" else torch.bfloat16
    x = torch.randn(batch, 16, device="cuda").to(dt)
    dy = (torch.randn(batch, 8, device="cuda") * 0.1).to(dt)
    ys = [torch.empty(batch, 8, device="cuda", dtype=dt) for _ in range(N + 1)]
    dx = torch.empty(batch, 16, device="cuda", dtype=dt)
    return spec, st, x, dy, ys, dx


def _expect(code, fn):
    from paper_1809_02839_amd import native
    with pytest.raises(native.SpecTrainError) as e:
        fn()
    assert e.value.code == code, e.value


def test_call_order_errors_leave_the_stage_usable():
    from paper_1809_02839_amd import native
    spec, st, x, dy, ys, dx = _fc_stage(k=1, N=3)           # N - k = 2 mini-batches in flight
    _expect(native.ESTATE, lambda: st.backward(0, dy, dx))   # nothing in flight
    _expect(native.ESTATE, lambda: st.update(0, 0))          # no gradient yet
    _expect(native.EINVAL, lambda: st.predict(-1, 0))
    _expect(native.EINVAL, lambda: st.predict(0, 2))
    _expect(native.EINVAL, lambda: st.forward(0, None, ys[0]))
    st.forward(0, x, ys[0])
    _expect(native.ESTATE, lambda: st.forward(0, x, ys[1]))  # same mini-batch twice
    st.forward(1, x, ys[1])
    _expect(native.ESTATE, lambda: st.forward(2, x, ys[2]))  # ring full
    W, v = st.get_state()
    _expect(native.ESTATE, lambda: st.set_state(W, v))       # mini-batches in flight
    st.backward(0, dy, dx)
    _expect(native.ESTATE, lambda: st.backward(1, dy, dx))   # previous gradient not applied
    st.update(1, 0)
    st.backward(1, dy, dx)
    st.update(1, 0)
    st.set_state(W, v)                                      # empty ring: allowed
    st.forward(2, x, ys[2])
    st.backward(2, dy, dx)
    st.update(1, 0)
    torch.cuda.synchronize()
    W2, v2 = st.get_state()
    assert np.all(np.isfinite(W2)) and not np.array_equal(W2, W)
    st.destroy()


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_gamma_one_freezes_the_weights(dtype):
    """gamma = 1: v = gamma v + (1 - gamma) g stays 0, so every update leaves
    W at W0 and both predicted slots at W0 in the operand format."""
    spec, st, x, dy, ys, dx = _fc_stage(k=0, N=2, momentum=1.0, dtype=dtype)
    W0 = synth.initial_params(spec)
    for m in range(2):
        st.forward(m, x, ys[m])
    for m in range(6):
        st.backward(m, dy, dx)
        st.update(1, 0)
        st.forward(m + 2, x, ys[(m + 2) % len(ys)])
    torch.cuda.synchronize()
    W, v = st.get_state()
    assert np.array_equal(W, W0) and not np.any(v)
    rnd = synth.to_bf16_values if dtype == "bf16" else (lambda a: a)
    for slot in (0, 1):
        assert np.array_equal(st.get_predicted(slot), rnd(W0))
    st.destroy()


def test_non_finite_update_is_reported():
    """A smoothed gradient of +inf makes the update produce non-finite W and v;
    once the update has run, the next call on the stage returns ENONFINITE."""
    from paper_1809_02839_amd import native
    spec, st, x, dy, ys, dx = _fc_stage(k=0, N=1)
    W0 = synth.initial_params(spec)
    v = np.zeros_like(W0)
    v[3] = np.inf
    st.set_state(W0, v)
    st.forward(0, x, ys[0])
    st.backward(0, dy, dx)
    st.update(0, 0)
    torch.cuda.synchronize()
    _expect(native.ENONFINITE, lambda: st.predict(0, 0))
    st.destroy()


# Batch 1 of every stage kind (the smallest ragged tile of every GEMM, one
# image, one sequence), stage k = 1 of 3 or the last stage with its head.
EDGE = {
    "fc": synth.StageSpec("fc", "bf16", "ce", 2, 3, 1, 2, (24, 16, 16), 0.05, 0.9),
    "conv3x3": synth.StageSpec("conv3x3", "bf16", "ce", 2, 3, 1, 2, (16, 24, 3, 5, 6), 0.01, 0.9),
    "bottleneck": synth.StageSpec("bottleneck", "bf16", "none", 1, 3, 1, 2, (32, 16, 5, 3), 0.01, 0.9),
    "transformer": synth.StageSpec("transformer", "bf16", "ce", 2, 3, 1, 1, (64, 2, 64, 8, 16), 0.01, 0.9),
    "reslstm": synth.StageSpec("reslstm", "bf16", "ce", 2, 3, 1, 2, (32, 32, 3, 24), 0.05, 0.9),
}


@pytest.mark.parametrize("kind", list(EDGE))
def test_batch_one_stage_stepwise(kind):
    wl = synth.Workload(f"{kind}_batch1", (EDGE[kind],), 8)
    print(f"[stepwise] {wl.name}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch)
    print(f"[stepwise] {wl.name}: {worst.report()}", flush=True)


def test_ksliced_conv_forward_ragged_edges_stepwise():
    # conv3x3 forward with 14490 x 200 outputs (B = 230 at 7 x 9): 114 x 2 tiles
    # of 128 x 128, one block on most CUs, so both layers' forwards run on 8-wave
    # blocks whose wave pairs split each K step, with a ragged last row tile
    # (14490 = 113 * 128 + 26) and a ragged last column tile (200 = 128 + 72);
    # the first layer (64 input channels) on the per-step tap gather, the
    # second (200) on the per-vector one. The second layer's data gradient
    # (into 200 channels, against the transposed filter) runs the same 8-wave
    # blocks; the first layer's (into 64 channels) 4-wave 128 x 128 tiles.
    spec = synth.StageSpec("conv3x3", "bf16", "none", 1, 4, 230, 2, (64, 200, 7, 9), 1e-3, 0.9)
    wl = synth.Workload("conv_ksliced_ragged", (spec,), 4)
    print(f"[stepwise] {wl.name}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch)
    print(f"[stepwise] {wl.name}: {worst.report()}", flush=True)


def test_narrow_tile_ragged_edges_stepwise():
    # 25000 x 200 outputs: the 128 x 128 tiles (196 x 2) cannot give every CU two
    # blocks but 128 x 64 tiles (196 x 4) can, so the forward GEMMs and the
    # second layer's data gradient run on 128 x 64 tiles with no K split, with
    # a ragged last row tile (25000 = 195 * 128 + 40) and a ragged last column
    # tile (200 = 3 * 64 + 8), on both a row-major and a transposed B operand
    spec = synth.StageSpec("fc", "bf16", "none", 1, 3, 25000, 2, (64, 200, 200), 0.01, 0.9)
    wl = synth.Workload("fc_narrow_ragged", (spec,), 4)
    print(f"[stepwise] {wl.name}", flush=True)
    worst = run_stepwise(wl, wl.steps, torch)
    print(f"[stepwise] {wl.name}: {worst.report()}", flush=True)


def test_bf16_rounding_through_predict():
    """The bf16 copies are rounded to nearest, ties to even, on every float32
    input class: ties going down and up, neighbours of ties, overflow of the
    largest float to infinity, subnormals (ties included) and signed zeros,
    plus random bit patterns. With v = 0 the prediction of Eq. 4 is W itself,
    so the predicted slot holds exactly the rounded W; the expected bits come
    from the integer definition (u + 0x7fff + bit 16 of u) >> 16."""
    from paper_1809_02839_amd import native
    spec = synth.StageSpec("fc", "bf16", "none", 0, 2, 4, 1, (256, 256, 256), 0.01, 0.9)
    st = native.Stage(native.desc_from_spec(spec), synth.initial_params(spec), torch.cuda.current_stream())
    try:
        n = st.n_params
        special = np.array([0x3f808000, 0x3f818000, 0x3f808001, 0x3f807fff, 0xbf818000, 0x7f7fffff, 0xff7fffff,
                            0x00000001, 0x00008000, 0x00018000, 0x807fffff, 0x80000000, 0x00000000, 0x7f7f8000,
                            0x477fe000, 0x477ff000], dtype=np.uint32)
        rng = np.random.default_rng(7)
        u = rng.integers(0, 2**32, size=n, dtype=np.uint64).astype(np.uint32)
        u = np.where((u & 0x7f800000) == 0x7f800000, u ^ 0x40000000, u).astype(np.uint32)   # finite inputs only
        u[:len(special)] = special
        W = u.view(np.float32)
        st.set_state(W, np.zeros(n, np.float32))
        st.predict(1, 0)
        got = st.get_predicted(0).view(np.uint32) >> 16
        want = ((u.astype(np.uint64) + 0x7fff + ((u >> 16) & 1)) >> 16).astype(np.uint32)
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, [(hex(u[i]), hex(got[i]), hex(want[i])) for i in bad[:8]]
        assert want[5] == 0x7f80 and want[7] == 0 and want[9] == 0x0002 and want[11] == 0x8000
    finally:
        st.destroy()
