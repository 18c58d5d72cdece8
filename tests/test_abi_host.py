"""Host-side checks of the C ABI library (no GPU needed): it loads, exports
every entry point the header declares, computes Eq. 5/6, rejects bad
descriptors before touching the device, and the pipeline driver's task order
is a valid one-forward-one-backward order."""
import ctypes
import os
import re

import numpy as np
import pytest

import synth
from oracle import method, schedule
from paper_1809_02839_amd import native, pipeline

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "spectrain.h")).read()
    return sorted(set(re.findall(r"\b(spectrain_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = native.lib()
    names = declared_functions()
    assert len(names) == len(native.EXPORTED) >= 15
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(names) == sorted(native.EXPORTED)


@pytest.mark.parametrize("N", range(1, 9))
def test_version_difference_matches_oracle(N):
    for k in range(N):
        assert native.version_difference(k, N, True) == method.version_difference(k, N, True)
        assert native.version_difference(k, N, False) == method.version_difference(k, N, False)
    assert native.version_difference(N, N, True) == -1
    assert native.version_difference(-1, N, False) == -1
    assert native.version_difference(0, 0, True) == -1


def _create(desc, n=None, W=None):
    lib = native.lib()
    h = ctypes.c_void_p()
    W = np.zeros(1 if n is None else n, np.float32) if W is None else W
    rc = lib.spectrain_stage_create(ctypes.byref(desc), W.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
                                    W.size if n is None else n, None, ctypes.byref(h))
    return rc, h, lib.spectrain_last_error().decode()


@pytest.mark.parametrize("change,needle", [
    (dict(stage_index=4), "stage_index"),
    (dict(stage_index=-1), "stage_index"),
    (dict(num_stages=0), "stage_index"),
    (dict(batch=0), "batch"),
    (dict(lr=0.0), "lr"),
    (dict(lr=float("nan")), "lr"),
    (dict(momentum=0.0), "momentum"),
    (dict(momentum=1.5), "momentum"),
    (dict(kind=9), "kind"),
    (dict(dtype=0), "bf16 only"),
    (dict(head=1), "dims[4]"),
    (dict(head=1, dims=(256, 512, 8, 8, 7)), "classes must be even"),
    (dict(dims=(250, 512, 8, 8)), "multiple of 8"),
    (dict(weight_policy=2), "weight_policy"),
    (dict(weight_policy=-1), "weight_policy"),
])
def test_bad_descriptor_is_rejected_before_any_device_work(change, needle):
    spec = synth.WORKLOADS["vgg_conv"].stages[0]
    fields = dict(kind=spec.kind, dtype=spec.dtype, head=spec.head, stage_index=spec.stage_index,
                  num_stages=spec.num_stages, batch=spec.batch, num_layers=spec.num_layers, dims=spec.dims,
                  lr=spec.lr, momentum=spec.momentum)
    fields.update(change)
    desc = native.make_desc(**fields)
    rc, h, msg = _create(desc, synth.num_params(spec))
    assert rc == native.EINVAL and not h.value, msg
    assert needle in msg


@pytest.mark.parametrize("dims,needle", [((512, 8, 2048, 128), "dims[4]"), ((512, 8, 2048, 128, 1001), "vocab")])
def test_transformer_ce_head_needs_a_vocabulary(dims, needle):
    spec = synth.WORKLOADS["transformer_enc"].stages[0]
    desc = native.make_desc(spec.kind, spec.dtype, "ce", 3, 4, spec.batch, spec.num_layers, dims, spec.lr,
                            spec.momentum)
    rc, h, msg = _create(desc, 1)
    assert rc == native.EINVAL and not h.value, msg
    assert needle in msg


def test_wrong_param_count_and_version_rejected():
    spec = synth.WORKLOADS["vgg_conv"].stages[0]
    desc = native.desc_from_spec(spec)
    rc, h, msg = _create(desc, synth.num_params(spec) - 1)
    assert rc == native.EINVAL and "n_params" in msg
    desc.abi_version = 99
    rc, h, msg = _create(desc, synth.num_params(spec))
    assert rc == native.EINVAL and "abi_version" in msg


def test_null_handle_calls_fail_cleanly():
    lib = native.lib()
    assert lib.spectrain_stage_destroy(None) == native.EINVAL
    assert lib.spectrain_stage_predict(None, 0, 0) == native.EINVAL
    assert lib.spectrain_stage_update(None, 0, 0) == native.EINVAL
    assert b"NULL" in lib.spectrain_last_error()


@pytest.mark.parametrize("N", range(1, 9))
def test_driver_stage_order_equals_oracle_order(N):
    M = 2 * N + 5
    for k in range(N):
        assert pipeline.stage_task_order(k, N, M) == schedule.stage_tasks(k, N, M)


@pytest.mark.parametrize("N", range(1, 9))
def test_driver_pipeline_order_respects_dependencies(N):
    M = 2 * N + 3
    seq = pipeline.pipeline_task_order(N, M)
    assert len(seq) == 2 * N * M
    pos = {t: i for i, t in enumerate(seq)}
    for k in range(N):
        assert [(kind, m) for kk, kind, m in seq if kk == k] == schedule.stage_tasks(k, N, M)
        for m in range(M):
            if k > 0:
                assert pos[(k - 1, "F", m)] < pos[(k, "F", m)]
            if k < N - 1:
                assert pos[(k + 1, "B", m)] < pos[(k, "B", m)]
            else:
                assert pos[(k, "F", m)] < pos[(k, "B", m)]


def test_binding_refuses_host_strided_and_mistyped_tensors():
    # the library reads raw device pointers; the binding stops these before any call
    torch = pytest.importorskip("torch")
    from paper_1809_02839_amd import native

    class FakeCuda:
        is_cuda = True

        def __init__(self, dtype, contiguous=True):
            self.dtype, self._c = dtype, contiguous

        def is_contiguous(self):
            return self._c

        def data_ptr(self):
            return 4096

    with pytest.raises(ValueError, match="GPU tensor"):
        native._dptr(torch.zeros(4), "torch.float32", "x")
    with pytest.raises(ValueError, match="contiguous"):
        native._dptr(FakeCuda(torch.float32, contiguous=False), "torch.float32", "x")
    with pytest.raises(ValueError, match="torch.bfloat16"):
        native._dptr(FakeCuda(torch.float32), "torch.bfloat16", "x")
    assert native._dptr(FakeCuda(torch.int32), "torch.int32", "labels").value == 4096
    assert native._dptr(None, "torch.float32") is None
