"""Host-side checks of the experiment inputs: the learnable teacher labels
have each head's label shape, stay inside its classes (the transformer's
inside the first 1024 tokens), and are deterministic per mini-batch."""
import numpy as np
import pytest

import synth


@pytest.mark.parametrize("name,kind", [("mlp3_small", "fc"), ("vgg_conv_small_pipe", "conv3x3"),
                                       ("transformer_enc_small_pipe", "transformer")])
def test_teacher_labels_shape_range_and_determinism(name, kind):
    from paper_1809_02839_amd import experiments
    wl = synth.ALL_WORKLOADS[name]
    last = wl.stages[-1]
    assert last.kind == kind and last.head == "ce"
    f, g = experiments.teacher_labels(wl), experiments.teacher_labels(wl)
    for m in range(3):
        lab = f(last, m)
        assert lab.shape == last.label_shape() and lab.dtype == np.int32
        assert lab.min() >= 0 and lab.max() < min(last.num_classes(), 1024 if kind == "transformer" else 10 ** 9)
        assert np.array_equal(lab, g(last, m))          # a fresh teacher gives the same labels
        assert f(last, m) is lab                         # cached per mini-batch
    assert not np.array_equal(f(last, 0), f(last, 1))

