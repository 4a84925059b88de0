"""Host-side checks of the seeded workloads: architectures against published
parameter counts and layer maps, generator determinism and representability."""
import hashlib

import numpy as np
import pytest

import workloads as W


@pytest.mark.parametrize("name,count", [
    # torchvision parameter counts of the published architectures
    ("resnet18", 11_689_512), ("resnet50", 25_557_032), ("resnet152", 60_192_808),
    ("vgg16", 138_357_544), ("mobilenet_v2", 3_504_872)])
def test_param_counts(name, count):
    assert W.param_count(W.model(name)) == count


def test_layer_maps():
    r50 = W.model("resnet50").layers
    assert len(r50) == 56
    assert r50[44].name == "layer4.0.conv1" and r50[44].c_in == 1024
    assert r50[25].name == "layer3.0.conv1" and r50[25].c_in == 512
    assert r50[54].op == "gap" and r50[55].op == "fc_softmax"
    r152 = W.model("resnet152").layers
    assert len(r152) == 158 and r152[37].name == "layer3.0.conv1" and r152[146].name == "layer4.0.conv1"
    assert len(W.model("resnet18").layers) == 23
    vgg = W.model("vgg16").layers
    assert len(vgg) == 21 and sum(L.op == "conv" for L in vgg) == 13
    mb = W.model("mobilenet_v2").layers
    assert len(mb) == 54 and sum(L.op == "conv" and L.groups > 1 for L in mb) == 17
    assert sum(L.res_src >= 0 for L in mb) == 10


def test_every_workload_range_reads_only_its_input():
    """Each stated partition is a valid split: its layers read only layers of
    the range or the output of layer begin-1 (-1 names the model input)."""
    for wl in W.WORKLOADS.values():
        m = wl.build_model()
        for i in range(wl.begin, wl.end):
            L = m.layers[i]
            assert L.src >= wl.begin - 1, (wl.name, i)
            assert L.res_src == -1 or L.res_src >= wl.begin - 1, (wl.name, i)


def test_generator_determinism_and_independence():
    m = W.model("resnet50")
    a = W.model_params(m, 2, "bf16", 44, 48)
    b = W.model_params(m, 2, "bf16", 40, 48)
    for i in range(44, 48):
        for k in a[i]:
            np.testing.assert_array_equal(a[i][k], b[i][k])
    c = W.model_params(m, 3, "bf16", 44, 45)
    assert not np.array_equal(a[44]["weight"], c[44]["weight"])
    x1 = W.partition_input((3, 8, 8), 4, 0, "f16", "image")
    x2 = W.partition_input((3, 8, 8), 2, 0, "f16", "image")
    np.testing.assert_array_equal(x1[:2], x2)     # image i is the same at any batch size
    h = hashlib.sha256(x1.tobytes()).hexdigest()
    assert h == hashlib.sha256(W.partition_input((3, 8, 8), 4, 0, "f16", "image").tobytes()).hexdigest()


@pytest.mark.parametrize("dt,np_t", [("f16", np.float16), ("f32", np.float32)])
def test_values_are_representable(dt, np_t):
    x = W.partition_input((3, 16, 16), 2, 5, dt, "image")
    np.testing.assert_array_equal(x.astype(np_t).astype(np.float32), x)


def test_bf16_values_have_zero_low_bits():
    x = W.partition_input((4, 8, 8), 2, 5, "bf16", "relu_normal")
    assert (x.view(np.uint32) & 0xFFFF == 0).all()
    assert (x >= 0).all()
    w = W.layer_params(W.model("resnet50").layers[44], 44, 2, "bf16")["weight"]
    assert (w.view(np.uint32) & 0xFFFF == 0).all()


def test_init_statistics():
    L = W.model("vgg16").layers[10]   # conv 256 -> 512 3x3
    p = W.layer_params(L, 10, 3, "f32")
    std = np.sqrt(2.0 / (L.c_in * 9))
    assert abs(p["weight"].std() / std - 1) < 0.01
    assert abs(p["bias"].std() / 0.01 - 1) < 0.1
    q = W.layer_params(W.model("resnet152", last_gamma=0.2).layers[5], 5, 1, "f16")
    assert np.all(q["bn_gamma"] == np.float32(0.2))
    assert (q["bn_var"] >= 0.5).all() and (q["bn_var"] <= 1.5).all()
