"""Seeded generators for weights, batch-norm statistics and partition inputs.

Every draw comes from ``numpy.random.default_rng`` (PCG64) with a seed
sequence that names what is drawn, so a layer's parameters do not depend on
which other layers are generated: input = ``[seed, 0]``, layer i =
``[seed, 1, i]``.  Values are drawn in float64, rounded to float32 and then
to the storage dtype (round to nearest even), and handed to both consumers as
float32 arrays whose values are exactly representable in that dtype.

Initialisation (random, not trained weights):
  conv / fc weight  N(0, 2 / fan_in), fan_in = (c_in / groups) * k * k or in_features
  bias              N(0, 0.01^2)
  batch norm        gamma = layer.gamma, beta = 0, mean ~ N(0, 0.1^2), var ~ U(0.5, 1.5)
  image input       U[0, 1) per pixel, then (u - mean_c) / std_c with the
                    ImageNet channel statistics (an input transform, not a layer)
  feature input     ReLU(N(0, 1)) for a partition that starts mid-network
"""
from dataclasses import dataclass
from typing import Dict, Optional, Tuple

import numpy as np

from .zoo import Model, model as _model

DTYPES = ("f32", "f16", "bf16")
IMAGENET_MEAN = (0.485, 0.456, 0.406)
IMAGENET_STD = (0.229, 0.224, 0.225)
BN_EPS = 1e-5


def _f32_to_bf16_values(x32: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def to_dtype_values(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp64 -> fp32 -> dtype (RNE each step); returned as a float32 array."""
    x32 = np.asarray(x, dtype=np.float64).astype(np.float32)
    if dtype == "f32":
        return x32
    if dtype == "f16":
        return x32.astype(np.float16).astype(np.float32)
    if dtype == "bf16":
        return _f32_to_bf16_values(x32)
    raise ValueError(f"unknown dtype {dtype!r}")


def layer_params(L, index: int, seed: int, dtype: str) -> Dict[str, np.ndarray]:
    """Parameters of one fused layer (empty dict for parameter-free ops)."""
    if L.op not in ("conv", "fc", "fc_softmax"):
        return {}
    rng = np.random.default_rng([seed, 1, index])
    if L.op == "conv":
        shape = (L.c_out, L.c_in // L.groups, L.k, L.k)
        fan_in = (L.c_in // L.groups) * L.k * L.k
    else:
        shape = (L.c_out, L.c_in)
        fan_in = L.c_in
    p = {"weight": to_dtype_values(rng.standard_normal(shape) * np.sqrt(2.0 / fan_in), dtype)}
    if L.bias:
        p["bias"] = (rng.standard_normal(L.c_out) * 0.01).astype(np.float32)
    if L.bn:
        p["bn_gamma"] = np.full(L.c_out, L.gamma, dtype=np.float32)
        p["bn_beta"] = np.zeros(L.c_out, dtype=np.float32)
        p["bn_mean"] = (rng.standard_normal(L.c_out) * 0.1).astype(np.float32)
        p["bn_var"] = rng.uniform(0.5, 1.5, L.c_out).astype(np.float32)
    return p


def model_params(m: Model, seed: int, dtype: str, begin: int = 0,
                 end: Optional[int] = None) -> Dict[int, Dict[str, np.ndarray]]:
    end = len(m.layers) if end is None else end
    return {i: layer_params(m.layers[i], i, seed, dtype) for i in range(begin, end)}


def partition_input(shape_chw: Tuple[int, int, int], batch: int, seed: int,
                    dtype: str, kind: str) -> np.ndarray:
    """Batch of partition inputs, NCHW float32 holding dtype-representable values."""
    rng = np.random.default_rng([seed, 0])
    shape = (batch,) + tuple(shape_chw)
    if kind == "image":
        u = rng.random(shape)
        mean = np.asarray(IMAGENET_MEAN, dtype=np.float64).reshape(1, 3, 1, 1)
        std = np.asarray(IMAGENET_STD, dtype=np.float64).reshape(1, 3, 1, 1)
        x = (u - mean) / std
    elif kind == "relu_normal":
        x = np.maximum(rng.standard_normal(shape), 0.0)
    elif kind == "normal":
        x = rng.standard_normal(shape)
    else:
        raise ValueError(f"unknown input kind {kind!r}")
    return np.ascontiguousarray(to_dtype_values(x, dtype))


@dataclass(frozen=True)
class Workload:
    """One partition [begin, end) of a model run at a batch size."""
    name: str
    model: str
    begin: int
    end: int
    batch: int
    dtype: str
    seed: int
    in_chw: Tuple[int, int, int]     # partition input shape, stated, not derived
    input_kind: str
    last_gamma: float = 1.0          # batch-norm gamma of each residual block's last conv
    description: str = ""

    def build_model(self) -> Model:
        if self.last_gamma != 1.0:
            return _model(self.model, last_gamma=self.last_gamma)
        return _model(self.model)

    def params(self, m: Optional[Model] = None):
        m = m or self.build_model()
        return model_params(m, self.seed, self.dtype, self.begin, self.end)

    def input(self, batch: Optional[int] = None) -> np.ndarray:
        return partition_input(self.in_chw, batch or self.batch, self.seed,
                               self.dtype, self.input_kind)


WORKLOADS = {
    "resnet18_stem_layer1": Workload(
        "resnet18_stem_layer1", "resnet18", 0, 6, 1, "f32", 0, (3, 224, 224), "image",
        description="ResNet-18 stem conv7x7/s2 + BN + ReLU + maxpool3x3/s2 + two "
                    "3x3/64 basic blocks, batch 1, fp32"),
    "resnet50_layer4_head": Workload(
        "resnet50_layer4_head", "resnet50", 44, 56, 8, "bf16", 2, (1024, 14, 14),
        "relu_normal",
        description="ResNet-50 second partition: layer4 (3 bottlenecks) + global "
                    "avgpool + FC-1000 + softmax on 8x1024x14x14 bf16"),
    "resnet50_layer3_layer4_head": Workload(
        "resnet50_layer3_layer4_head", "resnet50", 25, 56, 8, "bf16", 2, (512, 28, 28),
        "relu_normal",
        description="ResNet-50 layer3 + layer4 + head on 8x512x28x28 bf16"),
    "vgg16": Workload(
        "vgg16", "vgg16", 0, 21, 16, "f16", 3, (3, 224, 224), "image",
        description="VGG-16 (13 conv3x3, 5 maxpool, 3 FC), batch 16, fp16"),
    "mobilenet_v2": Workload(
        "mobilenet_v2", "mobilenet_v2", 0, 54, 32, "bf16", 4, (3, 224, 224), "image",
        description="MobileNetV2 width 1.0, batch 32, bf16"),
    "resnet152": Workload(
        "resnet152", "resnet152", 0, 158, 16, "f16", 1, (3, 224, 224), "image",
        last_gamma=0.2,
        description="ResNet-152 full model, fp16, profiled at batches 1..64"),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]
