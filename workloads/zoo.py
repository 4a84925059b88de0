"""CNN architectures as lists of fused layers.

A "layer" here is the unit the paper's planner reasons about: a node whose
latency is profiled per batch size and whose output feature map is the only
tensor that crosses a partition boundary placed after it (paper, Table of
MILP inputs: L_kbi and S_i; a partition spans layers i to j exclusive).  A
convolution carries its batch norm, activation and optional residual add, so a
split between two fused layers never changes the arithmetic.

Layer fields:
  op       'conv' | 'maxpool' | 'gap' (global average pool) | 'fc' | 'fc_softmax'
  src      index of the producing layer, -1 for the model input
  res_src  index of the layer whose output is added before the activation, or -1
  c_in, c_out, k, stride, pad, groups   (for 'fc': c_in = in_features)
  act      'none' | 'relu' | 'relu6'
  bn       conv followed by batch norm
  bias     layer has a bias vector
  gamma    value of the batch-norm scale used when generating parameters

Architectures follow the torchvision definitions (the paper serves
TorchVision/OpenMMLab models, Evaluation: Methodology): ResNet v1.5 with the
stride on the 3x3 convolution and the downsample projection placed before the
block's last convolution; VGG-16 configuration D with its adaptive average
pool omitted (identity at 224x224) and dropout as identity; MobileNetV2 width
1.0 with t=1 in its first inverted-residual block.
"""
from dataclasses import dataclass, field
from typing import List


@dataclass
class Layer:
    name: str
    op: str
    src: int
    c_in: int
    c_out: int
    k: int = 1
    stride: int = 1
    pad: int = 0
    groups: int = 1
    act: str = "none"
    res_src: int = -1
    bn: bool = False
    bias: bool = False
    gamma: float = 1.0


@dataclass
class Model:
    name: str
    in_c: int
    in_h: int
    in_w: int
    layers: List[Layer] = field(default_factory=list)

    def add(self, **kw) -> int:
        self.layers.append(Layer(**kw))
        return len(self.layers) - 1


def _stem(m: Model) -> int:
    x = m.add(name="conv1", op="conv", src=-1, c_in=3, c_out=64, k=7, stride=2,
              pad=3, act="relu", bn=True)
    return m.add(name="maxpool", op="maxpool", src=x, c_in=64, c_out=64, k=3,
                 stride=2, pad=1)


def _resnet(name: str, block: str, depths, last_gamma: float = 1.0) -> Model:
    m = Model(name, 3, 224, 224)
    x = _stem(m)
    cin = 64
    for si, (nb, width) in enumerate(zip(depths, (64, 128, 256, 512))):
        for bi in range(nb):
            s = 2 if (si > 0 and bi == 0) else 1
            tag = f"layer{si + 1}.{bi}"
            if block == "basic":
                cout = width
                a = m.add(name=f"{tag}.conv1", op="conv", src=x, c_in=cin,
                          c_out=width, k=3, stride=s, pad=1, act="relu", bn=True)
                ds = -1
                if s != 1 or cin != cout:
                    ds = m.add(name=f"{tag}.downsample", op="conv", src=x,
                               c_in=cin, c_out=cout, k=1, stride=s, bn=True)
                x = m.add(name=f"{tag}.conv2", op="conv", src=a, c_in=width,
                          c_out=cout, k=3, pad=1, act="relu", bn=True,
                          res_src=ds if ds >= 0 else x, gamma=last_gamma)
            else:
                cout = 4 * width
                r = m.add(name=f"{tag}.conv1", op="conv", src=x, c_in=cin,
                          c_out=width, k=1, act="relu", bn=True)
                c = m.add(name=f"{tag}.conv2", op="conv", src=r, c_in=width,
                          c_out=width, k=3, stride=s, pad=1, act="relu", bn=True)
                ds = -1
                if s != 1 or cin != cout:
                    ds = m.add(name=f"{tag}.downsample", op="conv", src=x,
                               c_in=cin, c_out=cout, k=1, stride=s, bn=True)
                x = m.add(name=f"{tag}.conv3", op="conv", src=c, c_in=width,
                          c_out=cout, k=1, act="relu", bn=True,
                          res_src=ds if ds >= 0 else x, gamma=last_gamma)
            cin = cout
    g = m.add(name="avgpool", op="gap", src=x, c_in=cin, c_out=cin)
    m.add(name="fc", op="fc_softmax", src=g, c_in=cin, c_out=1000, bias=True)
    return m


def resnet18() -> Model:
    return _resnet("resnet18", "basic", (2, 2, 2, 2))


def resnet50() -> Model:
    return _resnet("resnet50", "bottleneck", (3, 4, 6, 3))


def resnet152(last_gamma: float = 1.0) -> Model:
    return _resnet("resnet152", "bottleneck", (3, 8, 36, 3), last_gamma)


def vgg16() -> Model:
    m = Model("vgg16", 3, 224, 224)
    x, cin, n = -1, 3, 0
    for stage, (reps, width) in enumerate(((2, 64), (2, 128), (3, 256),
                                           (3, 512), (3, 512))):
        for r in range(reps):
            n += 1
            x = m.add(name=f"conv{stage + 1}_{r + 1}", op="conv", src=x,
                      c_in=cin, c_out=width, k=3, pad=1, act="relu", bias=True)
            cin = width
        x = m.add(name=f"pool{stage + 1}", op="maxpool", src=x, c_in=cin,
                  c_out=cin, k=2, stride=2)
    # classifier input: 512 channels x 7 x 7 flattened in (c, h, w) order
    x = m.add(name="fc6", op="fc", src=x, c_in=512 * 7 * 7, c_out=4096,
              act="relu", bias=True)
    x = m.add(name="fc7", op="fc", src=x, c_in=4096, c_out=4096, act="relu",
              bias=True)
    m.add(name="fc8", op="fc_softmax", src=x, c_in=4096, c_out=1000, bias=True)
    return m


def mobilenet_v2() -> Model:
    m = Model("mobilenet_v2", 3, 224, 224)
    x = m.add(name="features.0", op="conv", src=-1, c_in=3, c_out=32, k=3,
              stride=2, pad=1, act="relu6", bn=True)
    cin, blk = 32, 0
    for t, c, n, s in ((1, 16, 1, 1), (6, 24, 2, 2), (6, 32, 3, 2),
                       (6, 64, 4, 2), (6, 96, 3, 1), (6, 160, 3, 2),
                       (6, 320, 1, 1)):
        for i in range(n):
            blk += 1
            stride = s if i == 0 else 1
            hid = cin * t
            inp = x
            h = x
            if t != 1:
                h = m.add(name=f"features.{blk}.expand", op="conv", src=h,
                          c_in=cin, c_out=hid, k=1, act="relu6", bn=True)
            h = m.add(name=f"features.{blk}.dw", op="conv", src=h, c_in=hid,
                      c_out=hid, k=3, stride=stride, pad=1, groups=hid,
                      act="relu6", bn=True)
            use_res = stride == 1 and cin == c
            x = m.add(name=f"features.{blk}.project", op="conv", src=h,
                      c_in=hid, c_out=c, k=1, bn=True,
                      res_src=inp if use_res else -1)
            cin = c
    x = m.add(name="features.18", op="conv", src=x, c_in=cin, c_out=1280, k=1,
              act="relu6", bn=True)
    g = m.add(name="avgpool", op="gap", src=x, c_in=1280, c_out=1280)
    m.add(name="classifier", op="fc_softmax", src=g, c_in=1280, c_out=1000,
          bias=True)
    return m


MODELS = {
    "resnet18": resnet18,
    "resnet50": resnet50,
    "resnet152": resnet152,
    "vgg16": vgg16,
    "mobilenet_v2": mobilenet_v2,
}


def model(name: str, **kw) -> Model:
    return MODELS[name](**kw)


def param_count(m: Model) -> int:
    """Trainable parameters as torchvision counts them (BN scale and shift
    included, running statistics excluded)."""
    total = 0
    for L in m.layers:
        if L.op == "conv":
            total += L.c_out * (L.c_in // L.groups) * L.k * L.k
        elif L.op in ("fc", "fc_softmax"):
            total += L.c_out * L.c_in
        else:
            continue
        if L.bias:
            total += L.c_out
        if L.bn:
            total += 2 * L.c_out
    return total
