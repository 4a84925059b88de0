"""Kernel parity: each kernel family, tile configuration, split-K path and
dtype against the CPU oracle on small seeded layers that span several tiles
and ragged tails.  Runs through the C ABI on an MI355X."""
import numpy as np
import pytest

import oracle
import workloads as W
from workloads.zoo import Layer, Model

from gpu_util import gpu_forward, rel_inf, argmax_rows

pytestmark = pytest.mark.gpu

# one rounding to the storage dtype on each side plus fp32-vs-fp64 sums
LAYER_TOL = {"f32": 1e-5, "f16": 2.0 ** -9, "bf16": 2.0 ** -7}
DTYPES = ["f32", "f16", "bf16"]


def make(in_chw, specs):
    m = Model("t", *in_chw)
    for s in specs:
        m.add(**s)
    return m


def check(m, dtype, batch, begin=0, end=None, seed=0, kind="normal", in_chw=None, tol=None,
          exact=False, tuning=None):
    from paper_2507_18748_amd import Partition
    end = len(m.layers) if end is None else end
    P = W.model_params(m, seed, dtype, begin, end)
    in_chw = in_chw or (m.in_c, m.in_h, m.in_w)
    x = W.partition_input(in_chw, batch, seed, dtype, kind)
    print(f"[layer-parity] {[L.name for L in m.layers[begin:end]]} dtype={dtype} batch={batch}",
          flush=True)
    ref = oracle.forward(m.layers, P, begin, end, x, dtype)
    with Partition(m.layers, P, (m.in_c, m.in_h, m.in_w), begin, end, dtype, max_batch=batch,
                   tuning=tuning) as part:
        got = gpu_forward(part, x)
    got = got.reshape(ref.shape)
    if exact:
        np.testing.assert_array_equal(got, ref)
        return 0.0
    e = rel_inf(got, ref)
    assert e <= (tol or LAYER_TOL[dtype]), f"rel_inf {e:.3e}"
    if m.layers[end - 1].op == "fc_softmax":
        assert (argmax_rows(got) == argmax_rows(ref)).all()
    return e


def conv(name, src, ci, co, k=1, s=1, p=0, g=1, act="relu", res=-1, bn=True, bias=False):
    return dict(name=name, op="conv", src=src, c_in=ci, c_out=co, k=k, stride=s, pad=p,
                groups=g, act=act, res_src=res, bn=bn, bias=bias)


# Streaming 1x1 kernel, forced on small layers: (C, Co, H, W, batch,
# residual, activation).  Ragged channel slices (Co not a multiple of the
# slice), C below one k-step, ragged 16-pixel groups.
PW_CASES = [
    (8, 4, 5, 7, 3, False, "relu"),
    (16, 96, 9, 11, 4, False, "relu6"),
    (24, 144, 7, 7, 5, False, "relu6"),
    (32, 16, 13, 5, 2, False, "none"),
    (32, 192, 6, 6, 3, True, "relu"),
    (24, 36, 5, 5, 2, True, "none"),
    (16, 200, 4, 4, 1, False, "relu"),
    (32, 388, 3, 9, 3, False, "relu"),
    (96, 24, 9, 7, 3, False, "none"),       # several k-steps, at most 32 outputs
    (144, 24, 6, 7, 2, True, "none"),
    (160, 32, 5, 5, 2, False, "relu6"),
    (40, 20, 7, 3, 2, True, "relu"),
]


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("ci,co,h,w,batch,res,act", PW_CASES)
def test_pointwise_kernel(dtype, ci, co, h, w, batch, res, act):
    from paper_2507_18748_amd import Partition
    tuning = {"gemm_plan": (17,)}
    if res:   # residual source: a 3x3 convolution of the same input
        specs = [conv("r", -1, ci, co, 3, 1, 1), conv("c", -1, ci, co, act=act, res=0)]
    else:
        specs = [conv("c", -1, ci, co, act=act)]
    m = make((ci, h, w), specs)
    with Partition(m.layers, W.model_params(m, 0, dtype), (ci, h, w), 0, len(specs), dtype,
                   max_batch=batch, tuning=tuning) as part:
        li = part.layer_info(len(specs) - 1, batch)
        assert li["kernel"].startswith("pw_conv<") and li["forced"] == 1
        assert part.info["tuned"] == 1
    check(m, dtype, batch, tuning=tuning)


# Stems: (C, Co, k, stride, pad, H, W, batch) of images with C <= 4 channels.
STEM_CASES = [
    (3, 64, 3, 1, 1, 19, 17, 2),    # VGG conv1_1
    (3, 32, 3, 2, 1, 23, 21, 3),    # MobileNetV2 stem
    (3, 64, 7, 2, 3, 29, 27, 2),    # ResNet stem
    (3, 36, 5, 1, 2, 11, 13, 2),    # ragged channel slice, 25 taps
    (1, 16, 3, 1, 0, 9, 8, 3),      # one channel, no padding
    (3, 100, 7, 2, 3, 15, 15, 1),   # two channel slices
]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("ci,co,k,st,pd,h,w,batch", STEM_CASES)
def test_stem_kernel(dtype, ci, co, k, st, pd, h, w, batch):
    from paper_2507_18748_amd import Partition
    m = make((ci, h, w), [conv("s", -1, ci, co, k, st, pd)])
    with Partition(m.layers, W.model_params(m, 0, dtype), (ci, h, w), 0, 1, dtype,
                   max_batch=batch) as part:
        assert part.layer_info(0, batch)["kernel"].startswith("stem_conv<")
    check(m, dtype, batch, kind="image" if ci == 3 else "normal")


def test_stem_kernel_four_channels():
    """A 4-channel 16-bit image (below one 8-element vector) takes the stem
    kernel too."""
    m = make((4, 12, 10), [conv("s", -1, 4, 32, 3, 1, 1)])
    check(m, "bf16", 2)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("grid", [1, 5])
def test_stem_window_grid_stride(dtype, grid):
    """A 7x7 stride-2 stem (ragged: 23 x 20 outputs, tiles of 4 rows x 16
    columns) launched on 1 or 5 blocks, so that every block walks several
    tiles and loads the next tile's input window while it computes the
    current one: the oracle's result, and the default launch's bits."""
    from paper_2507_18748_amd import Partition
    m = make((3, 45, 39), [conv("s", -1, 3, 64, 7, 2, 3)])
    check(m, dtype, 2, kind="image", tuning={"stream_grid": grid})
    P = W.model_params(m, 0, dtype)
    x = W.partition_input((3, 45, 39), 2, 3, dtype, "image")
    outs = []
    for tuning in (None, {"stream_grid": grid}):
        with Partition(m.layers, P, (3, 45, 39), 0, 1, dtype, max_batch=2,
                       tuning=tuning) as part:
            assert part.layer_info(0, 2)["kernel"].startswith("stem_conv<")
            outs.append(gpu_forward(part, x))
    np.testing.assert_array_equal(outs[0], outs[1])


@pytest.mark.parametrize("grid", ["1", "8"])
def test_pointwise_grid_stride_matches_default(grid):
    """A pointwise launch capped at 1 or 8 blocks (every wave walks many
    16-pixel groups with loads in flight ahead) gives the default's bits."""
    from paper_2507_18748_amd import Partition
    m = make((24, 37, 29), [conv("c", -1, 24, 144, act="relu6")])
    P = W.model_params(m, 0, "bf16")
    x = W.partition_input((24, 37, 29), 3, 5, "bf16", "normal")
    outs = []
    for g in (None, grid):
        tuning = {"gemm_plan": (17,)}
        if g:
            tuning["stream_grid"] = int(g)
        with Partition(m.layers, P, (24, 37, 29), 0, 1, "bf16", max_batch=3,
                       tuning=tuning) as part:
            assert part.layer_info(0, 3)["kernel"].startswith("pw_conv<")
            outs.append(gpu_forward(part, x))
    np.testing.assert_array_equal(outs[0], outs[1])


@pytest.mark.parametrize("dtype", DTYPES)
def test_conv3x3_split_k(dtype):
    # M = 2*15*15 = 450 (ragged), Co = 128: 64x64 tiles with split-K
    check(make((64, 15, 15), [conv("c", -1, 64, 128, 3, 1, 1)]), dtype, 2)


@pytest.mark.parametrize("dtype", DTYPES)
def test_conv3x3_stride2_ragged(dtype):
    check(make((32, 17, 17), [conv("c", -1, 32, 64, 3, 2, 1)]), dtype, 3)


@pytest.mark.parametrize("dtype", DTYPES)
def test_conv1x1_k_tail(dtype):
    # C = 24 is not a multiple of the K stage: masked tail; Co = 40 ragged tile
    check(make((24, 10, 10), [conv("c", -1, 24, 40, act="none")]), dtype, 2)


@pytest.mark.parametrize("dtype", DTYPES)
def test_conv1x1_stride2_downsample(dtype):
    check(make((64, 14, 14), [conv("c", -1, 64, 128, 1, 2, 0, act="none")]), dtype, 2)


@pytest.mark.parametrize("dtype", DTYPES)
def test_residual_from_partition_input(dtype):
    m = make((16, 9, 9), [conv("c0", -1, 16, 32, 3, 1, 1),
                          conv("c1", 0, 32, 16, 1),
                          conv("c2", 1, 16, 32, 3, 1, 1, res=0)])
    check(m, dtype, 3, begin=1, end=3, in_chw=(32, 9, 9))


@pytest.mark.parametrize("dtype", DTYPES)
def test_stem7x7_gather(dtype):
    check(make((3, 32, 32), [conv("stem", -1, 3, 64, 7, 2, 3)]), dtype, 2, kind="image")


@pytest.mark.parametrize("dtype", DTYPES)
def test_stem3x3_relu6_gather(dtype):
    check(make((3, 33, 33), [conv("stem", -1, 3, 32, 3, 2, 1, act="relu6")]), dtype, 2,
          kind="image")


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("stride", [1, 2])
@pytest.mark.parametrize("chw", [(96, 13, 13), (24, 9, 11), (8, 5, 6), (40, 2, 3), (16, 3, 101)])
def test_depthwise3x3(dtype, stride, chw):
    """Ragged output rows (the last pixel group of a row is partial), one and
    several channel vectors, maps narrower than a pixel group."""
    c = chw[0]
    check(make(chw, [conv("dw", -1, c, c, 3, stride, 1, g=c, act="relu6")]), dtype, 2)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("k,s,p,hw", [(3, 2, 1, 15), (2, 2, 0, 12), (3, 2, 1, 112),
                                      (2, 2, 0, 13), (3, 1, 1, 9), (3, 2, 0, 14)])
def test_maxpool_bit_exact(dtype, k, s, p, hw):
    m = make((64, hw, hw), [dict(name="pool", op="maxpool", src=-1, c_in=64, c_out=64, k=k,
                                 stride=s, pad=p)])
    check(m, dtype, 2, exact=True)


@pytest.mark.parametrize("dtype", DTYPES)
def test_global_avgpool(dtype):
    check(make((256, 7, 7), [dict(name="gap", op="gap", src=-1, c_in=256, c_out=256)]),
          dtype, 3, kind="relu_normal")


@pytest.mark.parametrize("dtype", DTYPES)
def test_gap_fc_softmax(dtype):
    m = make((512, 7, 7), [dict(name="gap", op="gap", src=-1, c_in=512, c_out=512),
                           dict(name="fc", op="fc_softmax", src=0, c_in=512, c_out=1000,
                                bias=True)])
    check(m, dtype, 5, kind="relu_normal", tol={"f32": 1e-5, "f16": 1e-2, "bf16": 2e-2}[dtype])


@pytest.mark.parametrize("dtype", DTYPES)
def test_fc_on_feature_map(dtype):
    # FC over a 7x7x64 map flattened in (c, h, w) order, then FC + softmax
    m = make((64, 7, 7), [dict(name="fc6", op="fc", src=-1, c_in=64 * 49, c_out=256,
                               act="relu", bias=True),
                          dict(name="fc8", op="fc_softmax", src=0, c_in=256, c_out=100,
                               bias=True)])
    check(m, dtype, 3, kind="relu_normal", tol={"f32": 1e-5, "f16": 1e-2, "bf16": 2e-2}[dtype])


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_conv_large_tiles(dtype):
    # M = 8*64*64 = 32768, Co = 128: the 128x128 tile configuration
    check(make((32, 64, 64), [conv("c", -1, 32, 128, 3, 1, 1)]), dtype, 8)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_fc_large_k_small_batch(dtype):
    # M = batch = 1: 64x16 tiles, deep split-K over K = 4096
    m = make((4096, 1, 1), [dict(name="fc", op="fc", src=-1, c_in=4096, c_out=1000,
                                 act="relu", bias=True)])
    check(m, dtype, 1)


@pytest.mark.parametrize("dtype", ["f16", "bf16", "f32"])
def test_conv_lds_64x64(dtype):
    # M = 10*32*32 = 10240, Co = 64: the LDS-staged 64x64 configuration
    check(make((64, 32, 32), [conv("c", -1, 64, 64, 3, 1, 1)]), dtype, 10)


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_conv_lds_64x128(dtype):
    # M = 5*64*64 = 20480, Co = 64: the 64 x 128 configuration
    check(make((64, 64, 64), [conv("c", -1, 64, 64, 3, 1, 1)]), dtype, 5)


@pytest.mark.parametrize("dtype", DTYPES)
def test_skinny_32x32(dtype):
    # M = 4*16*16 = 1024, Co = 256: 32x32 skinny tiles
    check(make((64, 16, 16), [conv("c", -1, 64, 256, act="none")]), dtype, 4)


@pytest.mark.parametrize("dtype", DTYPES)
def test_skinny_32x16(dtype):
    # the ResNet-50 layer4 3x3 shape: M = 8*7*7 = 392, Co = 512, K = 4608
    check(make((512, 7, 7), [conv("c", -1, 512, 512, 3, 1, 1)]), dtype, 8)


@pytest.mark.parametrize("dtype", DTYPES)
def test_skinny_16x32(dtype):
    # a 4096-wide FC at batch 2 (the VGG classifier shape)
    m = make((512, 1, 1), [dict(name="fc", op="fc", src=-1, c_in=512, c_out=4096,
                                act="relu", bias=True)])
    check(m, dtype, 2, kind="relu_normal")


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
@pytest.mark.parametrize("ci,k,s", [(1024, 1, 1), (256, 3, 1), (256, 3, 2)])
def test_planned_skinny_16x16_on_small_16bit_grids(dtype, ci, k, s):
    """ResNet-152's layer3 shapes at batch 1 (196 output pixels, 256 output
    channels, K of 1024 or 2304): the planner picks the 16x16 skinny tile on
    four waves for 16-bit types, against the oracle."""
    from paper_2507_18748_amd import Partition
    h = 14 * s
    m = make((ci, h, h), [conv("c", -1, ci, 256, k, s, k // 2, act="relu")])
    with Partition(m.layers, W.model_params(m, 0, dtype, 0, 1), (ci, h, h), 0, 1, dtype,
                   max_batch=2) as part:
        assert "conv_gemm_skinny<" in part.layer_info(0, 1)["kernel"]
        assert "16x16" in part.layer_info(0, 1)["kernel"]
        assert "conv_gemm_skinny<" not in part.layer_info(0, 2)["kernel"]   # 392 pixels
    check(m, dtype, 1)


FORCED = [  # (configuration id, waves, splits): every kernel variant the planner can emit
    ("0,0,1", "conv_gemm<", "128x128"), ("0,0,4", "conv_gemm<", "128x128"),
    ("1,0,1", "conv_gemm<", "64x64"), ("1,0,3", "conv_gemm<", "64x64"),
    ("2,0,1", "conv_gemm<", "64x128"), ("2,0,2", "conv_gemm<", "64x128"),
    ("3,4", "conv_gemm_skinny<", "32x32"), ("3,8", "conv_gemm_skinny<", "32x32"),
    ("4,4", "conv_gemm_skinny<", "32x16"), ("4,8", "conv_gemm_skinny<", "32x16"),
    ("5,4", "conv_gemm_skinny<", "16x32"), ("5,8", "conv_gemm_skinny<", "16x32"),
    ("6,4", "conv_gemm_skinny<", "16x16"), ("6,8", "conv_gemm_skinny<", "16x16"),
    ("6,16", "conv_gemm_skinny<", "16x16"),
    ("7,0,1", "conv_gemm<", "128x128,kv8,8w"), ("7,0,2", "conv_gemm<", "128x128,kv8,8w"),
    ("8,0,1", "conv_gemm<", "128x64"), ("8,0,3", "conv_gemm<", "128x64"),
    ("9,0,1", "conv_gemm<", "64x64,kv8,dma2"), ("9,0,3", "conv_gemm<", "64x64,kv8,dma2"),
    ("10,0,1", "conv_gemm<", "64x64,kv8,dma3"), ("10,0,2", "conv_gemm<", "64x64,kv8,dma3"),
    ("11,0,1", "conv_gemm<", "128x128,kv8,8w,dma2"), ("11,0,4", "conv_gemm<", "128x128,kv8,8w,dma2"),
    ("12,0,1", "conv_gemm<", "128x128,kv8,8w,dma3"), ("12,0,2", "conv_gemm<", "128x128,kv8,8w,dma3"),
    ("13,0,1", "conv_gemm<", "64x64,kv8,8w,dma2"), ("13,0,3", "conv_gemm<", "64x64,kv8,8w,dma2"),
    ("14,0,1", "conv_gemm<", "64x64,kv8,8w,dma3"), ("14,0,2", "conv_gemm<", "64x64,kv8,8w,dma3"),
    ("15,0,1", "conv_gemm<", "64x64,kv8,8w,dma4"), ("15,0,3", "conv_gemm<", "64x64,kv8,8w,dma4"),
    ("16,0,1", "conv_gemm<", "64x64,kv8,8w,dma6"), ("16,0,2", "conv_gemm<", "64x64,kv8,8w,dma6"),
    ("19,0,1", "conv_gemm<", "64x128,kv8,8w,dma2"), ("19,0,2", "conv_gemm<", "64x128,kv8,8w,dma2"),
    ("20,0,1", "conv_gemm<", "64x256,kv8,8w,dma2"), ("20,0,3", "conv_gemm<", "64x256,kv8,8w,dma2"),
    # 32x32x16 matrix instructions, 64x64 per wave (16-bit types only)
    ("21,0,1", "conv_gemm_mx<", "128x128,4w,dma2"), ("21,0,3", "conv_gemm_mx<", "128x128,4w,dma2"),
    ("22,0,1", "conv_gemm_mx<", "128x128,4w,dma3"), ("22,0,2", "conv_gemm_mx<", "128x128,4w,dma3"),
    ("23,0,1", "conv_gemm_mx<", "128x128,4w,dma4"), ("23,0,3", "conv_gemm_mx<", "128x128,4w,dma4"),
    ("24,0,1", "conv_gemm_mx<", "256x128,8w,dma2"), ("24,0,2", "conv_gemm_mx<", "256x128,8w,dma2"),
    ("25,0,1", "conv_gemm_mx<", "128x256,8w,dma2"), ("25,0,3", "conv_gemm_mx<", "128x256,8w,dma2"),
    ("26,0,1", "conv_gemm_mx<", "256x128,8w,dma3"), ("26,0,2", "conv_gemm_mx<", "256x128,8w,dma3"),
    ("27,0,1", "conv_gemm_mx<", "128x128,8w,dma2"), ("27,0,3", "conv_gemm_mx<", "128x128,8w,dma2"),
    ("28,0,1", "conv_gemm_mx<", "128x128,8w,dma3"), ("28,0,2", "conv_gemm_mx<", "128x128,8w,dma3"),
]
FORCED += [
    ("29,0,1", "conv_gemm<", "64x64,kv8,2w,dma2"), ("29,0,3", "conv_gemm<", "64x64,kv8,2w,dma2"),
    ("30,0,1", "conv_gemm<", "64x64,kv8,1w,dma2"), ("30,0,2", "conv_gemm<", "64x64,kv8,1w,dma2"),
    ("31,0,1", "conv_gemm<", "64x64,kv8,2w,dma3"), ("31,0,3", "conv_gemm<", "64x64,kv8,2w,dma3"),
    ("32,0,1", "conv_gemm<", "128x128,kv8,8w,dma4"), ("32,0,2", "conv_gemm<", "128x128,kv8,8w,dma4"),
]
MX_FORCED = [f for f in FORCED if f[1] == "conv_gemm_mx<"]
FORCED_SHAPES = {  # ragged M and Co, padded 3x3 taps, a 1x1 with a K tail, an FC + softmax
    "3x3": ((64, 13, 13), [conv("c", -1, 64, 100, 3, 1, 1)], 3, "normal"),
    "1x1": ((24, 9, 9), [conv("c", -1, 24, 36, act="relu6")], 2, "normal"),
    "fc": ((96, 3, 3), [dict(name="fc", op="fc_softmax", src=-1, c_in=96 * 9, c_out=200,
                             bias=True)], 5, "relu_normal"),
    # 3-channel stem: channels padded to one vector, per-vector taps
    "stem": ((3, 23, 23), [conv("c", -1, 3, 64, 7, 2, 3)], 2, "image"),
    # several tiles of the large configurations in both dimensions, ragged
    "3x3w": ((64, 21, 23), [conv("c", -1, 64, 300, 3, 1, 1, act="relu")], 2, "relu_normal"),
}


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("shape", list(FORCED_SHAPES))
@pytest.mark.parametrize("plan,family,tile", FORCED)
def test_forced_gemm_configuration(plan, family, tile, shape, dtype):
    """Every tile configuration, wave count and split count against the oracle
    (forced through the planner override)."""
    from paper_2507_18748_amd import Partition
    in_chw, specs, batch, kind = FORCED_SHAPES[shape]
    if shape == "stem" and family == "conv_gemm_skinny<":
        pytest.skip("the skinny kernel has no per-vector-tap gather")
    if family == "conv_gemm_mx<" and dtype == "f32":
        pytest.skip("32x32x16 matrix instructions take 16-bit operands only")
    tuning = {"gemm_plan": tuple(int(v) for v in plan.split(","))}
    m = make(in_chw, specs)
    with Partition(m.layers, W.model_params(m, 0, dtype), in_chw, 0, 1, dtype,
                   max_batch=batch, tuning=tuning) as part:
        k = part.layer_info(0, batch)["kernel"]
    assert k.startswith(family) and tile in k, (plan, k)
    tol = {"f32": 1e-5, "bf16": 2.0 ** -7}[dtype] if shape != "fc" else 2e-2
    check(m, dtype, batch, kind=kind, tol=tol, tuning=tuning)


# A residual stage's first bottleneck: conv1 and the downsample projection read
# the stage input and go out as one launch when their plans match.
def _bottleneck(ci, mid, co, hw, s):
    return make((ci, hw, hw), [
        conv("conv1", -1, ci, mid),
        conv("conv2", 0, mid, mid, 3, s, 1),
        conv("down", -1, ci, co, 1, s, 0, act="none"),
        conv("conv3", 1, mid, co, act="relu", res=2),
        dict(name="pool", op="gap", src=3, c_in=co, c_out=co),
    ])


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("ci,mid,co,hw,s,batch", [
    (256, 128, 512, 14, 2, 4),     # ResNet-50 layer2-like stage entry, two tiles of each
    (64, 64, 256, 9, 1, 3),        # stride 1 (ResNet layer1), ragged tiles
    (512, 256, 1024, 7, 2, 8),
])
def test_paired_downsample_launch(dtype, ci, mid, co, hw, s, batch):
    """conv1 and the downsample run as one launch (the layer info says so),
    match the oracle, and equal the per-layer launch sequence of a timed run
    bit for bit, directly and from a captured graph replayed twice."""
    import torch
    from paper_2507_18748_amd import Partition
    from gpu_util import upload_nhwc, empty_out
    m = _bottleneck(ci, mid, co, hw, s)
    P = W.model_params(m, 3, dtype)
    x = W.partition_input((ci, hw, hw), batch, 3, dtype, "relu_normal")
    print(f"[paired] {ci},{mid},{co} hw={hw} s={s} dtype={dtype} batch={batch}", flush=True)
    ref = oracle.forward(m.layers, P, 0, len(m.layers), x, dtype)
    with Partition(m.layers, P, (ci, hw, hw), 0, len(m.layers), dtype, max_batch=batch) as part:
        k0 = part.layer_info(0, batch)["kernel"]
        k2 = part.layer_info(2, batch)["kernel"]
        paired = "paired=2" in k0
        assert paired == ("paired=0" in k2), (k0, k2)
        xd = upload_nhwc(x, dtype)
        outs = []
        for mode in ("timed", "direct", "graph"):
            out = empty_out(part, batch)
            out.fill_(float("nan"))
            st = torch.cuda.current_stream().cuda_stream
            if mode == "timed":
                part.timing_setup(batch, xd.data_ptr(), out.data_ptr())
                part.run_timed(st)
                part.timing_read()
            elif mode == "direct":
                part.run(batch, xd.data_ptr(), out.data_ptr(), st)
            else:
                part.capture(batch, xd.data_ptr(), out.data_ptr())
                for _ in range(2):
                    part.run(batch, xd.data_ptr(), out.data_ptr(), st)
                    torch.cuda.synchronize()
            torch.cuda.synchronize()
            outs.append(out.float().cpu().numpy().copy())
    for o in outs[1:]:
        np.testing.assert_array_equal(o, outs[0])
    got = outs[0].reshape(ref.shape)
    assert rel_inf(got, ref) <= LAYER_TOL[dtype]
    if dtype != "f32":
        assert paired, (k0, k2)


def test_no_pairing_when_the_later_layer_adds_the_earlier_one():
    """y = conv_b(x) + conv_a(x): conv_b reads conv_a's output as its residual,
    so the two must not run as one launch at conv_a's position; the layer info
    shows no pairing and the output matches the oracle."""
    from paper_2507_18748_amd import Partition
    ci, co, hw, batch = 128, 256, 7, 4
    m = make((ci, hw, hw), [
        conv("a", -1, ci, co, act="none"),
        conv("b", -1, ci, co, act="relu", res=0),
        dict(name="pool", op="gap", src=1, c_in=co, c_out=co),
    ])
    P = W.model_params(m, 1, "bf16")
    with Partition(m.layers, P, (ci, hw, hw), 0, 3, "bf16", max_batch=batch) as part:
        for i in (0, 1):
            assert "paired=" not in part.layer_info(i, batch)["kernel"]
    check(m, "bf16", batch, seed=1, kind="relu_normal")


@pytest.mark.parametrize("shape", ["3x3", "3x3w", "stem"])
@pytest.mark.parametrize("plan,family,tile", MX_FORCED)
def test_forced_mx_configuration_f16(plan, family, tile, shape):
    """The 32x32x16 configurations in fp16 (a separate instruction from bf16)."""
    from paper_2507_18748_amd import Partition
    in_chw, specs, batch, kind = FORCED_SHAPES[shape]
    tuning = {"gemm_plan": tuple(int(v) for v in plan.split(","))}
    m = make(in_chw, specs)
    with Partition(m.layers, W.model_params(m, 0, "f16"), in_chw, 0, 1, "f16",
                   max_batch=batch, tuning=tuning) as part:
        k = part.layer_info(0, batch)["kernel"]
    assert k.startswith(family) and tile in k, (plan, k)
    check(m, "f16", batch, kind=kind, tuning=tuning)
