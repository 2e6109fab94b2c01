"""Per-routine parity on the GPU: every routine (algorithm x layout x routine
parameter) of every layer type, in every dtype, against the float64 oracle
on the same seeded inputs, through the C ABI.  Shapes span several tiles
and ragged tails (channels not multiples of 8, odd spatial sizes)."""

import numpy as np
import pytest

from oracle import numeric as O
from tests.gpu_util import TOL, err, from_dev, oracle_layer, run_routine, single_layer_graph, to_dev
from workloads import random_tensor, to_f64

pytestmark = pytest.mark.gpu

DTYPES = ["f32", "f16", "bf16"]

CONV_CASES = [
    # (N, C, H, W, K, R, stride, pad, act)
    (2, 24, 13, 11, 40, 3, 1, 1, "relu"),     # ragged M and N tiles, Winograd odd sizes
    (1, 64, 16, 16, 72, 3, 2, 1, "relu6"),    # stride 2
    (2, 40, 9, 9, 136, 1, 1, 0, "none"),      # pointwise, N > 128
    (1, 3, 37, 37, 16, 7, 2, 3, "relu"),      # stem-like: C = 3
    (3, 16, 8, 8, 10, 3, 1, 1, "none"),       # K = 10 (not a multiple of 8)
    (1, 130, 7, 7, 24, 3, 1, 1, "relu"),      # C = 130: partial last channel chunk
    # channel counts that are multiples of the LDS-DMA reduction tile
    (2, 64, 15, 13, 200, 3, 1, 1, "relu"),    # 3x3/1, ragged M (390) and N (200)
    (1, 128, 9, 9, 64, 1, 1, 0, "none"),      # pointwise, one N tile
    (2, 32, 11, 11, 48, 3, 1, 1, "relu"),     # C = 32: only the BK = 32 tiles apply
    (3, 64, 5, 5, 40, 3, 1, 1, "relu6"),      # several whole images per patch tile
    (5, 32, 7, 7, 24, 3, 1, 1, "none"),       # image groups with a ragged last group
    (2, 64, 14, 14, 96, 3, 1, 1, "relu"),     # 14 x 14: two row tiles per image, ragged channel tile
    (3, 32, 28, 28, 40, 3, 1, 1, "relu6"),    # 28 x 28: four row tiles per image, K = 40
    (3, 1024, 7, 9, 200, 1, 1, 0, "relu"),    # long reduction (128-channel steps), ragged M and N
    (4, 512, 15, 17, 200, 1, 1, 0, "relu6"),  # C = 512: streaming kernel, ragged pixel and channel tiles
    (2, 512, 29, 27, 64, 1, 2, 0, "relu"),    # C = 512 at stride 2
    (2, 3, 45, 38, 64, 7, 2, 3, "relu"),      # stem: C = 3, 7x7/2, odd output sizes
    (1, 2, 21, 24, 72, 5, 2, 2, "relu6"),     # C = 2, 5x5/2, K = 72 (two channel tiles)
    (2, 3, 40, 36, 64, 3, 1, 1, "relu"),      # C = 3, 3x3/1: a VGG-style first layer, several rows per tile
    (1, 4, 19, 23, 24, 3, 2, 1, "relu6"),     # C = 4, 3x3/2: a MobileNet-style stem, K = 24
    # C = 64 pointwise (the streaming kernel): ragged pixel and channel tiles,
    # and enough pixels that persistent workgroups take several tiles
    (3, 64, 17, 19, 200, 1, 1, 0, "relu6"),
    (8, 64, 48, 50, 72, 1, 1, 0, "relu"),
    (6, 128, 56, 56, 136, 1, 1, 0, "relu"),   # C = 128 and 256 pointwise, several tiles per workgroup
    (12, 256, 40, 40, 72, 1, 1, 0, "none"),
    (16, 128, 57, 50, 264, 1, 2, 0, "relu6"),  # stride-2 pointwise projections (odd input sizes)
    (8, 64, 40, 41, 72, 1, 2, 0, "none"),
    (2, 1, 17, 15, 8, 3, 1, 1, "relu"),      # degenerate channel counts: one input channel,
    (1, 5, 9, 9, 1, 3, 1, 1, "none"),        # one output channel,
    (3, 8, 1, 1, 16, 1, 1, 0, "relu6"),      # a 1 x 1 image
    # 3x3 stride 2 at the ResNet-50 stage entries (the stride-2 patch tiles;
    # batch cut), and odd sizes
    (2, 128, 56, 56, 128, 3, 2, 1, "relu"),
    (2, 256, 28, 28, 256, 3, 2, 1, "relu"),
    (3, 512, 14, 14, 512, 3, 2, 1, "relu"),
    (2, 64, 27, 29, 96, 3, 2, 1, "relu6"),
]


def conv_layer(case):
    n, c, h, w, k, r, st, pad, act = case
    return {"type": "conv", "in": [0], "k": k, "r": r, "s": r, "stride": st, "pad": pad,
            "groups": 1, "act": act}


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("ci", range(len(CONV_CASES)))
def test_conv_every_routine(dtype, ci):
    case = CONV_CASES[ci]
    n, c, h, w, k, r = case[:6]
    layer = conv_layer(case)
    x = random_tensor((n, c, h, w), dtype, seed=10 + ci)
    wt = random_tensor((k, c, r, r), dtype, seed=20 + ci, dist="normal", scale=np.sqrt(2 / (c * r * r)))
    b = random_tensor((k,), "f32", seed=30 + ci, scale=0.1)
    ref = oracle_layer(layer, x, wt, b, dtype)
    g = single_layer_graph(dtype, (n, c, h, w), layer, wt, b)
    xd = to_dev(x, dtype)
    for rt in g.routines(1):
        out = from_dev(run_routine(g, rt["id"], xd), dtype)
        e = err(out, ref, dtype)
        print(f"{dtype} case{ci} {rt['name']}: err {e:.2e}", flush=True)
        assert e <= TOL[dtype], (rt["name"], e)
    g.close()


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("c,k", [(8, 16), (64, 72)])
def test_conv_bit_exact_small_integers(dtype, c, k):
    # values in {-1, 0, 1}: every product and partial sum is an integer of at
    # most C*R*S <= 576, exact in the fp32 accumulators, and the one rounding
    # to the storage dtype is the oracle's, so every routine must match exactly
    n, h, w = 2, 10, 9
    layer = {"type": "conv", "in": [0], "k": k, "r": 3, "s": 3, "stride": 1, "pad": 1,
             "groups": 1, "act": "none"}
    x = random_tensor((n, c, h, w), dtype, seed=1, dist="int")
    wt = random_tensor((k, c, 3, 3), dtype, seed=2, dist="int")
    b = np.zeros(k, np.float32)
    ref = oracle_layer(layer, x, wt, b, dtype)
    g = single_layer_graph(dtype, (n, c, h, w), layer, wt, b)
    xd = to_dev(x, dtype)
    for rt in g.routines(1):
        if "f4x4" in rt["name"]:
            continue  # F(4x4,3x3)'s filter transform (1/6, 1/24) is inexact in binary floating point
        out = from_dev(run_routine(g, rt["id"], xd), dtype)
        assert np.array_equal(out, ref), rt["name"]


@pytest.mark.parametrize("dtype", DTYPES)
# (N, C, H, W, stride): NHWC with C % 8 == 0 and NC8HW8 take the strip kernel
# (vertical strips of 4, 2 or 1 output rows per thread at stride 1, 2 or 1
# at stride 2, by the thread count; output heights not multiples of the
# strip leave short strips), C % 8 != 0 in NHWC and NCHW the general kernel
@pytest.mark.parametrize("case", [(2, 32, 15, 15, 1), (1, 96, 14, 14, 2), (2, 20, 9, 9, 2),
                                  (3, 144, 30, 27, 1), (2, 960, 7, 7, 1), (1, 12, 13, 11, 2),
                                  (2, 24, 33, 34, 2),
                                  (8, 32, 112, 110, 1),    # strips of 4
                                  (8, 32, 110, 112, 1),    # strips of 4, a short last one
                                  (4, 48, 100, 90, 1),     # strips of 2
                                  (8, 96, 112, 111, 2),    # stride 2, strips of 2
                                  (8, 96, 113, 110, 2)])   # ... and a short last one
def test_depthwise(dtype, case):
    n, c, h, w, st = case
    layer = {"type": "conv", "in": [0], "k": c, "r": 3, "s": 3, "stride": st, "pad": 1,
             "groups": c, "act": "relu6"}
    x = random_tensor((n, c, h, w), dtype, seed=3, scale=3.0)
    wt = random_tensor((c, 1, 3, 3), dtype, seed=4, dist="normal", scale=0.5)
    b = random_tensor((c,), "f32", seed=5, scale=0.1)
    ref = oracle_layer(layer, x, wt, b, dtype)
    g = single_layer_graph(dtype, (n, c, h, w), layer, wt, b)
    xd = to_dev(x, dtype)
    for rt in g.routines(1):
        out = from_dev(run_routine(g, rt["id"], xd), dtype)
        assert err(out, ref, dtype) <= TOL[dtype], rt["name"]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape,stride", [((2, 16, 17, 17), 2), ((1, 3, 12, 10), 2), ((2, 64, 56, 56), 2),
                                          ((1, 8, 9, 14), 2), ((1, 8, 1, 1), 2), ((3, 64, 112, 112), 2),
                                          ((2, 16, 9, 9), 1), ((1, 24, 8, 7), 1)])
def test_maxpool_exact(dtype, shape, stride):
    # stride 2 at 112 x 112 is ResNet's pooling layer
    layer = {"type": "maxpool", "in": [0], "k": 3, "stride": stride, "pad": 1}
    x = random_tensor(shape, dtype, seed=6)
    ref = oracle_layer(layer, x, None, None, dtype)
    g = single_layer_graph(dtype, shape, layer)
    xd = to_dev(x, dtype)
    for rt in g.routines(1):
        out = from_dev(run_routine(g, rt["id"], xd), dtype)
        assert out.size == ref.size, rt["name"]
        # a 1 x 1 output comes back as N x C
        assert np.array_equal(out.reshape(ref.shape), ref), rt["name"]          # max is exact


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape", [(2, 24, 7, 7), (1, 13, 5, 5), (4, 2048, 7, 7), (2, 96, 14, 14), (3, 20, 1, 1),
                                   (1, 1280, 7, 7)])
def test_gap(dtype, shape):
    layer = {"type": "gap", "in": [0]}
    x = random_tensor(shape, dtype, seed=7)
    ref = oracle_layer(layer, x, None, None, dtype)
    g = single_layer_graph(dtype, shape, layer)
    xd = to_dev(x, dtype)
    for rt in g.routines(1):
        out = from_dev(run_routine(g, rt["id"], xd), dtype).reshape(ref.shape)
        assert err(out, ref, dtype) <= TOL[dtype] * 0.1, rt["name"]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("case", [(1, 32, 10), (3, 2048, 1000), (32, 1280, 1000), (2, 12, 5),
                                  (40, 24, 37), (64, 2048, 1000)])
def test_fc(dtype, case):
    # 16-bit batches up to 64 with C % 8 == 0 take the MFMA kernel (1, 2 or 4
    # blocks of 16 batch rows; K = 37 leaves a ragged feature tile)
    n, cin, k = case
    from paper_2110_06037_amd import Graph
    x = random_tensor((n, cin, 1, 1), dtype, seed=8)
    wt = random_tensor((k, cin), dtype, seed=9, dist="normal", scale=np.sqrt(2 / cin))
    b = random_tensor((k,), "f32", seed=10, scale=0.1)
    ref = O.round_to(O.fc(to_f64(x, dtype), to_f64(wt, dtype), b.astype(np.float64)), dtype)
    g = Graph(dtype, n, cin, 1, 1, device=0)
    g.add_fc(0, wt, b)
    xd = to_dev(x, dtype)
    for rt in g.routines(1):
        out = from_dev(run_routine(g, rt["id"], xd), dtype).reshape(ref.shape)
        assert err(out, ref, dtype) <= TOL[dtype], rt["name"]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("case", [(32, 1024, 100, "relu"), (3, 64, 24, "relu6"), (2, 12, 5, "relu")])
def test_fc_activation(dtype, case):
    # y = act(W x + b) in every FC routine (dot products, MFMA, 1x1 childnet)
    n, cin, k, act = case
    from paper_2110_06037_amd import Graph
    x = random_tensor((n, cin, 1, 1), dtype, seed=12)
    wt = random_tensor((k, cin), dtype, seed=13, dist="normal", scale=np.sqrt(2 / cin))
    b = random_tensor((k,), "f32", seed=14, scale=0.5)
    ref = O.round_to(O.activate(O.fc(to_f64(x, dtype), to_f64(wt, dtype), b.astype(np.float64)), act), dtype)
    g = Graph(dtype, n, cin, 1, 1, device=0)
    g.add_fc(0, wt, b, act)
    xd = to_dev(x, dtype)
    for rt in g.routines(1):
        out = from_dev(run_routine(g, rt["id"], xd), dtype).reshape(ref.shape)
        assert err(out, ref, dtype) <= TOL[dtype], rt["name"]
        assert np.all(out >= 0) and (act != "relu6" or np.all(out <= 6)), rt["name"]


@pytest.mark.parametrize("dtype", DTYPES)
# C = 1 (NCHW and NHWC hold the same bytes) and C = 8 (NHWC and NC8HW8 do)
# take the void adapt between those layouts; C % 8 == 0 with partial
# 64-channel tiles (72, 136) takes the 16-byte vector converters
@pytest.mark.parametrize("c", [12, 3, 1, 8, 72, 136])
# H * W % 8 == 0 takes the 8-pixel transposes (40 x 40 spans several
# 64-pixel tiles with a ragged last one), 14 x 14 the 4-pixel NC8HW8 one,
# odd sizes the 1-pixel one; NCHW <-> NHWC with H * W % 8 != 0 moves single
# elements on the NCHW side of its tile; C % 8 != 0 takes the element-wise
# converters
@pytest.mark.parametrize("hw", [(9, 9), (12, 10), (40, 40), (14, 14), (7, 7)])
def test_add_and_converters_bit_exact(dtype, c, hw):
    # two maxpools feeding an add: every (layout_a, layout_b, layout_add)
    # combination exercises the converters between all layout pairs (few
    # channels take their own transpose kernel); max and an exactly
    # representable sum keep the result bit-exact
    from paper_2110_06037_amd import Graph
    n, (h, w) = 2, hw
    x = random_tensor((n, c, h, w), dtype, seed=11, dist="int")
    xs = to_f64(x, dtype)
    p = O.maxpool(xs, 3, 1, 1)
    ref = O.add(O.maxpool(p, 3, 1, 1), p, "relu")
    g = Graph(dtype, n, c, h, w, device=0)
    a = g.add_maxpool(0, 3, 1, 1)
    b2 = g.add_maxpool(a, 3, 1, 1)
    g.add_add(b2, a, "relu")
    xd = to_dev(x, dtype)
    for la in range(3):
        for lb in range(3):
            for lc in range(3):
                ids = [0, la, lb, lc]
                g.set_path(ids)
                out = from_dev(g.run(xd), dtype)
                assert np.array_equal(out, ref), ids


RESIDUAL_CASES = [
    # (N, C, H, W, R, act): K = C, stride 1, so the residual is an ADD of the input with itself
    (2, 64, 9, 11, 1, "relu"),      # pointwise, LDS-DMA tiles apply (C % 64 == 0)
    (1, 128, 7, 7, 1, "none"),      # linear, as in an inverted-residual projection
    (2, 24, 13, 11, 3, "relu6"),    # 3x3, C % 8 == 0 but not a multiple of 32
    (3, 40, 5, 5, 1, "relu"),       # K = 40: channel tiles with a ragged end
    (1, 256, 14, 14, 1, "relu"),    # split-reduction parameters apply
    (4, 64, 72, 64, 1, "relu"),     # C = 64: streaming kernel, several tiles per workgroup
    (8, 128, 50, 50, 1, "relu"),    # C = 128: streaming kernel with two 64-channel slabs
    (4, 512, 28, 28, 1, "relu"),    # C = 512: streaming kernel, half the threads store each tile
    (8, 384, 28, 28, 1, "relu"),    # C = 384: streaming kernel staging its sums in the pixel buffer
]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("ci", range(len(RESIDUAL_CASES)))
def test_conv_with_residual_every_routine(dtype, ci):
    # y = act(conv(x) + b + r): every routine that takes a residual, against
    # the oracle's conv (no activation) + add (with the activation) in fp64
    n, c, h, w, r, act = RESIDUAL_CASES[ci]
    spec_layers = [{"type": "add", "in": [0, 0], "act": "none"},
                   {"type": "conv", "in": [0, 1], "k": c, "r": r, "s": r, "stride": 1,
                    "pad": r // 2, "groups": 1, "act": act}]
    x = random_tensor((n, c, h, w), dtype, seed=40 + ci)
    wt = random_tensor((c, c, r, r), dtype, seed=50 + ci, dist="normal", scale=np.sqrt(2 / (c * r * r)))
    b = random_tensor((c,), "f32", seed=60 + ci, scale=0.1)
    xs = to_f64(x, dtype)
    res = O.round_to(O.layer_forward(spec_layers[0], [xs, xs]), dtype)
    ref = O.round_to(O.layer_forward(spec_layers[1], [xs, res], to_f64(wt, dtype), b.astype(np.float64)), dtype)
    g = single_layer_graph(dtype, (n, c, h, w), spec_layers[0])
    g.add_spec(spec_layers[1], wt, b)
    algos = {rt["algo"] for rt in g.routines(2)}
    assert 2 not in algos, "no Winograd routine takes a residual"
    xd = to_dev(x, dtype)
    for rt in g.routines(2):
        out = from_dev(run_routine(g, rt["id"], xd, n_layers=3), dtype)
        e = err(out, ref, dtype)
        print(f"{dtype} residual case{ci} {rt['name']}: err {e:.2e}", flush=True)
        assert e <= TOL[dtype], (rt["name"], e)
    g.close()


PROJECTION_RESIDUAL_CASES = [
    # (N, C, H, W, K, act): y = act(conv1x1(x) + b + r) with r a K-channel
    # tensor made by another 1x1 convolution of x (K != C); pixel counts large
    # enough that every persistent workgroup of the streaming kernel takes
    # several tiles (its residual prefetch alternates register sets)
    (32, 256, 14, 14, 1024, "relu"),   # the ResNet-50 stage-3 expand layers at batch 32
    (8, 64, 56, 56, 256, "relu"),      # stage-1 expand at batch 8
    (32, 512, 7, 7, 2048, "relu"),     # stage-4 expand at batch 32
    (5, 128, 21, 19, 200, "none"),     # ragged pixel and channel tiles
]


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("ci", range(len(PROJECTION_RESIDUAL_CASES)))
def test_conv_with_projection_residual_every_routine(dtype, ci):
    n, c, h, w, k, act = PROJECTION_RESIDUAL_CASES[ci]
    proj = {"type": "conv", "in": [0], "k": k, "r": 1, "s": 1, "stride": 1, "pad": 0, "groups": 1,
            "act": "none"}
    main = {"type": "conv", "in": [0, 1], "k": k, "r": 1, "s": 1, "stride": 1, "pad": 0, "groups": 1,
            "act": act}
    x = random_tensor((n, c, h, w), dtype, seed=70 + ci)
    sc = np.sqrt(2 / c)
    w1 = random_tensor((k, c, 1, 1), dtype, seed=80 + ci, dist="normal", scale=sc)
    w2 = random_tensor((k, c, 1, 1), dtype, seed=90 + ci, dist="normal", scale=sc)
    b1 = random_tensor((k,), "f32", seed=100 + ci, scale=0.1)
    b2 = random_tensor((k,), "f32", seed=110 + ci, scale=0.1)
    xs = to_f64(x, dtype)
    res = O.round_to(O.layer_forward(proj, [xs], to_f64(w1, dtype), b1.astype(np.float64)), dtype)
    ref = O.round_to(O.layer_forward(main, [xs, res], to_f64(w2, dtype), b2.astype(np.float64)), dtype)
    g = single_layer_graph(dtype, (n, c, h, w), proj, w1, b1)
    g.add_spec(main, w2, b2)
    xd = to_dev(x, dtype)
    names = []
    for rt in g.routines(2):
        # the projection runs its NHWC implicit-GEMM routine, so the residual
        # reaches an NHWC consumer without a converter
        p1 = next(r for r in g.routines(1) if r["layout"] == rt["layout"] and r["algo"] == 1)
        g.set_path([0, p1["id"], rt["id"]])
        out = g.run(xd)
        import torch
        torch.cuda.synchronize()
        e = err(from_dev(out, dtype), ref, dtype)
        print(f"{dtype} projection residual case{ci} {rt['name']}: err {e:.2e}", flush=True)
        assert e <= TOL[dtype], (rt["name"], e)
        names.append(rt["name"])
    g.close()
    if c in (64, 128, 256):
        assert any("nhwc/igemm" in nm for nm in names)


# The last six implicit-GEMM parameters split the reduction over workgroups
# when the tiles alone are few, and the last workgroup of each tile to finish
# sums the partial tiles (per-tile counters that every launch leaves at zero).
SPLIT_PARAMS = range(77, 83)
SPLIT_CASES = [
    # (N, C, H, W, K, R, stride, act): ResNet-50 small-M layers (batch cut) and ragged tiles
    (8, 512, 14, 14, 512, 3, 2, "relu"),    # stage-4 first 3x3 (stride 2)
    (8, 2048, 7, 7, 512, 1, 1, "relu"),     # stage-4 reduce
    (4, 1024, 14, 14, 256, 1, 1, "relu"),   # stage-3 reduce
    (3, 64, 9, 7, 40, 3, 1, "relu6"),       # ragged M and N, few reduction steps
]


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("ci", range(len(SPLIT_CASES)))
def test_split_reduction_routines_repeat_exactly(dtype, ci):
    # every split routine against the oracle, and three launches in a row
    # give the same bits (the partial tiles are summed in a fixed order, and
    # a counter left non-zero would make a tile skip or double its sum on the
    # next launch); then a launch on another input must not see any partial
    # tile of the previous ones (the slots are reused)
    n, c, h, w, k, r, st, act = SPLIT_CASES[ci]
    layer = {"type": "conv", "in": [0], "k": k, "r": r, "s": r, "stride": st, "pad": r // 2,
             "groups": 1, "act": act}
    x = random_tensor((n, c, h, w), dtype, seed=70 + ci)
    wt = random_tensor((k, c, r, r), dtype, seed=80 + ci, dist="normal", scale=np.sqrt(2 / (c * r * r)))
    b = random_tensor((k,), "f32", seed=90 + ci, scale=0.1)
    x2 = random_tensor((n, c, h, w), dtype, seed=170 + ci)
    ref = oracle_layer(layer, x, wt, b, dtype)
    ref2 = oracle_layer(layer, x2, wt, b, dtype)
    g = single_layer_graph(dtype, (n, c, h, w), layer, wt, b)
    xd, xd2 = to_dev(x, dtype), to_dev(x2, dtype)
    split = [rt for rt in g.routines(1) if rt["algo"] == 1 and rt["param"] in SPLIT_PARAMS]
    assert split, "the split routines apply"
    for rt in split:
        outs = [from_dev(run_routine(g, rt["id"], xd), dtype) for _ in range(3)]
        e = err(outs[0], ref, dtype)
        e2 = err(from_dev(run_routine(g, rt["id"], xd2), dtype), ref2, dtype)
        print(f"{dtype} split case{ci} {rt['name']}: err {e:.2e}, other input {e2:.2e}", flush=True)
        assert e <= TOL[dtype] and e2 <= TOL[dtype], (rt["name"], e, e2)
        assert all(np.array_equal(o, outs[0]) for o in outs[1:]), rt["name"]
    g.close()


PROJECTED_CASES = [
    # (N, C, H, W, K, R, stride, pad, C2, H2, W2, s2, act): y = act(conv(x) + b + conv1x1_s2(sc) + b2)
    (2, 64, 14, 14, 256, 1, 1, 0, 64, 14, 14, 1, "relu"),       # bottleneck stage 1 (shortcut at stride 1)
    (2, 128, 7, 7, 512, 1, 1, 0, 256, 14, 14, 2, "relu"),       # later stages (shortcut at stride 2)
    (8, 256, 14, 14, 1024, 1, 1, 0, 512, 28, 28, 2, "relu"),    # ResNet-50 stage 3 at batch 8: many tiles
    (3, 64, 9, 11, 72, 3, 1, 1, 128, 17, 21, 2, "relu6"),       # a 3x3 main convolution, ragged tiles
    (1, 40, 5, 5, 24, 1, 1, 0, 12, 9, 9, 2, "none"),            # channels off the tile depth: two launches only
    (3, 64, 13, 15, 72, 1, 1, 0, 64, 25, 29, 2, "relu"),        # streaming 1x1 tiles: ragged pixels and channels
    (4, 128, 28, 28, 512, 1, 1, 0, 256, 56, 56, 2, "relu"),     # ResNet-50 stage 2 entry: 384-channel streaming tiles
    (16, 128, 28, 28, 512, 1, 1, 0, 256, 56, 56, 2, "relu"),    # the same with several tiles per streaming workgroup
]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("ci", range(len(PROJECTED_CASES)))
def test_projected_shortcut_every_routine(dtype, ci):
    # every routine of a convolution with a projected shortcut (the shortcut
    # a second net input) against the oracle's two convolutions summed
    n, c, h, w, k, r, st, pad, c2, h2, w2, s2, act = PROJECTED_CASES[ci]
    if dtype == "f32" and ci == 2:
        pytest.skip("the two-launch float32 routine at this size is slow and covered by the smaller cases")
    from paper_2110_06037_amd import Graph
    import torch
    layer = {"type": "conv", "in": [0, 1], "k": k, "r": r, "s": r, "stride": st, "pad": pad, "groups": 1,
             "act": act, "proj": {"stride": s2}}
    x = random_tensor((n, c, h, w), dtype, seed=200 + ci)
    sc = random_tensor((n, c2, h2, w2), dtype, seed=210 + ci)
    wt = random_tensor((k, c, r, r), dtype, seed=220 + ci, dist="normal", scale=np.sqrt(2 / (c * r * r)))
    wp = random_tensor((k, c2, 1, 1), dtype, seed=230 + ci, dist="normal", scale=np.sqrt(2 / c2))
    b = random_tensor((k,), "f32", seed=240 + ci, scale=0.1)
    bp = random_tensor((k,), "f32", seed=250 + ci, scale=0.1)
    ref = O.round_to(O.layer_forward(layer, [to_f64(x, dtype), to_f64(sc, dtype)],
                                     (to_f64(wt, dtype), to_f64(wp, dtype)),
                                     (b.astype(np.float64), bp.astype(np.float64))), dtype)
    g = Graph(dtype, n, c, h, w, device=0)
    sid = g.add_input(c2, h2, w2)
    lid = g.add_projected_conv(0, sid, wt, b, wp, bp, st, pad, act, s2)
    xd, sd = to_dev(x, dtype), to_dev(sc, dtype)
    rts = g.routines(lid)
    assert {rt["algo"] for rt in rts} <= {0, 1}, "direct and implicit GEMM only"
    if dtype != "f32" and c % 32 == 0 and c2 % 32 == 0:
        assert any(rt["algo"] == 1 for rt in rts), "the one-kernel routines apply"
    for rt in rts:
        g.set_path([0, 0, rt["id"]])
        out = from_dev(g.run_mimo([xd, sd], output_layers=[lid])[0], dtype)
        torch.cuda.synchronize()
        e = err(out, ref, dtype)
        print(f"{dtype} projected case{ci} {rt['name']}: err {e:.2e}", flush=True)
        assert e <= TOL[dtype], (rt["name"], e)
    g.close()


@pytest.mark.parametrize("dtype", DTYPES)
def test_winograd_childnet_sub_routines(dtype):
    # the three-kernel Winograd routines (F(2x2,3x3) and F(4x4,3x3)) are
    # childnets (Sec. III-D): profiling times each of their sub-routines
    # (wgenc, every wgconv GEMM tile, wgdec)
    # on its own, the routine's time is the optimum over them, and each GEMM
    # tile, selected through the cost table, computes the layer (ragged K)
    from oracle.select import childnet_time
    n, c, h, w, k = 2, 64, 13, 14, 72
    layer = {"type": "conv", "in": [0], "k": k, "r": 3, "s": 3, "stride": 1, "pad": 1, "groups": 1,
             "act": "relu"}
    x = random_tensor((n, c, h, w), dtype, seed=301)
    wt = random_tensor((k, c, 3, 3), dtype, seed=302, dist="normal", scale=np.sqrt(2 / (c * 9)))
    b = random_tensor((k,), "f32", seed=303, scale=0.1)
    ref = oracle_layer(layer, x, wt, b, dtype)
    g = single_layer_graph(dtype, (n, c, h, w), layer, wt, b)
    g.profile(warmup=1, reps=3)
    kids = [r for r in g.costs()["layers"][1]["routines"] if "child" in r]
    assert kids and all(r["algo"] == 2 and "fused" not in r["name"] for r in kids)
    xd = to_dev(x, dtype)
    for r in kids:
        rows = r["child"]["ns"]
        assert all(v > 0 for row in rows for v in row), rows
        t, choice = childnet_time(rows)
        assert r["ns"] == t and tuple(r["child"]["path"]) == choice
        for q in range(len(rows[1])):
            costs = g.costs()
            mine = costs["layers"][1]["routines"][r["rid"]]
            mine["child"]["ns"][1] = [1 if j == q else 10 ** 6 for j in range(len(rows[1]))]
            g.set_costs(costs)
            assert g.costs()["layers"][1]["routines"][r["rid"]]["child"]["path"][1] == q
            out = from_dev(run_routine(g, r["rid"], xd), dtype)
            e = err(out, ref, dtype)
            print(f"{dtype} {r['name']} wgconv:p{q}: err {e:.2e}", flush=True)
            assert e <= TOL[dtype], (r["name"], q, e)
    g.close()
