"""Pins of the numerical oracle against what the mathematics fixes.

Each test checks the oracle against something other than itself: hand-counted
closed forms, the GEMM (im2col) formulation, Winograd's minimal filtering
F(2x2, 3x3) (the method the paper cites for its Winograd routines, Sec. II-B),
special cases with exact answers, and torch's float64 CPU layer routines as an
independent library implementation.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import numeric as O
from workloads import generate, materialise, tiny_chain, to_f64


def rng(seed=0):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- conv: closed forms

def test_conv_neighbour_counts_pad1():
    # all-ones 4x4 input, all-ones 3x3 kernel, pad 1: each output counts the
    # in-bounds neighbours (corner 4, edge 6, interior 9)
    x = np.ones((1, 1, 4, 4))
    w = np.ones((1, 1, 3, 3))
    y = O.conv2d(x, w, None, stride=1, pad=1)
    expect = np.array([[4, 6, 6, 4], [6, 9, 9, 6], [6, 9, 9, 6], [4, 6, 6, 4]], float)
    assert np.array_equal(y[0, 0], expect)


def test_conv_stride2_picks_every_other_centre():
    x = np.ones((1, 1, 4, 4))
    w = np.ones((1, 1, 3, 3))
    y = O.conv2d(x, w, None, stride=2, pad=1)
    assert np.array_equal(y[0, 0], np.array([[4, 6], [6, 9]], float))


def test_conv_is_cross_correlation_not_convolution():
    # a kernel with a single 1 at (0, 0) reads x[p - 1, q - 1] (pad 1): no flip
    x = np.arange(16, dtype=float).reshape(1, 1, 4, 4)
    w = np.zeros((1, 1, 3, 3))
    w[0, 0, 0, 0] = 1.0
    y = O.conv2d(x, w, None, stride=1, pad=1)
    expect = np.zeros((4, 4))
    expect[1:, 1:] = x[0, 0, :3, :3]
    assert np.array_equal(y[0, 0], expect)


def test_delta_kernel_is_identity_bitexact():
    x = rng(1).standard_normal((2, 5, 7, 6))
    w = np.zeros((5, 5, 3, 3))
    for c in range(5):
        w[c, c, 1, 1] = 1.0
    y = O.conv2d(x, w, None, stride=1, pad=1)
    assert np.array_equal(y, x)


# ---------------------------------------------------------------- conv: GEMM identity

def _im2col(x, r, s, stride, pad):
    """Independent im2col: rows (c, r, s), columns (n, p, q)."""
    n, c, h, w = x.shape
    xp = np.zeros((n, c, h + 2 * pad, w + 2 * pad))
    xp[:, :, pad:pad + h, pad:pad + w] = x
    p = (h + 2 * pad - r) // stride + 1
    q = (w + 2 * pad - s) // stride + 1
    cols = np.empty((c * r * s, n * p * q))
    row = 0
    for ci in range(c):
        for ri in range(r):
            for si in range(s):
                patch = xp[:, ci, ri:ri + stride * p:stride, si:si + stride * q:stride]
                cols[row] = patch.reshape(-1)
                row += 1
    return cols, p, q


@pytest.mark.parametrize("shape", [
    (2, 3, 9, 11, 4, 3, 3, 1, 1), (1, 5, 8, 8, 6, 3, 3, 2, 1), (3, 4, 7, 5, 2, 1, 1, 1, 0),
    (1, 3, 15, 15, 8, 7, 7, 2, 3), (2, 6, 6, 6, 3, 5, 3, 1, 2)])
def test_conv_equals_im2col_matmul(shape):
    n, c, h, w_, k, r, s, st, pad = shape
    g = rng(2)
    x = g.standard_normal((n, c, h, w_))
    w = g.standard_normal((k, c, r, s))
    b = g.standard_normal(k)
    y = O.conv2d(x, w, b, stride=st, pad=pad)
    cols, p, q = _im2col(x, r, s, st, pad)
    ref = (w.reshape(k, -1) @ cols + b[:, None]).reshape(k, n, p, q).transpose(1, 0, 2, 3)
    assert y.shape == ref.shape
    assert np.max(np.abs(y - ref)) <= 1e-13 * np.max(np.abs(ref))


def test_pointwise_conv_is_matmul():
    g = rng(3)
    x = g.standard_normal((2, 16, 5, 4))
    w = g.standard_normal((8, 16, 1, 1))
    y = O.conv2d(x, w, None)
    ref = np.einsum("kc,nchw->nkhw", w[:, :, 0, 0], x)
    assert np.max(np.abs(y - ref)) <= 1e-13 * np.max(np.abs(ref))


# ---------------------------------------------------------------- conv: Winograd identity

# F(2, 3) minimal filtering matrices (Lavin and Gray's construction).
BT = np.array([[1, 0, -1, 0], [0, 1, 1, 0], [0, -1, 1, 0], [0, 1, 0, -1]], float)
G = np.array([[1, 0, 0], [0.5, 0.5, 0.5], [0.5, -0.5, 0.5], [0, 0, 1]], float)
AT = np.array([[1, 1, 1, 0], [0, 1, -1, -1]], float)


def test_winograd_1d_f23_matches_direct():
    g = rng(4)
    for _ in range(20):
        d = g.standard_normal(4)
        f = g.standard_normal(3)
        y = AT @ ((G @ f) * (BT @ d))
        direct = np.array([d[0] * f[0] + d[1] * f[1] + d[2] * f[2],
                           d[1] * f[0] + d[2] * f[1] + d[3] * f[2]])
        assert np.max(np.abs(y - direct)) <= 1e-13


@pytest.mark.parametrize("hw", [(8, 8), (7, 9)])
def test_winograd_2d_f2x2_3x3_matches_oracle(hw):
    h, w_ = hw
    g = rng(5)
    n, c, k = 2, 3, 4
    x = g.standard_normal((n, c, h, w_))
    wt = g.standard_normal((k, c, 3, 3))
    y = O.conv2d(x, wt, None, stride=1, pad=1)
    # Winograd over 2x2 output tiles; input zero-extended beyond the padding
    th, tw = (h + 1) // 2, (w_ + 1) // 2
    xp = np.zeros((n, c, 2 * th + 2, 2 * tw + 2))
    xp[:, :, 1:1 + h, 1:1 + w_] = x
    U = np.einsum("ij,kcjl,ml->kcim", G, wt, G)            # G g G^T
    out = np.zeros((n, k, 2 * th, 2 * tw))
    for ty in range(th):
        for tx in range(tw):
            d = xp[:, :, 2 * ty:2 * ty + 4, 2 * tx:2 * tx + 4]
            V = np.einsum("ij,ncjl,ml->ncim", BT, d, BT)     # B^T d B
            M = np.einsum("kcim,ncim->nkim", U, V)
            Y = np.einsum("ij,nkjl,ml->nkim", AT, M, AT)     # A^T M A
            out[:, :, 2 * ty:2 * ty + 2, 2 * tx:2 * tx + 2] = Y
    out = out[:, :, :h, :w_]
    assert np.max(np.abs(out - y)) <= 1e-12 * np.max(np.abs(y))


# ---------------------------------------------------------------- conv vs torch (library)

@pytest.mark.parametrize("cfg", [
    dict(n=2, c=6, h=9, w=7, k=5, r=3, st=1, pad=1, groups=1, act="relu"),
    dict(n=1, c=3, h=17, w=17, k=8, r=7, st=2, pad=3, groups=1, act="none"),
    dict(n=2, c=8, h=10, w=10, k=8, r=3, st=2, pad=1, groups=8, act="relu6"),
    dict(n=1, c=12, h=7, w=7, k=12, r=3, st=1, pad=1, groups=12, act="relu6"),
    dict(n=3, c=4, h=5, w=5, k=7, r=1, st=2, pad=0, groups=1, act="relu")])
def test_conv_matches_torch_f64(cfg):
    g = rng(6)
    x = g.standard_normal((cfg["n"], cfg["c"], cfg["h"], cfg["w"])) * 3
    w = g.standard_normal((cfg["k"], cfg["c"] // cfg["groups"], cfg["r"], cfg["r"]))
    b = g.standard_normal(cfg["k"])
    y = O.conv2d(x, w, b, cfg["st"], cfg["pad"], cfg["groups"], cfg["act"])
    t = F.conv2d(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b),
                 stride=cfg["st"], padding=cfg["pad"], groups=cfg["groups"])
    if cfg["act"] == "relu":
        t = t.clamp_min(0)
    elif cfg["act"] == "relu6":
        t = t.clamp(0, 6)
    assert np.max(np.abs(y - t.numpy())) <= 1e-12 * max(1.0, np.max(np.abs(y)))


def test_conv_points_match_full():
    g = rng(7)
    x = g.standard_normal((2, 6, 9, 8))
    w = g.standard_normal((4, 6, 3, 3))
    b = g.standard_normal(4)
    y = O.conv2d(x, w, b, 2, 1, 1, "relu")
    idx = np.stack([g.integers(0, s, 50) for s in y.shape], axis=1)
    pts = O.conv2d_points(x, w, b, idx, 2, 1, 1, "relu")
    assert np.array_equal(pts, y[idx[:, 0], idx[:, 1], idx[:, 2], idx[:, 3]])


def test_depthwise_equals_per_channel_dense():
    g = rng(8)
    x = g.standard_normal((2, 5, 8, 8))
    w = g.standard_normal((5, 1, 3, 3))
    y = O.conv2d(x, w, None, 2, 1, groups=5)
    for c in range(5):
        yc = O.conv2d(x[:, c:c + 1], w[c:c + 1], None, 2, 1)
        assert np.array_equal(y[:, c:c + 1], yc)


# ---------------------------------------------------------------- other layers

def test_maxpool_hand_example_and_torch():
    x = np.arange(25, dtype=float).reshape(1, 1, 5, 5)
    y = O.maxpool(x, 3, 2, 1)
    assert np.array_equal(y[0, 0], np.array([[6, 8, 9], [16, 18, 19], [21, 23, 24]], float))
    g = rng(9)
    x = g.standard_normal((2, 3, 11, 10))
    t = F.max_pool2d(torch.from_numpy(x), 3, 2, 1).numpy()
    assert np.array_equal(O.maxpool(x, 3, 2, 1), t)


def test_maxpool_padding_is_minus_infinity():
    x = -np.ones((1, 1, 4, 4)) * 5.0
    assert np.all(O.maxpool(x, 3, 2, 1) == -5.0)


def test_gap_constant_and_torch():
    x = np.full((2, 3, 7, 7), 1.25)
    assert np.all(O.gap(x) == 1.25)
    g = rng(10)
    x = g.standard_normal((2, 4, 6, 5))
    t = F.adaptive_avg_pool2d(torch.from_numpy(x), 1).numpy()
    assert np.max(np.abs(O.gap(x) - t)) <= 1e-15


def test_add_activation():
    a = np.array([1.0, -2.0, 5.0, 3.5]).reshape(1, 4, 1, 1)
    b = np.array([0.5, 1.0, 4.0, -0.5]).reshape(1, 4, 1, 1)
    assert np.array_equal(O.add(a, b, "none").ravel(), [1.5, -1.0, 9.0, 3.0])
    assert np.array_equal(O.add(a, b, "relu").ravel(), [1.5, 0.0, 9.0, 3.0])
    assert np.array_equal(O.add(a, b, "relu6").ravel(), [1.5, 0.0, 6.0, 3.0])


def test_fc_matches_torch_and_pointwise_conv():
    g = rng(11)
    x = g.standard_normal((3, 32, 1, 1))
    w = g.standard_normal((10, 32))
    b = g.standard_normal(10)
    y = O.fc(x, w, b)
    t = F.linear(torch.from_numpy(x.reshape(3, 32)), torch.from_numpy(w), torch.from_numpy(b))
    assert np.max(np.abs(y.reshape(3, 10) - t.numpy())) <= 1e-13
    # the paper's dense childnet: reshape -> 1x1 conv -> reshape (Sec. III-D)
    yc = O.conv2d(x, w.reshape(10, 32, 1, 1), b)
    assert np.max(np.abs(yc - y)) <= 1e-13


def test_activate_hand_values():
    y = np.array([-1.5, 0.0, 2.0, 7.25, 6.0])
    assert np.array_equal(O.activate(y, "none"), y)
    assert np.array_equal(O.activate(y, "relu"), [0.0, 0.0, 2.0, 7.25, 6.0])
    assert np.array_equal(O.activate(y, "relu6"), [0.0, 0.0, 2.0, 6.0, 6.0])


def test_fc_layer_activation_matches_the_conv_oracles():
    # an FC layer with an activation == the same dense childnet as a 1x1
    # convolution whose activation the C oracle applies
    g = rng(31)
    x = g.standard_normal((2, 24, 1, 1))
    w = g.standard_normal((9, 24))
    b = g.standard_normal(9)
    for act in ("none", "relu", "relu6"):
        y = O.layer_forward({"type": "fc", "in": [0], "k": 9, "act": act}, [x], w, b)
        yc = O.conv2d(x, w.reshape(9, 24, 1, 1), b, act=act)
        assert np.max(np.abs(y - yc)) <= 1e-13, act


def test_full_window_conv_is_flatten_then_fc():
    # a convolution whose kernel covers the whole C x H x W input (no padding)
    # is the dense layer on the NCHW-flattened input: how a classifier that
    # flattens a feature map is expressed with an H x W convolution
    g = rng(32)
    x = g.standard_normal((3, 5, 4, 4))
    w = g.standard_normal((7, 5, 4, 4))
    b = g.standard_normal(7)
    yc = O.conv2d(x, w, b, 1, 0)
    yf = O.fc(x.reshape(3, 80, 1, 1), w.reshape(7, 80), b)
    assert yc.shape == (3, 7, 1, 1)
    assert np.max(np.abs(yc - yf)) <= 1e-13


# ---------------------------------------------------------------- storage rounding

def test_round_f32_f16_match_numpy_casts():
    g = rng(12)
    v = g.standard_normal(20000) * 10.0 ** g.integers(-9, 6, 20000)
    assert np.array_equal(O.round_to(v, "f32"), v.astype(np.float32).astype(np.float64))
    v16 = g.standard_normal(20000) * 10.0 ** g.integers(-9, 5, 20000)
    with np.errstate(over="ignore"):
        ref = v16.astype(np.float16).astype(np.float64)
    assert np.array_equal(O.round_to(v16, "f16"), ref)


def test_round_bf16_matches_generator_and_hand_cases():
    g = rng(13)
    v = g.standard_normal(20000) * 10.0 ** g.integers(-40, 38, 20000)
    assert np.array_equal(O.round_to(v, "bf16"), to_f64(materialise(v, "bf16"), "bf16"))
    # ties to even at 1: ulp(1) = 2**-7
    cases = {1 + 2 ** -8: 1.0, 1 + 3 * 2 ** -8: 1 + 2 ** -6, 1 + 2 ** -8 + 2 ** -30: 1 + 2 ** -7,
             -(1 + 2 ** -8): -1.0, 2 ** -133: 2 ** -133, 2 ** -134: 0.0}
    for a, b in cases.items():
        assert O.round_to([a], "bf16")[0] == b, a


def test_round_f16_overflow_and_subnormal():
    assert O.round_to([65519.0], "f16")[0] == 65504.0
    assert np.isinf(O.round_to([65520.0], "f16")[0])
    assert O.round_to([2 ** -25], "f16")[0] == 0.0           # tie -> even (0)
    assert O.round_to([3 * 2 ** -26], "f16")[0] == 2 ** -24


# ---------------------------------------------------------------- whole-net forward

def test_tiny_chain_forward_matches_torch():
    spec = tiny_chain()
    t = generate(spec)
    tens = {"x": to_f64(t["x"], "f32"), "w": [None if w is None else to_f64(w, "f32") for w in t["w"]],
            "b": [None if b is None else b.astype(np.float64) for b in t["b"]]}
    outs = O.forward(spec, tens, storage="f64", keep=True)
    h = torch.from_numpy(tens["x"])
    L = spec["layers"]
    ws, bs = [torch.from_numpy(w) if w is not None else None for w in tens["w"]], \
        [torch.from_numpy(b) if b is not None else None for b in tens["b"]]
    h1 = F.conv2d(h, ws[0], bs[0], 1, 1).clamp_min(0)
    h2 = F.conv2d(h1, ws[1], bs[1], 2, 1).clamp_min(0)
    h3 = F.conv2d(h2, ws[2], bs[2])
    h4 = h3.mean(dim=(2, 3))
    h5 = F.linear(h4, ws[4], bs[4])
    assert len(L) == 5
    assert np.max(np.abs(outs[5].reshape(1, 10) - h5.numpy())) <= 1e-12
    assert outs[2].shape == (1, 32, 16, 16)
