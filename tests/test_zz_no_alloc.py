"""The allocation-free run (sn_run_noalloc): the same plan as sn_run with its
intermediate tensors and workspaces in the library's static per-device
region, called through the C ABI, checked against sn_run of the same graph
bit for bit on two calls in a row (the second graph smaller, so it runs on
what the first left in the shared region), and a plan too large for the
region is refused."""

import numpy as np
import pytest

from paper_2110_06037_amd import build_from_spec, native as N
from tests.gpu_util import from_dev, to_dev
from workloads import fuse_residual, generate, mobilenet_v2, resnet18, resnet50, tiny_chain

pytestmark = pytest.mark.gpu


def _both(spec, path_mode):
    import torch
    t = generate(spec)
    g = build_from_spec(spec, t)
    if path_mode == "dprs":
        g.profile(warmup=1, reps=3)
        g.select("dprs")
    else:
        g.select("fixed", *path_mode)
    x = to_dev(t["x"], spec["dtype"])
    ref = g.run(x)
    torch.cuda.synchronize()
    out = torch.full_like(ref, float("nan"))
    g.run_noalloc(x, out)
    torch.cuda.synchronize()
    a = from_dev(ref, spec["dtype"])
    b = from_dev(out, spec["dtype"])
    g.close()
    return a, b


def test_noalloc_run_equals_run_on_two_calls_in_a_row():
    # first a larger plan (ResNet-18 at batch 4, split-reduction and Winograd
    # workspaces included), then a smaller one (the tiny chain): the second
    # runs on the region the first left written
    cases = [(fuse_residual(resnet18(4)), ("NHWC", "winograd")),
             (tiny_chain(), "dprs"),
             (mobilenet_v2(1), ("NC8HW8", "igemm"))]
    for spec, mode in cases:
        a, b = _both(spec, mode)
        assert np.all(np.isfinite(a)), spec["name"]
        assert np.array_equal(a, b), spec["name"]


def test_noalloc_rejects_a_plan_larger_than_the_region():
    import torch
    spec = resnet50(32, "bf16")
    t = generate(spec)
    g = build_from_spec(spec, t)
    g.select("fixed", "NHWC", "igemm")
    x = to_dev(t["x"], "bf16")
    out = g.empty_output()
    with pytest.raises(N.SNError) as e:
        g.run_noalloc(x, out)
    assert e.value.code == -4 and "static region" in str(e.value)
    torch.cuda.synchronize()
    g.close()
