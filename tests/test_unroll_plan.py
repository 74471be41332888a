"""The few-channel folding plans (qconv.few_channel_plan), checked on the CPU:
the unroll written out from its definition in include/qconv.h, then the
oracle's convolution of the unrolled operands under the plan's descriptor
must equal the oracle's direct convolution of the original layer."""
import numpy as np
import pytest

import oracle

from _util import unroll_def


@pytest.mark.parametrize("case", [
    # n, h, w, c, k, r, s, stride, pad
    (2, 23, 21, 3, 8, 7, 7, 2, 3),     # the stem's filter, stride and padding on a small image
    (1, 17, 19, 2, 4, 5, 5, 3, 1),     # a stride that does not divide the filter
    (1, 9, 9, 3, 4, 3, 3, 1, 1),       # stride 1: row groups of one
    (1, 12, 10, 1, 4, 4, 2, 2, 0),     # even filter, no padding
])
@pytest.mark.parametrize("fold", ["rows", "all"])
def test_folding_equals_direct_convolution(case, fold):
    from paper_2202_06819_amd import qconv
    n, h, w, c, k, r, s, st, pad = case
    rng = np.random.default_rng([31, h, w, c, r, st, len(fold)])
    x = rng.integers(-128, 128, size=(n, c, h, w), dtype=np.int8)
    f = rng.integers(-128, 128, size=(k, c, r, s), dtype=np.int8)
    d = dict(n=n, h=h, w=w, c=c, k=k, r=r, s=s, stride_h=st, stride_w=st, pad_h=pad, pad_w=pad, bits=8, x_signed=1,
             w_signed=1)
    taps_h = r if fold == "all" else st
    c_out = -(-taps_h * s * c // 16) * 16
    plan = qconv.few_channel_plan(d, c_out, fold)
    xu = unroll_def(x, c_out, **plan["x"])
    wu = unroll_def(f, c_out, **plan["w"])
    e = plan["desc"]
    assert xu.shape[1:3] == (e["h"], e["w"]) and wu.shape == (k, e["r"], 1, c_out)
    got = oracle.conv2d(xu, wu, stride=(e["stride_h"], e["stride_w"]), pad=(e["pad_h"], e["pad_w"]))
    want = oracle.conv2d(x.transpose(0, 2, 3, 1), f.transpose(0, 2, 3, 1), stride=(st, st), pad=(pad, pad))
    assert got.shape == want.shape
    assert np.array_equal(got, want)
