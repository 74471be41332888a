"""Pins for the CPU oracle (no GPU).

Each test ties the oracle to something other than its own code: a library
routine written independently (torch's float64 convolution, numpy's integer
matrix product), a closed form, an invariant the mathematics fixes, exact
rational arithmetic, the operation count printed in Table 1, or words built by
hand.  A plausible slip anywhere in the oracle -- a dropped tap, a flipped
kernel, a wrong stride or padding index, a transposed operand, a rounding
direction, a nibble order -- fails at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from oracle import brute
import qconv_inputs as qi

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(g, shape, lo, hi):
    return g.integers(lo, hi + 1, size=shape).astype(np.int32)


def _torch_conv(x_nhwc, w_krsc, stride, pad):
    """torch.nn.functional.conv2d in float64 on integer-valued tensors (exact below 2^53)."""
    x = torch.from_numpy(x_nhwc.astype(np.float64)).permute(0, 3, 1, 2)
    w = torch.from_numpy(w_krsc.astype(np.float64)).permute(0, 3, 1, 2)
    y = torch.nn.functional.conv2d(x, w, stride=stride, padding=pad)
    return y.permute(0, 2, 3, 1).numpy()


# ----------------------------------------------------------------- op count (Table 1)

def test_table1_op_count():
    gold = json.load(open(os.path.join(GOLDEN, "table1_ops.json")))
    r, s = gold["kernel"]
    for st in gold["stages"]:
        hw, ch = st["hw"], st["channels"]
        p = oracle.out_dim(hw, r, gold["stride"], gold["pad"])
        q = oracle.out_dim(hw, s, gold["stride"], gold["pad"])
        assert (p, q) == (hw, hw)
        assert 2 * 8 * p * q * ch * ch * r * s == gold["ops_per_conv"]
        # no other batch size reproduces the printed value
        assert [n for n in range(1, 65) if 2 * n * p * q * ch * ch * r * s == gold["ops_per_conv"]] == [8]
    for L in qi.table1_layers(8):
        assert L.ops == gold["ops_per_conv"]
    assert qi.workload1()[0].ops == gold["ops_per_conv"]


def test_out_dim_cases():
    assert oracle.out_dim(56, 3, 1, 1) == 56
    assert oracle.out_dim(56, 3, 2, 1) == 28
    assert oracle.out_dim(56, 1, 2, 0) == 28
    assert oracle.out_dim(7, 7, 1, 0) == 1
    assert oracle.out_dim(224, 7, 2, 3) == 112
    with pytest.raises(oracle.OracleError):
        oracle.out_dim(2, 5, 1, 1)


# ----------------------------------------------------------------- convolution

CONV_CASES = [
    # n, h, w, c, k, r, s, sh, sw, ph, pw
    (1, 5, 5, 3, 2, 3, 3, 1, 1, 1, 1),
    (2, 7, 6, 5, 4, 3, 3, 2, 2, 1, 1),
    (1, 9, 8, 4, 3, 5, 5, 1, 2, 2, 1),
    (2, 6, 6, 8, 8, 1, 1, 2, 2, 0, 0),
    (1, 10, 7, 3, 2, 7, 3, 3, 1, 3, 0),
    (3, 4, 4, 16, 8, 3, 3, 1, 1, 0, 0),
    (1, 8, 8, 8, 4, 2, 3, 2, 1, 0, 2),
]


@pytest.mark.parametrize("case", CONV_CASES)
def test_conv_matches_torch_float64(case):
    n, h, w, c, k, r, s, sh, sw, ph, pw = case
    g = np.random.default_rng(list(case))
    x = _rand(g, (n, h, w, c), -128, 127)
    wt = _rand(g, (k, r, s, c), -128, 127)
    got = oracle.conv2d(x, wt, (sh, sw), (ph, pw))
    ref = _torch_conv(x, wt, (sh, sw), (ph, pw))
    assert got.shape == ref.shape
    assert np.array_equal(got.astype(np.float64), ref)


def test_conv_1x1_is_integer_gemm():
    g = np.random.default_rng(11)
    x = _rand(g, (2, 5, 7, 24), -8, 7)
    wt = _rand(g, (16, 1, 1, 24), -8, 7)
    got = oracle.conv2d(x, wt)
    ref = x.reshape(-1, 24).astype(np.int64) @ wt.reshape(16, 24).astype(np.int64).T
    assert np.array_equal(got.reshape(-1, 16), ref)


@pytest.mark.parametrize("r0,s0", [(0, 0), (0, 2), (1, 1), (2, 0), (2, 1)])
@pytest.mark.parametrize("stride", [1, 2])
def test_shifted_delta_kernel(r0, s0, stride):
    """w[k, r0, s0, c] = [k == c] picks x at (p*st - 1 + r0, q*st - 1 + s0): pins the
    direction of the taps (cross-correlation) and the padding offset."""
    g = np.random.default_rng(5)
    c = 6
    x = _rand(g, (2, 7, 9, c), 0, 15)
    wt = np.zeros((c, 3, 3, c), dtype=np.int32)
    for ch in range(c):
        wt[ch, r0, s0, ch] = 1
    got = oracle.conv2d(x, wt, (stride, stride), (1, 1))
    xp = np.pad(x, ((0, 0), (1, 1), (1, 1), (0, 0)))
    p, q = got.shape[1], got.shape[2]
    ref = xp[:, r0:r0 + stride * (p - 1) + 1:stride, s0:s0 + stride * (q - 1) + 1:stride, :]
    assert np.array_equal(got, ref)


def test_centre_delta_is_identity():
    g = np.random.default_rng(6)
    x = _rand(g, (1, 56, 56, 8), 0, 15)
    wt = np.zeros((8, 3, 3, 8), dtype=np.int32)
    wt[np.arange(8), 1, 1, np.arange(8)] = 1
    assert np.array_equal(oracle.conv2d(x, wt, (1, 1), (1, 1)), x)


@pytest.mark.parametrize("h,w,r,s,st,pad", [(5, 5, 3, 3, 1, 1), (6, 4, 3, 3, 2, 1), (7, 7, 5, 5, 1, 2),
                                            (4, 4, 3, 3, 1, 0), (5, 5, 3, 3, 3, 2)])
def test_all_ones_counts_valid_taps(h, w, r, s, st, pad):
    """x = 1, w = 1: each output counts the taps that land inside the image, times C."""
    c, k = 4, 3
    x = np.ones((1, h, w, c), dtype=np.int32)
    wt = np.ones((k, r, s, c), dtype=np.int32)
    got = oracle.conv2d(x, wt, (st, st), (pad, pad))
    p, q = got.shape[1:3]
    for pi in range(p):
        rows = sum(1 for ri in range(r) if 0 <= pi * st - pad + ri < h)
        for qj in range(q):
            cols = sum(1 for si in range(s) if 0 <= qj * st - pad + si < w)
            assert (got[0, pi, qj] == c * rows * cols).all()


def test_linearity_and_sign():
    g = np.random.default_rng(7)
    x = _rand(g, (2, 8, 8, 16), 0, 15)
    w1 = _rand(g, (8, 3, 3, 16), -8, 7)
    w2 = _rand(g, (8, 3, 3, 16), -8, 7)
    a1 = oracle.conv2d(x, w1, (1, 1), (1, 1)).astype(np.int64)
    a2 = oracle.conv2d(x, w2, (1, 1), (1, 1)).astype(np.int64)
    a12 = oracle.conv2d(x, w1 + w2, (1, 1), (1, 1)).astype(np.int64)
    assert np.array_equal(a12, a1 + a2)
    assert np.array_equal(oracle.conv2d(x, -w1, (1, 1), (1, 1)), -a1)
    x2 = _rand(g, (2, 8, 8, 16), 0, 15)
    b = oracle.conv2d(x2, w1, (1, 1), (1, 1)).astype(np.int64)
    assert np.array_equal(oracle.conv2d(x + x2, w1, (1, 1), (1, 1)), a1 + b)
    assert not oracle.conv2d(np.zeros_like(x), w1, (1, 1), (1, 1)).any()


def test_translation_equivariance_interior():
    g = np.random.default_rng(8)
    x = _rand(g, (1, 12, 12, 4), 0, 15)
    wt = _rand(g, (3, 3, 3, 4), -8, 7)
    xs = np.roll(x, shift=(2, 3), axis=(1, 2))
    a = oracle.conv2d(x, wt, (1, 1), (1, 1))
    b = oracle.conv2d(xs, wt, (1, 1), (1, 1))
    # interior outputs whose windows do not touch the wrapped or padded border
    assert np.array_equal(b[:, 4:11, 5:11], a[:, 2:9, 2:8])


def test_stride_is_subsampled_stride1():
    g = np.random.default_rng(9)
    x = _rand(g, (2, 11, 10, 8), -8, 7)
    wt = _rand(g, (4, 3, 3, 8), -8, 7)
    full = oracle.conv2d(x, wt, (1, 1), (1, 1))
    assert np.array_equal(oracle.conv2d(x, wt, (2, 2), (1, 1)), full[:, ::2, ::2])
    assert np.array_equal(oracle.conv2d(x, wt, (3, 2), (1, 1)), full[:, ::3, ::2])


@pytest.mark.parametrize("seed", range(4))
def test_conv_matches_pure_python_lowering(seed):
    g = np.random.default_rng(100 + seed)
    n, h, w = 1 + seed % 2, int(g.integers(3, 7)), int(g.integers(3, 7))
    c, k = int(g.integers(1, 5)), int(g.integers(1, 4))
    r, s = int(g.integers(1, 4)), int(g.integers(1, 4))
    st, pad = int(g.integers(1, 3)), int(g.integers(0, 2))
    if h + 2 * pad < r or w + 2 * pad < s:
        pytest.skip("window larger than padded input")
    x = _rand(g, (n, h, w, c), -128, 127)
    wt = _rand(g, (k, r, s, c), -128, 127)
    got = oracle.conv2d(x, wt, (st, st), (pad, pad))
    ref = np.array(brute.conv2d(x.tolist(), wt.tolist(), (st, st), (pad, pad)))
    assert np.array_equal(got, ref)


def test_sampled_pixels_equal_full():
    g = np.random.default_rng(12)
    x = _rand(g, (2, 9, 9, 16), 0, 15)
    wt = _rand(g, (8, 3, 3, 16), -8, 7)
    full = oracle.conv2d(x, wt, (2, 2), (1, 1))
    pix = np.array([0, 5, 17, 31, 49], dtype=np.int64)
    part = oracle.conv2d(x, wt, (2, 2), (1, 1), pixels=pix)
    assert np.array_equal(part, full.reshape(-1, 8)[pix])


def test_threads_do_not_change_result():
    g = np.random.default_rng(13)
    x = _rand(g, (4, 14, 14, 32), 0, 15)
    wt = _rand(g, (16, 3, 3, 32), -8, 7)
    a = oracle.conv2d(x, wt, (1, 1), (1, 1), threads=1)
    b = oracle.conv2d(x, wt, (1, 1), (1, 1), threads=4)
    assert np.array_equal(a, b)


def test_accumulator_bound_is_enforced():
    """Sec. 3.2.1: sums must fit the 32-bit accumulator; 2^31 itself does not."""
    c = 1 << 17
    x = np.full((1, 1, 1, c), -128, dtype=np.int32)
    wt = np.full((1, 1, 1, c), -128, dtype=np.int32)
    with pytest.raises(oracle.OracleError):
        oracle.conv2d(x, wt)            # 2^14 * 2^17 = 2^31
    wt[0, 0, 0, 0] = -127               # 2^31 - 128
    assert oracle.conv2d(x, wt)[0, 0, 0, 0] == 2 ** 31 - 128


def test_worst_case_accumulators_of_the_workloads_fit():
    """Largest |acc| any workload can reach stays below 2^31 (Sec. 3.2.1)."""
    for cfg in (2, 3, 4):
        for L in qi.WORKLOADS[cfg]():
            xm = max(abs(v) for v in L.x_range)
            wm = max(abs(v) for v in L.w_range)
            assert L.c * L.r * L.s * xm * wm < 2 ** 31


# ----------------------------------------------------------------- requantiser

def _exact_requant(acc, mult, shift, relu, lo, hi):
    """Round half up written with exact rationals: floor(acc*mult/2^shift + 1/2)."""
    v = math.floor(Fraction(acc * mult, 2 ** shift) + Fraction(1, 2))
    if relu:
        v = max(v, 0)
    return min(max(v, lo), hi)


def test_requant_closed_forms():
    m = np.full(1, 1 << 14, dtype=np.int32)

    def rq(a, relu=False, lo=-1000, hi=1000):
        return int(oracle.requant(np.array([[a]], dtype=np.int32), m, 20, relu, lo, hi)[0, 0])

    # acc * 2^14 / 2^20 = acc / 64
    assert rq(32) == 1          # exactly 0.5 -> rounds up
    assert rq(31) == 0
    assert rq(33) == 1
    assert rq(96) == 2          # 1.5 -> 2
    assert rq(-32) == 0         # -0.5 -> 0 (half up, not away from zero)
    assert rq(-33) == -1
    assert rq(-96) == -1        # -1.5 -> -1
    assert rq(-97) == -2
    assert rq(-96, relu=True) == 0
    assert rq(64 * 40, hi=15) == 15
    assert rq(-64 * 40, lo=-8) == -8
    assert rq(0) == 0


def test_requant_matches_exact_rationals():
    g = np.random.default_rng(21)
    acc = g.integers(-(2 ** 31), 2 ** 31, size=(64, 8)).astype(np.int32)
    acc[0, :] = [-(2 ** 31), 2 ** 31 - 1, 0, 1, -1, 32, -32, 96]
    for shift in (1, 7, 20, 31, 40, 62):
        mult = g.integers(-(2 ** 31), 2 ** 31, size=8).astype(np.int32)
        mult[0] = 2 ** 31 - 1
        mult[1] = -(2 ** 31)
        for relu, lo, hi in ((True, 0, 15), (False, -128, 127), (False, -(2 ** 31), 2 ** 31 - 1)):
            got = oracle.requant(acc, mult, shift, relu, lo, hi)
            ref = np.array([[_exact_requant(int(a), int(mm), shift, relu, lo, hi)
                             for a, mm in zip(row, mult)] for row in acc])
            assert np.array_equal(got, ref)


def test_requant_bias_and_residual_closed_forms():
    """Bias is an accumulator offset added before scaling; the residual is added
    in output units after rounding and before ReLU and clipping."""
    m = np.full(1, 1 << 14, dtype=np.int32)      # scale 1/64 at shift 20

    def rq(a, bias=0, res=0, relu=False, lo=-1000, hi=1000):
        return int(oracle.requant(np.array([[a]], dtype=np.int32), m, 20, relu, lo, hi,
                                  bias=np.array([bias], dtype=np.int32),
                                  residual=np.array([[res]], dtype=np.int32))[0, 0])

    assert rq(0, bias=32) == 1                # the bias alone rounds: 32/64 = 0.5 -> 1
    assert rq(32, bias=-32) == 0              # cancels before scaling (after it would give 1 + 0 = 1)
    assert rq(64, bias=64 * 3) == 4           # (64 + 192) / 64
    assert rq(64, res=3) == 4                 # 1 + 3
    assert rq(-128, res=1, relu=True) == 0    # -2 + 1 = -1, then ReLU (ReLU first would give 1)
    assert rq(-128, res=3, relu=True) == 1    # -2 + 3
    assert rq(960, res=3, relu=True, lo=0, hi=15) == 15   # 15 + 3 saturates
    assert rq(31, res=0) == 0 and rq(31, bias=1) == 1     # the bias enters before the rounding
    assert rq(-33, bias=1, res=-1) == -1      # -32/64 -> 0, then -1


def test_requant_extensions_reduce_to_the_plain_epilogue():
    g = np.random.default_rng(22)
    acc = g.integers(-(2 ** 20), 2 ** 20, size=(32, 16)).astype(np.int32)
    mult = g.integers(1 << 14, 1 << 15, size=16).astype(np.int32)
    plain = oracle.requant(acc, mult, 20, True, 0, 15)
    zero_b = oracle.requant(acc, mult, 20, True, 0, 15, bias=np.zeros(16, np.int32))
    zero_r = oracle.requant(acc, mult, 20, True, 0, 15, residual=np.zeros_like(acc))
    assert np.array_equal(plain, zero_b) and np.array_equal(plain, zero_r)
    # a bias is the same as adding it to every accumulator of its channel
    bias = g.integers(-(2 ** 18), 2 ** 18, size=16).astype(np.int32)
    for relu, lo, hi in ((True, 0, 15), (False, -128, 127)):
        assert np.array_equal(oracle.requant(acc, mult, 20, relu, lo, hi, bias=bias),
                              oracle.requant(acc + bias, mult, 20, relu, lo, hi))
    # without clipping, a residual shifts the rounded result exactly
    res = g.integers(-8, 8, size=acc.shape).astype(np.int32)
    wide = (-(2 ** 31), 2 ** 31 - 1)
    assert np.array_equal(oracle.requant(acc, mult, 20, False, *wide, residual=res),
                          oracle.requant(acc, mult, 20, False, *wide) + res)


def test_requant_rejects_bad_shift():
    a = np.zeros((1, 1), dtype=np.int32)
    m = np.ones(1, dtype=np.int32)
    for sh in (0, 63, -1):
        with pytest.raises(oracle.OracleError):
            oracle.requant(a, m, sh, False, 0, 15)


# ----------------------------------------------------------------- packing

def test_pack_words_fixture():
    gold = json.load(open(os.path.join(GOLDEN, "pack_words.json")))
    for case in gold["cases"]:
        words = oracle.pack4(np.array(case["values"]), case["signed"])
        assert words.tolist() == [int(case["word"], 16)]
        assert oracle.unpack4(words, 8, case["signed"]).tolist() == case["values"]


@pytest.mark.parametrize("signed", [False, True])
def test_pack_unpack_roundtrip_all_values_all_positions(signed):
    vals = np.arange(-8, 8) if signed else np.arange(16)
    grid = np.array([[vals[(i + j) % 16] for i in range(8)] for j in range(16)]).reshape(-1)
    words = oracle.pack4(grid, signed)
    assert np.array_equal(oracle.unpack4(words, grid.size, signed), grid)
    # every nibble value occurs in every position
    for pos in range(8):
        assert sorted(((words >> (4 * pos)) & 0xF).tolist()) == list(range(16))


def test_pack_rejects_out_of_range():
    with pytest.raises(oracle.OracleError):
        oracle.pack4(np.array([16, 0, 0, 0, 0, 0, 0, 0]), False)
    with pytest.raises(oracle.OracleError):
        oracle.pack4(np.array([-9, 0, 0, 0, 0, 0, 0, 0]), True)


@pytest.mark.parametrize("bits,signed", [(4, False), (4, True), (8, True)])
def test_relayout_pack_is_saturated_transpose(bits, signed):
    g = np.random.default_rng(31)
    src = g.integers(-128, 128, size=(2, 16, 3, 5)).astype(np.int8)
    packed = oracle.relayout_pack(src, bits, signed)
    vals = oracle.unpack_tensor(packed, 16, bits, signed)
    lo = -(1 << (bits - 1)) if signed else 0
    hi = (1 << (bits - 1)) - 1 if signed else (1 << bits) - 1
    ref = np.clip(src.astype(np.int32), lo, hi).transpose(0, 2, 3, 1)
    assert np.array_equal(vals, ref)
    if bits == 4:
        assert packed.shape == (2, 3, 5, 2) and packed.dtype == np.uint32


def test_relayout_pack_word_layout_by_hand():
    """Pixel (0,0,0), channels 0..7 = 1..8 -> word 0x87654321; channels 8..15 -> second word."""
    src = np.zeros((1, 16, 1, 2), dtype=np.int8)
    src[0, :8, 0, 0] = np.arange(1, 9)
    src[0, 8:, 0, 1] = 15
    packed = oracle.relayout_pack(src, 4, False)
    assert packed.tolist() == [[[[0x87654321, 0], [0, 0xFFFFFFFF]]]]


def test_saturate():
    assert oracle.saturate(-5, 4, False) == 0
    assert oracle.saturate(20, 4, False) == 15
    assert oracle.saturate(-9, 4, True) == -8
    assert oracle.saturate(8, 4, True) == 7
    assert oracle.saturate(-128, 8, True) == -128


# ----------------------------------------------------------------- the composed layer

def test_qconv_layer_composes_the_steps():
    L = qi.scaled(qi.workload1()[0], n=1, h=9, w=11)
    t = qi.layer_tensors(1, 0, L)
    out = oracle.qconv_layer(t["x"], t["w"], bits=4, x_signed=False, w_signed=True,
                             stride=(1, 1), pad=(1, 1), mult=t["mult"], shift=20, relu=True, lo=0, hi=15)
    ref = _torch_conv(t["x"].astype(np.int32).transpose(0, 2, 3, 1), t["w"].astype(np.int32).transpose(0, 2, 3, 1),
                      (1, 1), (1, 1))
    assert np.array_equal(out["acc"].astype(np.float64), ref)
    y = oracle.unpack_tensor(out["y_packed"], L.k, 4, False)
    assert np.array_equal(y, out["y"])
    assert y.min() >= 0 and y.max() <= 15
