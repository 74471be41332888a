"""C-ABI checks that need no GPU: the library loads, exports every function
include/qconv.h declares, sizes match their closed forms, and every argument
error is reported before anything is launched.

Pointer arguments here are plain integers that are never dereferenced: every
call below is rejected by host-side validation first.
"""
import ctypes
import json
import os
import re

import pytest

import qconv_inputs as qi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qconv.h")


@pytest.fixture(scope="module")
def q():
    from paper_2202_06819_amd import build, qconv
    build.ensure_built()
    return qconv


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(qconv\w*)\s*\(", text, flags=re.M)))


def test_header_declares_the_boundary():
    names = _declared_functions()
    for must in ("qconv_layout", "qconv_pack", "qconv2d", "qconv_strerror"):
        assert must in names


def test_library_exports_every_declared_symbol(q):
    lib = ctypes.CDLL(q.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_selftest(q):
    assert q.selftest() == 0


def test_build_digest_matches_sources(q):
    from paper_2202_06819_amd import build
    assert q.build_digest() == build.source_digest() == build.built_digest()
    assert re.fullmatch(r"[0-9a-f]{16}", q.build_digest())


def test_noalloc_limits_and_oversized_split(q):
    """The no-alloc entry point states its scratch capacity and rejects a
    split-K whose partial sums exceed it on the host, before any device call."""
    lim = q.noalloc_limits()
    assert lim == {"scratch_bytes": (16 << 20) - (64 << 10), "max_tiles": 16384}
    d = q.make_desc(D(n=64, c=256, k=256))
    e = q.QConvEpilogue()
    e.mode = q.OUT_RAW_I32
    t = next(t["id"] for t in q.tiles() if t["variant"] == 2 and t["bits"] == 4 and q.tile_status(D(n=64, c=256, k=256), t["id"]) == 0)
    splits = q.max_splits(D(n=64, c=256, k=256), t)
    assert splits >= 2
    rc = q.lib().qconv2d_prepared_noalloc(ctypes.byref(d), 1 << 20, 2 << 20, 1 << 40, ctypes.byref(e), 1 << 40,
                                           t, splits, None)
    assert rc == q.EWORKSPACE, q.lib().qconv_last_error()
    assert b"no-alloc scratch" in q.lib().qconv_last_error()


def D(**kw):
    base = dict(n=8, h=56, w=56, c=64, k=64, r=3, s=3, stride_h=1, stride_w=1, pad_h=1, pad_w=1, bits=4,
                x_signed=0, w_signed=1)
    base.update(kw)
    return base


def test_layout_matches_table1(q):
    gold = json.load(open(os.path.join(ROOT, "tests", "golden", "table1_ops.json")))
    for st in gold["stages"]:
        info = q.layout(D(h=st["hw"], w=st["hw"], c=st["channels"], k=st["channels"]))
        assert (info["p"], info["q"]) == (st["hw"], st["hw"])
        assert 2 * info["macs"] == gold["ops_per_conv"]


def test_layout_sizes(q):
    info = q.layout(D())
    assert info["m"] == 8 * 56 * 56
    assert info["gemm_k"] == 576
    assert info["x_bytes"] == 8 * 56 * 56 * 32
    assert info["w_bytes"] == 64 * 9 * 32
    assert info["y_raw_bytes"] == 8 * 56 * 56 * 64 * 4
    assert info["y_packed_bytes"] == 8 * 56 * 56 * 32
    assert info["max_abs_acc"] == 576 * 15 * 8
    i8 = q.layout(D(bits=8, x_signed=1))
    assert i8["x_bytes"] == 8 * 56 * 56 * 64 and i8["y_packed_bytes"] == 8 * 56 * 56 * 64
    s2 = q.layout(D(stride_h=2, stride_w=2, r=1, s=1, pad_h=0, pad_w=0))
    assert (s2["p"], s2["q"]) == (28, 28)


@pytest.mark.parametrize("kw,status", [
    (dict(n=0), -1), (dict(h=-1), -1), (dict(c=0), -1), (dict(k=0), -1), (dict(r=0), -1),
    (dict(stride_h=0), -1), (dict(pad_w=-1), -1), (dict(h=2, pad_h=0), -1), (dict(x_signed=2), -1),
    (dict(bits=2), -2), (dict(bits=16), -2), (dict(c=12), -2), (dict(k=20), -2),
    (dict(bits=8, x_signed=0), -2), (dict(bits=8, x_signed=1, c=6), -2),
    (dict(c=4096, r=7, s=7, x_signed=1), -2),           # accumulator bound with the widening factor
    (dict(bits=8, x_signed=1, c=131072, r=1, s=1), -2), # 128*128*2^17 = 2^31
    # dimensions whose byte counts wrap 64 bits are rejected as too large
    (dict(n=1 << 30, h=1 << 30, w=1 << 30, c=64, r=1, s=1, pad_h=0, pad_w=0), -2),
    (dict(n=1 << 30, h=1 << 20, w=1 << 20, c=8, k=8, r=1, s=1, pad_h=0, pad_w=0), -2),
])
def test_descriptor_errors(q, kw, status):
    with pytest.raises(q.QConvError) as e:
        q.layout(D(**kw))
    assert e.value.status == status


def test_null_descriptor(q):
    assert q.lib().qconv_layout(None, None) == -1
    assert q.lib().qconv2d(None, 16, 16, None, 64, None, 0, -1, None) == -1


def _conv_call(q, d, x=1 << 32, w=1 << 33, y=1 << 34, epi=None, ws=None, wsb=0, tile=-1):
    desc = q.make_desc(d)
    return q.lib().qconv2d(ctypes.byref(desc), x, w, ctypes.byref(epi) if epi else None, y, ws, wsb, tile, None)


def _epi(q, **kw):
    e = q.QConvEpilogue()
    e.mode, e.mult, e.shift, e.relu, e.clamp_lo, e.clamp_hi = 1, 1 << 35, 20, 1, 0, 15
    for k, v in kw.items():
        setattr(e, k, v)
    return e


@pytest.mark.parametrize("kw", [dict(shift=0), dict(shift=63), dict(relu=2), dict(clamp_lo=5, clamp_hi=4),
                                dict(clamp_lo=0, clamp_hi=16), dict(clamp_lo=-8, clamp_hi=8),
                                dict(clamp_lo=-9, clamp_hi=0), dict(mode=7), dict(mult=None)])
def test_epilogue_errors(q, kw):
    assert _conv_call(q, D(), epi=_epi(q, **kw)) == -1


def test_int8_clamp_range(q):
    assert _conv_call(q, D(bits=8, x_signed=1), epi=_epi(q, clamp_lo=-129, clamp_hi=0)) == -1
    assert _conv_call(q, D(bits=8, x_signed=1), epi=_epi(q, clamp_lo=0, clamp_hi=128)) == -1


def test_pointer_errors(q):
    assert _conv_call(q, D(), x=0) == -1
    assert _conv_call(q, D(), y=0) == -1
    assert _conv_call(q, D(), x=(1 << 32) + 4) == -1    # misaligned
    assert _conv_call(q, D(), w=(1 << 33) + 8) == -1
    assert _conv_call(q, D(), y=(1 << 34) + 4) == -1
    assert _conv_call(q, D(), y=(1 << 32) + 4096) == -1  # y overlaps x
    assert _conv_call(q, D(), y=(1 << 33) - 64) == -1    # y overlaps w
    assert _conv_call(q, D(), tile=10 ** 6) == -1


def test_tile_errors(q):
    # a 4-bit tile cannot run an 8-bit layer
    t4 = [t["id"] for t in q.tiles() if t["bits"] == 4][0]
    assert q.tile_status(D(bits=8, x_signed=1), t4) == -2
    assert _conv_call(q, D(bits=8, x_signed=1), tile=t4) == -2
    # a very wide image does not fit the LDS band of any tile
    assert all(q.tile_status(D(w=20000, h=3), t["id"]) == -2 for t in q.tiles())
    with pytest.raises(q.QConvError):
        q.default_tile(D(w=20000, h=3))
    assert q.tile_status(D(), -5) == -1


def test_pack_errors(q):
    L = q.lib()
    assert L.qconv_pack(4096, 8192, 1, 12, 4, 4, 4, 0, None) == -2     # c % 8
    assert L.qconv_pack(4096, 8192, 1, 16, 4, 4, 5, 0, None) == -2     # bits
    assert L.qconv_pack(4096, 8192, 1, 16, 4, 4, 8, 0, None) == -2     # unsigned 8-bit
    assert L.qconv_pack(4096, 8192, -1, 16, 4, 4, 4, 0, None) == -1
    assert L.qconv_pack(0, 8192, 1, 16, 4, 4, 4, 0, None) == -1
    assert L.qconv_pack(4096, 4096 + 64, 1, 16, 4, 4, 4, 0, None) == -1   # overlap
    assert L.qconv_pack(4096, 8194, 1, 16, 4, 4, 4, 0, None) == -1        # dst misaligned
    assert L.qconv_pack(0, 0, 0, 16, 4, 4, 4, 0, None) == 0               # empty: no-op
    # sizes whose product wraps 64 bits (2^30 * 2^30 * 2^8 * 2^28 = 2^96) are too large, not small
    assert L.qconv_pack(4096, 1 << 40, 1 << 30, 1 << 30, 1 << 8, 1 << 28, 4, 0, None) == -2


def test_strerror_and_last_error(q):
    L = q.lib()
    assert L.qconv_strerror(0) == b"ok"
    assert L.qconv_strerror(-2) == b"unsupported configuration"
    with pytest.raises(q.QConvError):
        q.layout(D(c=12))
    assert b"c % 8" in L.qconv_last_error()


def test_tile_table_is_consistent(q):
    tiles = q.tiles()
    assert len(tiles) == q.lib().qconv_tile_count() >= 8
    for i, t in enumerate(tiles):
        assert t["id"] == i
        assert t["tile_p"] == 16 * t["waves_p"] * t["frag_p"]
        assert t["tile_k"] == 16 * t["waves_k"] * t["frag_k"]
        assert t["threads"] == 64 * t["waves_p"] * t["waves_k"]
        assert t["chunk_c"] % 64 == 0
        if t["bits"] == 4:
            assert t["frag_k"] % 2 == 0


def test_every_workload_layer_has_a_tile(q):
    for cfg, make in qi.WORKLOADS.items():
        for L in make():
            tid = q.default_tile(L.desc())
            assert q.tile_status(L.desc(), tid) == 0


def test_prepared_filter_bytes(q):
    d = D()
    info = q.layout(d)
    for t in q.tiles():
        if q.tile_status(d, t["id"]) != 0:
            continue
        n = q.prepared_filter_bytes(d, t["id"])
        if t["variant"] == 2:       # wide tiles: padded per-(K tile, chunk) images
            assert n >= info["gemm_k"] * d["k"]      # at least one int8 byte per filter weight
            assert n % 1024 == 0
        else:
            assert n == info["w_bytes"]
    assert q.prepared_filter_bytes(d, -1) == q.prepared_filter_bytes(d, q.default_tile(d))
    with pytest.raises(q.QConvError):
        q.prepared_filter_bytes(d, 10 ** 6)


def test_prepare_filters_errors(q):
    L = q.lib()
    d = D()
    desc = q.make_desc(d)
    tid = q.default_tile(d)
    need = q.prepared_filter_bytes(d, tid)
    ref = ctypes.byref(desc)
    assert L.qconv_prepare_filters(ref, 0, tid, 1 << 34, need, None) == -1            # NULL source
    assert L.qconv_prepare_filters(ref, 1 << 33, tid, 0, need, None) == -1            # NULL destination
    assert L.qconv_prepare_filters(ref, (1 << 33) + 4, tid, 1 << 34, need, None) == -1  # misaligned
    assert L.qconv_prepare_filters(ref, 1 << 33, tid, 1 << 34, need - 16, None) == -1   # too small
    assert L.qconv_prepare_filters(ref, 1 << 33, tid, (1 << 33) + 64, need, None) == -1  # overlap
    assert L.qconv_prepare_filters(ref, 1 << 33, 10 ** 6, 1 << 34, need, None) == -1    # unknown tile
    assert L.qconv_prepare_filters(None, 1 << 33, tid, 1 << 34, need, None) == -1


def test_conv_prepared_errors(q):
    L = q.lib()
    d = D()
    desc = q.make_desc(d)
    tid = q.default_tile(d)
    need = q.prepared_filter_bytes(d, tid)
    ref = ctypes.byref(desc)
    ok_epi = _epi(q)
    epi = ctypes.byref(ok_epi)
    # prepared buffer smaller than the tile's layout
    assert L.qconv2d_prepared(ref, 1 << 32, 1 << 33, need - 16, epi, 1 << 34, tid, 1, None, 0, None) == -1
    assert L.qconv2d_prepared(ref, 0, 1 << 33, need, epi, 1 << 34, tid, 1, None, 0, None) == -1
    assert L.qconv2d_prepared(ref, 1 << 32, 1 << 33, need, ctypes.byref(_epi(q, shift=0)), 1 << 34, tid, 1, None, 0,
                              None) == -1
    assert L.qconv2d_prepared(None, 1 << 32, 1 << 33, need, None, 1 << 34, tid, 1, None, 0, None) == -1


def _wide_tile(q, d):
    return [t["id"] for t in q.tiles() if t["variant"] == 2 and q.tile_status(d, t["id"]) == 0][0]


def test_split_k_workspace(q):
    d = D(h=7, w=7, c=512, k=512, n=2)
    tid = _wide_tile(q, d)
    chunks = q.max_splits(d, tid)
    assert chunks == 512 // [t for t in q.tiles() if t["id"] == tid][0]["chunk_c"]
    assert q.workspace_bytes(d, tid, 1) == 0
    info = q.layout(d)
    t = q.tiles()[tid]
    mt = -(-info["m"] // t["tile_p"])
    kt = -(-d["k"] // t["tile_k"])
    for s in (2, chunks):
        n = q.workspace_bytes(d, tid, s)
        assert n >= mt * kt * s * t["tile_p"] * t["tile_k"] * 4 + mt * kt * 4
    with pytest.raises(q.QConvError):
        q.workspace_bytes(d, tid, chunks + 1)
    staged = [x["id"] for x in q.tiles() if x["variant"] == 0 and q.tile_status(d, x["id"]) == 0]
    if staged:
        assert q.max_splits(d, staged[0]) == 1
        with pytest.raises(q.QConvError):
            q.workspace_bytes(d, staged[0], 2)


def test_split_k_errors(q):
    L = q.lib()
    d = D(h=7, w=7, c=512, k=512, n=2)
    tid = _wide_tile(q, d)
    desc = q.make_desc(d)
    need = q.prepared_filter_bytes(d, tid)
    wsb = q.workspace_bytes(d, tid, 2)
    epi = ctypes.byref(_epi(q))
    ref = ctypes.byref(desc)
    args = (ref, 1 << 32, 1 << 33, need, epi, 1 << 34, tid)
    assert L.qconv2d_prepared(*args, 2, None, 0, None) == -3                 # no workspace
    assert L.qconv2d_prepared(*args, 2, 1 << 35, wsb - 16, None) == -3       # too small
    assert L.qconv2d_prepared(*args, 2, (1 << 35) + 8, wsb, None) == -1      # misaligned
    assert L.qconv2d_prepared(*args, 2, (1 << 32) + 64, wsb, None) == -1     # overlaps x
    assert L.qconv2d_prepared(*args, 10 ** 6, 1 << 35, wsb, None) == -2      # more splits than chunks
    assert L.qconv2d_prepared(*args, 0, None, 0, None) == -2


def test_grid_meet_probe_argument_errors(q):
    # rejected before any device is queried or anything is enqueued
    L = q.lib()
    a, e = 1 << 32, (1 << 32) + 4 * 144
    assert L.qconv_probe_grid_meet(0, 1, 0, a, e, None) == -1
    assert L.qconv_probe_grid_meet(1, -1, 0, a, e, None) == -1
    assert L.qconv_probe_grid_meet(1, 4097, 0, a, e, None) == -1
    assert L.qconv_probe_grid_meet(1, 1, 2, a, e, None) == -1
    assert L.qconv_probe_grid_meet(1, 1, 0, None, e, None) == -1
    assert L.qconv_probe_grid_meet(1, 1, 0, a + 2, e, None) == -1
    assert L.qconv_probe_grid_meet(1, 1, 1, a, None, None) == -1


def test_mfma_probe_shape_argument_errors(q):
    L = q.lib()
    ops = ctypes.c_int64(0)
    assert L.qconv_probe_mfma_i8_shape(2, 1, 1, 1 << 32, 1 << 33, ctypes.byref(ops), None) == -1
    assert L.qconv_probe_mfma_i8_shape(-1, 1, 1, 1 << 32, 1 << 33, ctypes.byref(ops), None) == -1
    assert L.qconv_probe_mfma_i8_shape(1, 0, 1, 1 << 32, 1 << 33, ctypes.byref(ops), None) == -1
    assert L.qconv_probe_mfma_i8_shape(1, 1, 1, None, 1 << 33, ctypes.byref(ops), None) == -1


def test_mfma_probe_argument_errors(q):
    L = q.lib()
    ops = ctypes.c_int64(0)
    assert L.qconv_probe_mfma_i8(0, 1, 1 << 32, 1 << 33, ctypes.byref(ops), None) == -1
    assert L.qconv_probe_mfma_i8(1, 0, 1 << 32, 1 << 33, ctypes.byref(ops), None) == -1
    assert L.qconv_probe_mfma_i8((1 << 20) + 1, 1, 1 << 32, 1 << 33, ctypes.byref(ops), None) == -1
    assert L.qconv_probe_mfma_i8(1, 1, None, 1 << 33, ctypes.byref(ops), None) == -1
    assert L.qconv_probe_mfma_i8(1, 1, 1 << 32, (1 << 33) + 4, ctypes.byref(ops), None) == -1
    assert ops.value == 0


def test_schedule_check_and_errors(q):
    L = q.lib()
    d = D(h=14, w=14, c=256, k=256, n=4)
    tid = _wide_tile(q, d)
    staged = [t["id"] for t in q.tiles() if t["variant"] == 0 and q.tile_status(d, t["id"]) == 0][0]
    base = {"tile_id": tid}
    assert q.schedule_status(d, base) == 0
    assert q.schedule_status(d, dict(base, splits=q.max_splits(d, tid), wg_per_cu=3, band_buffers=1,
                                     xcd_order=0)) == 0
    assert q.schedule_status(d, dict(base, wg_per_cu=17)) == -1
    assert q.schedule_status(d, dict(base, wg_per_cu=-1)) == -1
    assert q.schedule_status(d, dict(base, band_buffers=3)) == -1
    assert q.schedule_status(d, dict(base, xcd_order=2)) == 0
    assert q.schedule_status(d, dict(base, xcd_order=-1)) == 0
    assert q.schedule_status(d, dict(base, xcd_order=3)) == -1
    assert q.schedule_status(d, dict(base, xcd_order=-2)) == -1
    assert q.schedule_status(d, dict(base, splits=0)) == -2
    assert q.schedule_status(d, dict(base, splits=q.max_splits(d, tid) + 1)) == -2
    assert q.schedule_status(d, {"tile_id": staged, "splits": 2}) == -2
    assert q.schedule_status(d, {"tile_id": 10 ** 6}) < 0
    assert q.schedule_status(D(bits=8, x_signed=1), base) == -2     # tile built for 4-bit
    desc = q.make_desc(d)
    need = q.prepared_filter_bytes(d, tid)
    args = (ctypes.byref(desc), 1 << 32, 1 << 33, need, ctypes.byref(_epi(q)), 1 << 34)
    assert L.qconv2d_scheduled(*args, None, None, 0, None) == -1          # no schedule
    bad = q.make_schedule(dict(base, band_buffers=5))
    assert L.qconv2d_scheduled(*args, ctypes.byref(bad), None, 0, None) == -1
    two = q.make_schedule(dict(base, splits=2))
    assert L.qconv2d_scheduled(*args, ctypes.byref(two), None, 0, None) == -3   # split-K without workspace


def test_bias_and_residual_argument_errors(q):
    L = q.lib()
    d = D()
    desc = q.make_desc(d)
    info = q.layout(d)
    ref = ctypes.byref(desc)
    x, w, y = 1 << 32, 1 << 33, 1 << 34
    raw = _epi(q, mode=0, bias=1 << 36)
    assert L.qconv2d(ref, x, w, ctypes.byref(raw), y, None, 0, -1, None) == -1           # raw mode takes no bias
    assert L.qconv2d(ref, x, w, ctypes.byref(_epi(q, residual=(1 << 36) + 8)), y, None, 0, -1, None) == -1
    assert L.qconv2d(ref, x, w, ctypes.byref(_epi(q, residual=1 << 36, residual_signed=2)), y, None, 0, -1,
                     None) == -1
    part = _epi(q, residual=y + 16 * (info["y_packed_bytes"] // 32))                   # overlaps y, is not y
    assert L.qconv2d(ref, x, w, ctypes.byref(part), y, None, 0, -1, None) == -1
    over_x = _epi(q, residual=x + 64)
    assert L.qconv2d(ref, x, w, ctypes.byref(over_x), y, None, 0, -1, None) == -1


def test_ablation_schedules(q):
    d = D(n=2)
    names = {t["name"]: t["id"] for t in q.tiles()}
    for name in ("wide_b4_w4x1_f1x4_c64", "wide_b4_w8x1_f1x4_c64", "wide_b4_w4x1_f2x4_c64"):
        for mask in range(1, 8):
            assert q.schedule_status(d, {"tile_id": names[name], "ablation": mask}) == 0, (name, mask)
    assert q.schedule_status(d, {"tile_id": names["wide_b4_w4x1_f4x4_c64"], "ablation": 1}) == -2   # not compiled
    assert q.schedule_status(d, {"tile_id": names["wide_b4_w4x1_f1x4_c64"], "ablation": 8}) == -1
    # keeping the band packed halves its LDS: with the int32 tile also in LDS,
    # the lowered operand of a deeper layer fits only packed
    deep = D(n=2, h=28, w=28, c=128, k=128)
    t = names["wide_b4_w8x1_f1x4_c64"]
    assert q.schedule_status(deep, {"tile_id": t, "ablation": 3}) == -2
    assert q.schedule_status(deep, {"tile_id": t, "ablation": 7}) == 0
    assert q.schedule_status(D(bits=8, x_signed=1), {"tile_id": t, "ablation": 4}) == -2
    assert q.schedule_status(D(r=1, s=1, pad_h=0, pad_w=0), {"tile_id": names["wide_b4_w4x1_f1x4_c64"],
                                                           "ablation": 1}) == -2              # 3x3 only


def test_unroll_argument_errors(q):
    L = q.lib()
    src, dst = 1 << 32, 1 << 34
    rows = (1, 1, 0, 8)   # taps_h, stride_h, pad_h, out_h: width unrolling only

    def call(s, d, n, c, h, w, rows, cols, c_out):
        return L.qconv_unroll(s, d, n, c, h, w, *rows, *cols, c_out, None)

    assert call(src, dst, 1, 3, 8, 8, rows, (7, 2, 3), 20) == -1          # c_out not a multiple of 16
    assert call(src, dst, 1, 3, 8, 8, rows, (7, 2, 3), 16) == -1          # 7 * 3 > 16
    assert call(src, dst, 1, 3, 8, 8, (7, 2, 3, 4), (7, 2, 3), 144) == -1  # 7 * 7 * 3 > 144
    assert call(src, dst, 1, 3, 8, 8, rows, (0, 2, 3), 32) == -1          # no taps
    assert call(src, dst, 1, 3, 8, 8, (1, 0, 0, 8), (7, 2, 3), 32) == -1  # row stride 0
    assert call(src, dst, 1, 3, 8, 8, (1, 1, -1, 8), (7, 2, 3), 32) == -1 # negative row padding
    assert call(src, dst, 1, 3, 8, 8, (1, 1, 0, -1), (7, 2, 3), 32) == -1 # negative row count
    assert call(src, dst, 1, 3, 8, 2, rows, (7, 1, 0), 32) == -1          # window wider than the input
    assert call(src, dst + 8, 1, 3, 8, 8, rows, (7, 2, 3), 32) == -1      # misaligned
    assert call(src, src + 64, 1, 3, 8, 8, rows, (7, 2, 3), 32) == -1     # overlap
    assert call(None, dst, 1, 3, 8, 8, rows, (7, 2, 3), 32) == -1         # NULL source of a non-empty input
    assert call(src, dst, 1, 64, 8, 4000, (8, 1, 0, 8), (1, 1, 0), 512) == -2   # stages more than 64 KiB per row
    assert call(None, None, 0, 3, 8, 8, rows, (7, 2, 3), 32) == 0         # empty: no-op
    # row arithmetic and byte counts that would leave 32 (or wrap 64) bits
    assert call(src, dst, 1, 3, 8, 8, (1, 1 << 20, 0, 1 << 12), (7, 2, 3), 32) == -2
    assert call(src, dst, 1 << 30, 16, 1 << 30, 64, (1, 1, 0, 1 << 30), (1, 1, 0), 16) == -2
    assert call(src, None, 1, 3, 8, 8, (1, 1, 0, 0), (7, 2, 3), 32) == 0  # no output rows: no-op


def test_few_channel_plan_shapes(q):
    """The folding plans of the 7x7 stride-2 stem: the unrolled shapes and the
    equivalent convolution (the arithmetic is checked in test_oracle and on
    the GPU)."""
    d = dict(n=2, h=224, w=224, c=3, k=64, r=7, s=7, stride_h=2, stride_w=2, pad_h=3, pad_w=3, bits=8, x_signed=1,
             w_signed=1)
    rows = q.few_channel_plan(d, 64, "rows")
    assert rows["x"] == dict(taps_h=2, stride_h=2, pad_h=3, out_h=115, taps_w=7, stride_w=2, pad_w=3)
    assert rows["w"] == dict(taps_h=2, stride_h=2, pad_h=0, out_h=4, taps_w=7, stride_w=1, pad_w=0)
    assert (rows["desc"]["h"], rows["desc"]["w"], rows["desc"]["c"], rows["desc"]["r"], rows["desc"]["s"]) == \
        (115, 112, 64, 4, 1)
    assert q.layout(rows["desc"])["p"] == 112 and q.layout(rows["desc"])["q"] == 112
    full = q.few_channel_plan(d, 192, "all")
    assert full["x"] == dict(taps_h=7, stride_h=2, pad_h=3, out_h=112, taps_w=7, stride_w=2, pad_w=3)
    assert full["w"] == dict(taps_h=7, stride_h=1, pad_h=0, out_h=1, taps_w=7, stride_w=1, pad_w=0)
    assert (full["desc"]["h"], full["desc"]["r"], full["desc"]["stride_h"], full["desc"]["pad_h"]) == (112, 1, 1, 0)
    with pytest.raises(q.QConvError):
        q.few_channel_plan(d, 64, "cols")


def test_interleaved_layout_rules(q):
    """The batch-interleaved layout: sizes equal the plain layout's, n must
    divide by nb, stride_w must be 1, and only the wide tiles' generic
    kernels read it (no staged tile, no ablation instance)."""
    plain = q.layout(D())
    for nb in (2, 4, 8):
        assert q.layout(D(nb=nb)) == plain
    assert q.layout(D(nb=0)) == plain and q.layout(D(nb=1)) == plain
    with pytest.raises(q.QConvError) as e:
        q.layout(D(nb=3))
    assert e.value.status == -1
    with pytest.raises(q.QConvError) as e:
        q.layout(D(nb=-1))
    assert e.value.status == -1
    with pytest.raises(q.QConvError) as e:
        q.layout(D(nb=2, stride_h=2, stride_w=2))
    assert e.value.status == -2
    assert q.layout(D(nb=2, stride_h=2, stride_w=1))["p"] == 28        # row stride alone is fine
    usable = 0
    for t in q.tiles():
        st = q.tile_status(D(nb=4), t["id"])
        if t["variant"] != 2:
            assert st == -2, t["name"]
        usable += st == 0
    assert usable >= 4
    names = {t["name"]: t["id"] for t in q.tiles()}
    assert q.schedule_status(D(nb=4), {"tile_id": names["wide_b4_w4x1_f1x4_c64"], "ablation": 1}) == -2
    from paper_2202_06819_amd import sweep
    assert sweep.shape_key(D(nb=4)) != sweep.shape_key(D()) and sweep.shape_key(D(nb=1)) == sweep.shape_key(D())


def test_pack_interleaved_argument_errors(q):
    L = q.lib()
    src, dst = 1 << 32, 1 << 34
    assert L.qconv_pack_interleaved(src, dst, 6, 64, 8, 8, 4, 0, 4, None) == -1   # 4 does not divide 6
    assert L.qconv_pack_interleaved(src, dst, 6, 64, 8, 8, 4, 0, 0, None) == -1   # nb 0
    assert L.qconv_pack_interleaved(src, dst, 4, 60, 8, 8, 4, 0, 2, None) == -2   # c % 8 for 4-bit
    assert L.qconv_pack_interleaved(src, dst + 2, 4, 64, 8, 8, 4, 0, 2, None) == -1   # misaligned
    assert L.qconv_pack_interleaved(None, None, 0, 64, 8, 8, 4, 0, 2, None) == 0  # empty: no-op


def test_fused_pack_argument_errors(q):
    """qconv2d_packing rejects what its fused instance does not run, before
    anything is launched."""
    import ctypes as C
    L = q.lib()
    names = {t["name"]: t["id"] for t in q.tiles()}
    tid = names["wide_b4_w4x2_f2x2_c64"]
    x, xp, w, y = 1 << 32, 1 << 33, 1 << 34, 1 << 35
    epi = q.QConvEpilogue()
    epi.mode = 0

    def call(d, x_=x, xp_=xp, tile=tid):
        desc = q.make_desc(d)
        wb = q.prepared_filter_bytes(d, tile) if q.tile_status(d, tile) == 0 else 1 << 20
        return L.qconv2d_packing(C.byref(desc), x_, xp_, w, wb, C.byref(epi), y, tile, None)

    assert call(D(n=2), x_=None) == -1                                   # no input
    assert call(D(n=2, r=1, s=1, pad_h=0, pad_w=0)) == -2                # no 1x1 fused instance
    assert call(D(n=2), tile=names["staged_b4_w4x1_f1x4_c64"]) == -2     # staged tile
    assert call(D(n=2, nb=2)) == -2                                      # interleaved layout
    assert call(D(n=2, stride_h=4, stride_w=4)) == -2                    # bands skip rows: no packed copy
    assert call(D(n=2), xp_=xp + 8) == -1                                # misaligned packed copy
    assert call(D(n=2), xp_=x + 64) == -1                                # packed copy overlaps x


def test_projection_entry_points_validate_on_the_host(q):
    """Shapes a fused projection cannot ride on are refused before any launch."""
    d = D(n=2, h=9, w=9, stride_h=2, stride_w=2)
    t = q.proj_default_tile(d)
    assert q.proj_tile_status(d, t) == q.OK
    assert q.tiles()[t]["name"] in {"wide_b4_w4x2_f2x2_c64", "wide_b4_w2x2_f2x2_c64", "wide_b4_w4x1_f2x4_c64",
                                    "wide_b4_w4x2_f2x2_c128"}
    assert q.proj_tile_status(D(pad_h=0, pad_w=0), t) == q.EUNSUPPORTED        # the centre tap moves
    assert q.proj_tile_status(D(r=1, s=1, pad_h=0, pad_w=0), t) == q.EUNSUPPORTED
    assert q.proj_tile_status(D(nb=2), t) == q.EUNSUPPORTED
    staged = next(tt["id"] for tt in q.tiles() if tt["variant"] == 0 and tt["bits"] == 4)
    assert q.proj_tile_status(d, staged) == q.EUNSUPPORTED
    # the image carries one more tap than the plain 3x3 image of the same tile
    plain = q.prepared_filter_bytes(d, t)
    n = ctypes.c_size_t(0)
    assert q.lib().qconv_prepared_proj_filter_bytes(ctypes.byref(q.make_desc(d)), t, ctypes.byref(n)) == q.OK
    assert n.value >= plain
    # mismatched epilogue modes and residuals are refused
    desc = q.make_desc(d)
    raw, rq = q.QConvEpilogue(), q.QConvEpilogue()
    raw.mode = q.OUT_RAW_I32
    rq.mode, rq.mult, rq.shift, rq.relu, rq.clamp_lo, rq.clamp_hi = q.OUT_REQUANT, 1 << 20, 20, 1, 0, 15
    args = (ctypes.byref(desc), 1 << 20, 2 << 20, 1 << 30)
    assert q.lib().qconv2d_proj(*args, ctypes.byref(raw), 3 << 20, ctypes.byref(rq), 4 << 20, t, 1, None, 0,
                                None) == -1
    rq2 = q.QConvEpilogue.from_buffer_copy(rq)
    rq2.residual = 5 << 20
    assert q.lib().qconv2d_proj(*args, ctypes.byref(rq), 3 << 20, ctypes.byref(rq2), 4 << 20, t, 1, None, 0,
                                None) == q.EUNSUPPORTED
    assert q.lib().qconv2d_proj(*args, ctypes.byref(rq), 3 << 20, ctypes.byref(rq), None, t, 1, None, 0,
                                None) == -1
    # split-K (over 64-channel chunks): the projection's partial sums double the
    # workspace; a missing one is refused
    d2 = D(n=2, h=9, w=9, c=256, stride_h=2, stride_w=2)
    t2 = next(tt["id"] for tt in q.tiles() if tt["name"] == "wide_b4_w4x2_f2x2_c64")
    assert q.proj_tile_status(d2, t2) == q.OK
    assert q.proj_workspace_bytes(d2, t2, 1) == 0
    assert q.max_splits(d2, t2) == 4
    plain_ws, proj_ws = q.workspace_bytes(d2, t2, 2), q.proj_workspace_bytes(d2, t2, 2)
    assert plain_ws < proj_ws < 2 * plain_ws
    desc2 = q.make_desc(d2)
    args2 = (ctypes.byref(desc2), 1 << 20, 2 << 20, 1 << 30)
    assert q.lib().qconv2d_proj(*args2, ctypes.byref(rq), 3 << 20, ctypes.byref(rq), 4 << 20, t2, 2, None, 0,
                                None) == q.EWORKSPACE
    with pytest.raises(q.QConvError):
        q.proj_workspace_bytes(d2, t2, 5)


def test_validation_fuzz(q):
    """Random and extreme descriptor fields, tile ids, split factors and
    schedule knobs into every host-side query: each returns a status (no
    crash), and for shapes a tile runs, the split-K queries are consistent
    (at least one chunk, no workspace without a split)."""
    import random
    L = q.lib()
    fields = [f for f, _ in q.QConvDesc._fields_]
    knobs = [f for f, _ in q.QConvSchedule._fields_]
    extreme = [-(1 << 31), -(1 << 30), -7, -1, 0, 1, 2, 3, 4, 7, 8, 9, 15, 16, 31, 32, 63, 64, 65, 128, 1000, 4096,
               1 << 16, 1 << 20, 1 << 30, (1 << 31) - 1]
    base = dict(n=2, h=14, w=14, c=64, k=64, r=3, s=3, stride_h=1, stride_w=1, pad_h=1, pad_w=1, bits=4, x_signed=0,
                w_signed=1, nb=0)
    nt = L.qconv_tile_count()
    rng = random.Random(11)
    valid = running = 0
    for _ in range(3000):
        d = dict(base)
        for f in fields:
            u = rng.random()
            if u < 0.15:
                d[f] = rng.choice(extreme)
            elif u < 0.3:
                d[f] = rng.randint(-3, 300)
        desc = q.QConvDesc(**d)
        info = q.QConvLayoutInfo()
        rc = L.qconv_layout(ctypes.byref(desc), ctypes.byref(info))
        assert rc <= 0
        valid += rc == 0
        n = ctypes.c_size_t(0)
        for tile in (rng.choice([-7, -1, 0, nt - 1, nt, 1 << 20]), rng.randrange(nt)):
            st = L.qconv_tile_check(ctypes.byref(desc), tile)
            ms = L.qconv_max_splits(ctypes.byref(desc), tile)
            assert st <= 0
            if st == 0:
                running += 1
                assert rc == 0 and ms >= 1
                assert L.qconv_workspace_bytes(ctypes.byref(desc), tile, 1, ctypes.byref(n)) == 0 and n.value == 0
            assert L.qconv_workspace_bytes(ctypes.byref(desc), tile, rng.choice([-1, 0, 2, 3, 64, 1 << 20]),
                                           ctypes.byref(n)) <= 0
            assert L.qconv_prepared_filter_bytes(ctypes.byref(desc), tile, ctypes.byref(n)) <= 0
            assert L.qconv_proj_tile_check(ctypes.byref(desc), tile) <= 0
            assert L.qconv_proj_workspace_bytes(ctypes.byref(desc), tile, rng.choice([-1, 0, 1, 2, 7]),
                                                ctypes.byref(n)) <= 0
            sch = q.QConvSchedule(**{k: rng.choice([-(1 << 31), -1, 0, 1, 2, 3, 4, 8, 1 << 20, (1 << 31) - 1, tile])
                                     for k in knobs})
            assert L.qconv_schedule_check(ctypes.byref(desc), ctypes.byref(sch)) <= 0
        L.qconv_default_tile(ctypes.byref(desc))
        L.qconv_proj_default_tile(ctypes.byref(desc))
    assert valid > 100 and running > 50
