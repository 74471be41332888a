"""qconv2d_prepared_noalloc (the entry point for callers that cannot allocate)
against qconv2d_prepared with a caller-owned split-K workspace and against the
oracle, element by element: two calls in a row, the second on a smaller input,
then the first shape again (the library's scratch keeps the previous call's
contents; its arrival counters must be back at zero)."""
import ctypes

import numpy as np
import pytest

import qconv_inputs as qi
from _util import announce, assert_same, ref_layer, stress_shift

pytestmark = pytest.mark.gpu

# (layer, split-K factor): a deep layer split over its channel chunks, then a
# smaller one; 4-bit requantised and 8-bit raw accumulators
CASES = [
    (qi.Layer("na_4x14x14_256to256_3x3", 4, 14, 14, 256, 256, 3, 3, 1, 1, w_range=(-7, 7)), 4),
    (qi.Layer("na_1x7x7_128to128_3x3", 1, 7, 7, 128, 128, 3, 3, 1, 1, w_range=(-7, 7)), 2),
    (qi.Layer("na_2x9x9_256to64_3x3_s2_b8", 2, 9, 9, 256, 64, 3, 3, 2, 1, bits=8, x_signed=True, w_signed=True,
              x_range=qi.S8, w_range=qi.S8, epilogue=None), 3),
]


def _wide_tile(q, d, bits, splits):
    for t in q.tiles():
        if t["variant"] == 2 and t["bits"] == bits and t["chunk_c"] == 64 and q.tile_status(d, t["id"]) == 0 \
                and q.max_splits(d, t["id"]) >= splits:
            return t["id"]
    raise AssertionError("no wide tile for the case")


def _run(q, torch, L, splits, lid):
    dev = torch.device("cuda:0")
    t = qi.layer_tensors(70, lid, L)
    d = L.desc()
    requant = L.epilogue is not None
    shift = stress_shift(L, L.x_range, L.w_range) if requant else None
    xp = q.pack(torch.from_numpy(t["x"]).to(dev), L.bits, L.x_signed)
    wp = q.pack(torch.from_numpy(t["w"]).to(dev), L.bits, L.w_signed)
    tile = _wide_tile(q, d, L.bits, splits)
    wprep = q.prepare_filters(d, wp, tile)
    kw = {}
    if requant:
        kw = dict(requant=True, mult=torch.from_numpy(t["mult"]).to(dev), shift=shift, relu=True, clamp=(0, 15))
    announce(f"no-alloc {L.name} tile {tile} splits {splits}")
    y_na = q.conv2d(d, xp, wprep, tile=tile, prepared=True, splits=splits, noalloc=True, **kw)
    ws = q.make_workspace(d, tile, splits, dev)
    assert ws is not None, "the case must use split-K"
    y_ws = q.conv2d(d, xp, wprep, tile=tile, prepared=True, splits=splits, workspace=ws, **kw)
    torch.cuda.synchronize()
    ref = ref_layer(L, t, requant=requant, shift=shift)
    want = ref["y_packed"] if requant else ref["acc"]
    assert_same(y_na.cpu().numpy(), y_ws.cpu().numpy(), f"{L.name}: noalloc vs caller workspace")
    assert_same(y_na.cpu().numpy(), want, f"{L.name}: noalloc vs oracle")


def test_noalloc_matches_workspace_entry_and_oracle():
    torch = pytest.importorskip("torch")
    from paper_2202_06819_amd import qconv as q
    # the C-ABI symbol itself is what the binding calls
    assert hasattr(ctypes.CDLL(q.LIB_PATH), "qconv2d_prepared_noalloc")
    for lid, (L, splits) in enumerate(CASES):
        _run(q, torch, L, splits, lid)
    # the first (larger) shape once more, after the smaller ones
    _run(q, torch, CASES[0][0], CASES[0][1], 0)


def test_noalloc_rejects_oversized_split():
    torch = pytest.importorskip("torch")
    from paper_2202_06819_amd import qconv as q
    dev = torch.device("cuda:0")
    L = qi.Layer("na_big", 64, 56, 56, 256, 256, 3, 3, 1, 1)
    d = L.desc()
    tile = _wide_tile(q, d, 4, 4)
    x = torch.zeros(q.layout(d)["x_bytes"] // 4, dtype=torch.int32, device=dev)
    w = torch.zeros(q.prepared_filter_bytes(d, tile), dtype=torch.uint8, device=dev)
    with pytest.raises(q.QConvError) as ei:
        q.conv2d(d, x, w, tile=tile, prepared=True, splits=4, noalloc=True)
    assert ei.value.status == q.EWORKSPACE
