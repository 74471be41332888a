"""Helpers shared by the GPU parity tests: run a layer through the HIP path and
through the oracle on the same seeded inputs."""
from __future__ import annotations

import os
import sys

import numpy as np

import oracle
import qconv_inputs as qi


def announce(msg: str) -> None:
    """Name the case before a GPU step (a crash then still says which one)."""
    print(f"\n[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def oracle_threads() -> int:
    return max(1, min(16, oracle.max_threads()))


def stress_shift(L: qi.Layer, x_range, w_range, mult_mid: float = 2 ** 14.5, target: float = None) -> int:
    """A shift that spreads requantised outputs over the clamp range for
    zero-mean filters: the accumulator's spread is about sqrt(C*R*S) times the
    spread of one product.  (Input statistics only; nothing of the method.)"""
    xv = np.arange(x_range[0], x_range[1] + 1, dtype=np.float64)
    wv = np.arange(w_range[0], w_range[1] + 1, dtype=np.float64)
    spread = np.sqrt(L.c * L.r * L.s * (xv ** 2).mean() * (wv ** 2).mean())
    target = target or (8.0 if L.bits == 4 else 64.0)
    return int(max(1, min(62, round(np.log2(spread * mult_mid / target)))))


def ref_layer(L: qi.Layer, t: dict, *, requant: bool, shift=None, relu=None, lo=None, hi=None, threads=None,
              packed_x=None) -> dict:
    e = L.epilogue or qi.Epilogue()
    kw = {}
    if requant:
        kw = dict(mult=t["mult"], shift=e.shift if shift is None else shift, relu=e.relu if relu is None else relu,
                  lo=e.lo if lo is None else lo, hi=e.hi if hi is None else hi)
    return oracle.qconv_layer(t["x"], t["w"], bits=L.bits, x_signed=L.x_signed, w_signed=L.w_signed,
                              stride=(L.stride, L.stride), pad=(L.pad, L.pad), threads=threads or oracle_threads(),
                              packed_x=packed_x, **kw)


def as_u32(a) -> np.ndarray:
    return np.ascontiguousarray(a).view(np.uint32) if a.dtype in (np.int32, np.uint32) else np.ascontiguousarray(a)


def gpu_layer(L: qi.Layer, t: dict, *, requant: bool, tile: int = -1, shift=None, relu=None, lo=None, hi=None,
              x_packed_dev=None, prepared: bool = False):
    """Pack x and w on the GPU, run the conv (from packed filters, or from
    filters prepared for `tile`); returns host numpy arrays."""
    import torch
    from paper_2202_06819_amd import qconv

    dev = torch.device("cuda:0")
    e = L.epilogue or qi.Epilogue()
    if x_packed_dev is None:
        x_dev = torch.from_numpy(t["x"]).to(dev)
        xp = qconv.pack(x_dev, L.bits, L.x_signed)
    else:
        xp = x_packed_dev
    w_dev = torch.from_numpy(t["w"]).to(dev)
    wp = qconv.pack(w_dev, L.bits, L.w_signed)
    kw = {}
    if requant:
        kw = dict(requant=True, mult=torch.from_numpy(t["mult"]).to(dev), shift=e.shift if shift is None else shift,
                  relu=e.relu if relu is None else relu,
                  clamp=(e.lo if lo is None else lo, e.hi if hi is None else hi))
    if prepared:
        tile = qconv.default_tile(L.desc()) if tile == -1 else tile
        wprep = qconv.prepare_filters(L.desc(), wp, tile)
        y = qconv.conv2d(L.desc(), xp, wprep, tile=tile, prepared=True, **kw)
    else:
        y = qconv.conv2d(L.desc(), xp, wp, tile=tile, **kw)
    torch.cuda.synchronize()
    return {"x_packed": xp.cpu().numpy(), "w_packed": wp.cpu().numpy(), "y": y.cpu().numpy(), "y_dev": y}


def assert_same(got: np.ndarray, ref: np.ndarray, what: str) -> None:
    g = as_u32(got)
    r = as_u32(ref)
    assert g.shape == r.shape, f"{what}: shape {g.shape} vs {r.shape}"
    if not np.array_equal(g, r):
        bad = np.argwhere(g != r)
        raise AssertionError(f"{what}: {len(bad)} of {g.size} elements differ; first at {bad[0].tolist()}: "
                             f"got {g[tuple(bad[0])]} want {r[tuple(bad[0])]}")


def unroll_def(src, c_out, taps_h, stride_h, pad_h, out_h, taps_w, stride_w, pad_w):
    """The patch unroll of include/qconv.h written out with numpy:
    dst[n][u][q][(b*taps_w + s)*c + ci] = src[n][ci][u*stride_h + b - pad_h][q*stride_w + s - pad_w],
    0 outside the input and for channels from taps_h*taps_w*c on."""
    n, c, h, w = src.shape
    wout = (w + 2 * pad_w - taps_w) // stride_w + 1
    dst = np.zeros((n, out_h, wout, c_out), dtype=np.int8)
    u, q = np.arange(out_h), np.arange(wout)
    for b in range(taps_h):
        y = u * stride_h + b - pad_h
        uu = np.nonzero((y >= 0) & (y < h))[0]
        for s in range(taps_w):
            col = q * stride_w + s - pad_w
            qq = np.nonzero((col >= 0) & (col < w))[0]
            base = (b * taps_w + s) * c
            # src[:, :, y, col] -> n x c x |uu| x |qq|, moved to n x |uu| x |qq| x c
            block = src[:, :, y[uu]][:, :, :, col[qq]]
            dst[:, uu[:, None], qq[None, :], base:base + c] = block.transpose(0, 2, 3, 1)
    return dst


def random_layer(seed: int, big: bool) -> qi.Layer:
    """A random layer of the random-shape parity tests: ragged sizes, strides
    1-3, paddings beyond the filter's half width, 1x1 to 7x7 filters (some
    non-square), 4-bit or 8-bit operands of either signedness; `big` allows
    batches up to 24 and 60 pixels a side."""
    g = np.random.default_rng([4242, seed])
    bits = 8 if seed % 3 == 2 else 4
    r = int(g.choice([1, 1, 3, 3, 3, 5, 7, 2]))
    s = int(g.choice([r, r, r, 1, 3]))
    stride = int(g.choice([1, 1, 1, 2, 2, 3]))
    pad = int(g.integers(0, max(r, s) // 2 + 2))
    h = int(g.integers(max(1, r - 2 * pad), 61 if big else 40))
    w = int(g.integers(max(1, s - 2 * pad), 61 if big else 40))
    n = int(g.integers(1, 25 if big else 6))
    if bits == 4:
        c, k = 8 * int(g.integers(1, 48)), 8 * int(g.integers(1, 40))
        xs, ws = bool(g.random() < 0.2), bool(g.random() < 0.85)
        signed_out = bool(g.random() < 0.4)
        epi = qi.Epilogue(relu=bool(g.random() < 0.5), lo=-8 if signed_out else 0, hi=7 if signed_out else 15)
        return qi.Layer(f"rand{seed}", n, h, w, c, k, r, s, stride, pad, 4, xs, ws, qi.S4 if xs else qi.U4,
                        qi.S4 if ws else qi.U4, epi)
    c, k = 4 * int(g.integers(1, 96)), 4 * int(g.integers(1, 80))
    epi = qi.Epilogue(relu=bool(g.random() < 0.5), lo=-128, hi=127)
    return qi.Layer(f"rand{seed}", n, h, w, c, k, r, s, stride, pad, 8, True, True, qi.S8, qi.S8, epi)
