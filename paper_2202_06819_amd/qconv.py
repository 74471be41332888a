"""ctypes binding of libqconv: argument marshalling only.

Every step of the path runs in the HIP kernels behind the C ABI
(``include/qconv.h``).  PyTorch supplies device memory and the stream; this
module turns tensors into pointers and sizes and status codes into
exceptions.  There is no fallback: if ``libqconv.so`` is missing or a call
fails, an exception is raised.

Tensor conventions
  4-bit packed tensors are torch.int32 with the last axis = channels / 8 (each
  element holds eight nibbles, channel 8j+i in bits [4i, 4i+3]); 8-bit tensors
  are torch.int8 with the last axis = channels; raw accumulators are
  torch.int32 N x P x Q x K.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

from .build import LIB as LIB_PATH
from .build import source_digest

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP = 0, -1, -2, -3, -4
OUT_RAW_I32, OUT_REQUANT = 0, 1

_i32, _i64, _vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p


class QConvDesc(ctypes.Structure):
    _fields_ = [(f, _i32) for f in ("n", "h", "w", "c", "k", "r", "s", "stride_h", "stride_w", "pad_h", "pad_w",
                                    "bits", "x_signed", "w_signed", "nb")]


class QConvLayoutInfo(ctypes.Structure):
    _fields_ = [("p", _i32), ("q", _i32)] + [(f, _i64) for f in (
        "m", "gemm_k", "macs", "x_bytes", "w_bytes", "y_raw_bytes", "y_packed_bytes", "workspace_bytes",
        "max_abs_acc")]


class QConvEpilogue(ctypes.Structure):
    _fields_ = [("mode", _i32), ("mult", _vp), ("shift", _i32), ("relu", _i32), ("clamp_lo", _i32),
                ("clamp_hi", _i32), ("bias", _vp), ("residual", _vp), ("residual_signed", _i32)]


class QConvTileInfo(ctypes.Structure):
    _fields_ = [(f, _i32) for f in ("id", "bits", "waves_p", "waves_k", "frag_p", "frag_k", "chunk_c", "tile_p",
                                    "tile_k", "threads", "variant", "x_signed", "w_signed")] + [("name", ctypes.c_char * 64)]


SCHEDULE_KNOBS = ("tile_id", "splits", "wg_per_cu", "band_buffers", "xcd_order", "ablation")


class QConvSchedule(ctypes.Structure):
    _fields_ = [(f, _i32) for f in SCHEDULE_KNOBS]


def make_schedule(sch: dict | QConvSchedule) -> QConvSchedule:
    """A qconv_schedule from a dict (missing launch knobs take their defaults)."""
    if isinstance(sch, QConvSchedule):
        return sch
    full = {"tile_id": -1, "splits": 1, "wg_per_cu": 0, "band_buffers": 0, "xcd_order": 1, "ablation": 0}
    full.update({k: int(v) for k, v in sch.items() if k in SCHEDULE_KNOBS})
    return QConvSchedule(**full)


class QConvError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(what)


_lock = threading.Lock()
_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libqconv.so; raises if it has not been built."""
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        if not os.path.exists(LIB_PATH):
            raise QConvError(EHIP, f"{LIB_PATH} is not built; run `python -m paper_2202_06819_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.qconv_build_digest.argtypes = []
        L.qconv_build_digest.restype = ctypes.c_char_p
        got, want = L.qconv_build_digest().decode(), source_digest()
        if got != want:
            raise QConvError(EHIP, f"{LIB_PATH} was built from other sources (digest {got}, sources {want}); "
                                   "rebuild it with `python -m paper_2202_06819_amd.build`")
        P = ctypes.POINTER
        L.qconv_layout.argtypes = [P(QConvDesc), P(QConvLayoutInfo)]
        L.qconv_pack.argtypes = [_vp, _vp, _i32, _i32, _i32, _i32, _i32, _i32, _vp]
        L.qconv2d.argtypes = [P(QConvDesc), _vp, _vp, P(QConvEpilogue), _vp, _vp, ctypes.c_size_t, _i32, _vp]
        L.qconv_tile_count.argtypes = []
        L.qconv_tile_get.argtypes = [_i32, P(QConvTileInfo)]
        L.qconv_tile_check.argtypes = [P(QConvDesc), _i32]
        L.qconv_default_tile.argtypes = [P(QConvDesc)]
        L.qconv_strerror.argtypes = [ctypes.c_int]
        L.qconv_strerror.restype = ctypes.c_char_p
        L.qconv_last_error.argtypes = []
        L.qconv_last_error.restype = ctypes.c_char_p
        L.qconv_selftest.argtypes = []
        L.qconv_prepared_filter_bytes.argtypes = [P(QConvDesc), _i32, P(ctypes.c_size_t)]
        L.qconv_prepare_filters.argtypes = [P(QConvDesc), _vp, _i32, _vp, ctypes.c_size_t, _vp]
        L.qconv2d_prepared.argtypes = [P(QConvDesc), _vp, _vp, ctypes.c_size_t, P(QConvEpilogue), _vp, _i32, _i32,
                                       _vp, ctypes.c_size_t, _vp]
        L.qconv_workspace_bytes.argtypes = [P(QConvDesc), _i32, _i32, P(ctypes.c_size_t)]
        L.qconv_max_splits.argtypes = [P(QConvDesc), _i32]
        L.qconv_probe_mfma_i8.argtypes = [_i32, _i32, _vp, _vp, P(_i64), _vp]
        L.qconv_probe_mfma_i8_shape.argtypes = [_i32, _i32, _i32, _vp, _vp, P(_i64), _vp]
        L.qconv_schedule_check.argtypes = [P(QConvDesc), P(QConvSchedule)]
        L.qconv_unroll.argtypes = [_vp, _vp] + [_i32] * 12 + [_vp]
        L.qconv_pack_interleaved.argtypes = [_vp, _vp] + [_i32] * 7 + [_vp]
        L.qconv2d_packing.argtypes = [P(QConvDesc), _vp, _vp, _vp, ctypes.c_size_t, P(QConvEpilogue), _vp, _i32,
                                      _vp]
        L.qconv2d_scheduled.argtypes = [P(QConvDesc), _vp, _vp, ctypes.c_size_t, P(QConvEpilogue), _vp,
                                        P(QConvSchedule), _vp, ctypes.c_size_t, _vp]
        L.qconv2d_prepared_noalloc.argtypes = [P(QConvDesc), _vp, _vp, ctypes.c_size_t, P(QConvEpilogue), _vp,
                                               _i32, _i32, _vp]
        L.qconv_noalloc_limits.argtypes = [P(_i64), P(_i64)]
        L.qconv_probe_launch.argtypes = [_i32, _i32, _i32, _vp]
        L.qconv_probe_grid_meet.argtypes = [_i32, _i32, _i32, _vp, _vp, _vp]
        L.qconv_last_launch.argtypes = [P(_i64), P(_i64), P(_i64)]
        L.qconv_proj_default_tile.argtypes = [P(QConvDesc)]
        L.qconv_proj_tile_check.argtypes = [P(QConvDesc), _i32]
        L.qconv_prepared_proj_filter_bytes.argtypes = [P(QConvDesc), _i32, P(ctypes.c_size_t)]
        L.qconv_prepare_filters_proj.argtypes = [P(QConvDesc), _vp, _vp, _i32, _vp, ctypes.c_size_t, _vp]
        L.qconv_proj_workspace_bytes.argtypes = [P(QConvDesc), _i32, _i32, P(ctypes.c_size_t)]
        L.qconv2d_proj.argtypes = [P(QConvDesc), _vp, _vp, ctypes.c_size_t, P(QConvEpilogue), _vp,
                                   P(QConvEpilogue), _vp, _i32, _i32, _vp, ctypes.c_size_t, _vp]
        for f in ("qconv_layout", "qconv_pack", "qconv2d", "qconv_tile_count", "qconv_tile_get", "qconv_tile_check",
                  "qconv_default_tile", "qconv_selftest", "qconv_prepared_filter_bytes", "qconv_prepare_filters",
                  "qconv2d_prepared", "qconv_workspace_bytes", "qconv_max_splits", "qconv_probe_mfma_i8", "qconv_schedule_check", "qconv2d_scheduled", "qconv_unroll", "qconv_pack_interleaved",
                  "qconv2d_packing", "qconv2d_prepared_noalloc", "qconv_noalloc_limits", "qconv_probe_launch",
                  "qconv_probe_grid_meet", "qconv_probe_mfma_i8_shape",
                  "qconv_last_launch", "qconv_proj_default_tile", "qconv_proj_tile_check",
                  "qconv_prepared_proj_filter_bytes", "qconv_prepare_filters_proj", "qconv_proj_workspace_bytes",
                  "qconv2d_proj"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
        return L


def _check(rc: int, what: str) -> int:
    if rc < 0:
        L = lib()
        raise QConvError(rc, f"{what}: {L.qconv_strerror(rc).decode()} ({L.qconv_last_error().decode()})")
    return rc


def make_desc(d: dict | QConvDesc) -> QConvDesc:
    if isinstance(d, QConvDesc):
        return d
    return QConvDesc(**{f: int(d.get(f, 0) if f == "nb" else d[f]) for f, _ in QConvDesc._fields_})


def layout(d: dict) -> dict:
    """Output extent and buffer sizes of a descriptor (host only)."""
    info = QConvLayoutInfo()
    _check(lib().qconv_layout(ctypes.byref(make_desc(d)), ctypes.byref(info)), "qconv_layout")
    return {f: getattr(info, f) for f, _ in QConvLayoutInfo._fields_}


def tiles() -> list[dict]:
    out = []
    for i in range(lib().qconv_tile_count()):
        t = QConvTileInfo()
        _check(lib().qconv_tile_get(i, ctypes.byref(t)), "qconv_tile_get")
        row = {f: getattr(t, f) for f, _ in QConvTileInfo._fields_ if f != "name"}
        row["name"] = t.name.decode()
        out.append(row)
    return out


def tile_status(d: dict, tile_id: int) -> int:
    """QCONV_OK if the tile can run the shape, else the status qconv2d would return."""
    return lib().qconv_tile_check(ctypes.byref(make_desc(d)), int(tile_id))


def default_tile(d: dict) -> int:
    return _check(lib().qconv_default_tile(ctypes.byref(make_desc(d))), "qconv_default_tile")


def selftest() -> int:
    return lib().qconv_selftest()


def build_digest() -> str:
    """Digest of the sources the loaded library was built from (equal to
    build.source_digest(): lib() refuses a library built from other sources)."""
    return lib().qconv_build_digest().decode()


def prepared_filter_bytes(d: dict, tile: int = -1) -> int:
    """Bytes of the prepared filters of `tile` for this shape (host only)."""
    n = ctypes.c_size_t(0)
    _check(lib().qconv_prepared_filter_bytes(ctypes.byref(make_desc(d)), int(tile), ctypes.byref(n)),
           "qconv_prepared_filter_bytes")
    return int(n.value)


def schedule_status(d: dict, sch: dict) -> int:
    """QCONV_OK if the schedule can run the shape, else the status the call would return."""
    return lib().qconv_schedule_check(ctypes.byref(make_desc(d)), ctypes.byref(make_schedule(sch)))


def max_splits(d: dict, tile: int = -1) -> int:
    """Largest split-K factor of `tile` for this shape (its channel chunks)."""
    rc = lib().qconv_max_splits(ctypes.byref(make_desc(d)), int(tile))
    if rc < 0:
        _check(rc, "qconv_max_splits")
    return int(rc)


def workspace_bytes(d: dict, tile: int = -1, splits: int = 1) -> int:
    """Split-K workspace bytes for (tile, splits); 0 without a split."""
    n = ctypes.c_size_t(0)
    _check(lib().qconv_workspace_bytes(ctypes.byref(make_desc(d)), int(tile), int(splits), ctypes.byref(n)),
           "qconv_workspace_bytes")
    return int(n.value)


def noalloc_limits() -> dict:
    """Capacity of qconv2d_prepared_noalloc's device scratch: bytes of split-K
    partial sums and output tiles (arrival counters)."""
    b, t = _i64(0), _i64(0)
    _check(lib().qconv_noalloc_limits(ctypes.byref(b), ctypes.byref(t)), "qconv_noalloc_limits")
    return {"scratch_bytes": int(b.value), "max_tiles": int(t.value)}


def make_workspace(d: dict, tile: int, splits: int, device) -> torch.Tensor | None:
    """A zero-filled split-K workspace (None when none is needed)."""
    n = workspace_bytes(d, tile, splits)
    return torch.zeros(n, dtype=torch.uint8, device=device) if n else None


def prepare_filters(d: dict, w_packed: torch.Tensor, tile: int = -1, out: torch.Tensor | None = None,
                    stream=None) -> torch.Tensor:
    """Packed KRSC filters -> the layout `tile` stages directly (done once, offline)."""
    desc = make_desc(d)
    nbytes = prepared_filter_bytes(d, tile)
    info = layout(d)
    if out is None:
        out = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=w_packed.device)
    rc = lib().qconv_prepare_filters(ctypes.byref(desc), _dev_ptr(w_packed, "w_packed", info["w_bytes"]), int(tile),
                                     _dev_ptr(out, "w_prepared", nbytes), out.numel() * out.element_size(),
                                     _vp(_stream(stream)))
    _check(rc, "qconv_prepare_filters")
    return out


def probe_mfma_i8(blocks: int, iters: int, sink: torch.Tensor, stamps: torch.Tensor, stream=None,
                  shape: int = 0) -> int:
    """Launch the MFMA-only rate probe (a measurement aid); returns the int8
    operations the launch performs.  `sink` is int32 [blocks*256] and `stamps`
    int64 [blocks*4] on the device (shader-clock start/end, 100 MHz start/end
    per workgroup).  shape 0: v_mfma_i32_16x16x64_i8; 1: v_mfma_i32_32x32x32_i8."""
    if sink.dtype != torch.int32 or stamps.dtype != torch.int64:
        raise QConvError(EINVAL, "sink must be int32 and stamps int64")
    ops = _i64(0)
    rc = lib().qconv_probe_mfma_i8_shape(int(shape), int(blocks), int(iters),
                                         _dev_ptr(sink, "sink", 4 * 256 * int(blocks)),
                                         _dev_ptr(stamps, "stamps", 8 * 4 * int(blocks)), ctypes.byref(ops),
                                         _vp(_stream(stream)))
    _check(rc, "qconv_probe_mfma_i8_shape")
    return int(ops.value)


def last_launch() -> dict:
    """Grid, threads and dynamic LDS of this thread's most recent convolution launch."""
    g, t, l = _i64(0), _i64(0), _i64(0)
    _check(lib().qconv_last_launch(ctypes.byref(g), ctypes.byref(t), ctypes.byref(l)), "qconv_last_launch")
    return {"grid": int(g.value), "threads": int(t.value), "lds_bytes": int(l.value)}


class ProbeGridMeetCall:
    """The device-wide meeting probe (a measurement aid): ``()`` enqueues one
    launch of `blocks` workgroups that meet `rounds` times (flat, or counted in
    per XCD group with `two_level`) on the int32 device tensor `state`:
    elements 0..143 the arrival counters (element 0 the top one), element 144
    the give-up flag, which the caller zeroes."""

    STATE_ELEMS = 145

    def __init__(self, blocks: int, rounds: int, state: torch.Tensor, two_level: bool = False, stream=None):
        if state.dtype != torch.int32 or state.numel() < self.STATE_ELEMS or not state.is_cuda:
            raise ValueError(f"state must be a device int32 tensor of at least {self.STATE_ELEMS} elements")
        base = _dev_ptr(state, "state", 4 * self.STATE_ELEMS)
        self._args = (int(blocks), int(rounds), int(bool(two_level)), _vp(base), _vp(base + 4 * 144),
                      _vp(_stream(stream)))
        self._fn = lib().qconv_probe_grid_meet

    def __call__(self) -> None:
        _check(self._fn(*self._args), "qconv_probe_grid_meet")


class ProbeLaunchCall:
    """The empty-kernel launch probe (a measurement aid) with its arguments
    marshalled once; ``()`` enqueues one launch."""

    def __init__(self, blocks: int, threads: int, lds_bytes: int = 0, stream=None):
        self._args = (int(blocks), int(threads), int(lds_bytes), _vp(_stream(stream)))
        self._fn = lib().qconv_probe_launch

    def __call__(self) -> None:
        _check(self._fn(*self._args), "qconv_probe_launch")


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev_ptr(t: torch.Tensor, name: str, min_bytes: int = 0) -> int:
    if not t.is_cuda:
        raise QConvError(EINVAL, f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise QConvError(EINVAL, f"{name} must be contiguous")
    if t.numel() * t.element_size() < min_bytes:
        raise QConvError(EINVAL, f"{name} holds {t.numel() * t.element_size()} bytes, needs {min_bytes}")
    return t.data_ptr()


def packed_shape(n: int, h: int, w: int, c: int, bits: int, nb: int = 1) -> tuple:
    """N x H x W x C' packed; with nb > 1 the batch-interleaved N/nb x H x W x nb x C'."""
    cw = c // 8 if bits == 4 else c
    return (n // nb, h, w, nb, cw) if nb > 1 else (n, h, w, cw)


def raw_shape(desc: QConvDesc, info: dict) -> tuple:
    """int32 output: N x P x Q x K, or N/nb x P x Q x nb x K in the batch-interleaved layout."""
    if desc.nb > 1:
        return (desc.n // desc.nb, info["p"], info["q"], desc.nb, desc.k)
    return (desc.n, info["p"], info["q"], desc.k)


def packed_dtype(bits: int) -> torch.dtype:
    return torch.int32 if bits == 4 else torch.int8


def pack(src: torch.Tensor, bits: int, is_signed: bool, out: torch.Tensor | None = None, stream=None,
         nb: int = 1) -> torch.Tensor:
    """int8 N x C x H x W (or K x C x R x S) -> saturated channel-packed N x H x W x ... ;
    nb > 1: the batch-interleaved layout (qconv_pack_interleaved)."""
    if src.dtype != torch.int8 or src.dim() != 4:
        raise QConvError(EINVAL, "pack expects a 4-d int8 tensor")
    n, c, h, w = src.shape
    nb = max(int(nb), 1)
    if out is None:
        if n % nb:
            raise QConvError(EINVAL, f"nb={nb} does not divide n={n}")
        out = torch.empty(packed_shape(n, h, w, c, bits, nb), dtype=packed_dtype(bits), device=src.device)
    dst = _dev_ptr(out, "dst", n * c * h * w * bits // 8)
    if nb == 1:
        rc = lib().qconv_pack(_dev_ptr(src, "src"), dst, n, c, h, w, int(bits), int(bool(is_signed)),
                              _vp(_stream(stream)))
    else:
        rc = lib().qconv_pack_interleaved(_dev_ptr(src, "src"), dst, n, c, h, w, int(bits), int(bool(is_signed)),
                                          nb, _vp(_stream(stream)))
    _check(rc, "qconv_pack")
    return out


def _epilogue_extras(epi: QConvEpilogue, desc: QConvDesc, y_bytes: int, bias, residual, residual_signed) -> None:
    """Fill the optional bias and residual of a requant epilogue."""
    if bias is not None:
        if bias.dtype != torch.int32 or bias.numel() != desc.k:
            raise QConvError(EINVAL, "bias needs one int32 per output channel")
        epi.bias = _dev_ptr(bias, "bias", 4 * desc.k)
    if residual is not None:
        epi.residual = _dev_ptr(residual, "residual", y_bytes)
        epi.residual_signed = int(bool(residual_signed))


def unroll(src: torch.Tensor, c_out: int, *, taps_w: int, stride_w: int = 1, pad_w: int = 0, taps_h: int = 1,
           stride_h: int = 1, pad_h: int = 0, out_h: int | None = None, out: torch.Tensor | None = None,
           stream=None) -> torch.Tensor:
    """int8 N x C x H x W -> N x out_h x Wout x c_out with filter taps folded
    into channels (see qconv_unroll).  ``out_h`` defaults to the rows a
    stride_h window of taps_h rows covers."""
    if src.dtype != torch.int8 or src.dim() != 4:
        raise QConvError(EINVAL, "unroll expects a 4-d int8 tensor")
    n, c, h, w = src.shape
    wout = max((w + 2 * pad_w - taps_w) // stride_w + 1, 0)
    if out_h is None:
        out_h = max((h + 2 * pad_h - taps_h) // stride_h + 1, 0)
    if out is None:
        out = torch.empty((n, out_h, wout, c_out), dtype=torch.int8, device=src.device)
    rc = lib().qconv_unroll(_dev_ptr(src, "src"), _dev_ptr(out, "dst", n * out_h * wout * c_out), n, c, h, w,
                            int(taps_h), int(stride_h), int(pad_h), int(out_h), int(taps_w), int(stride_w),
                            int(pad_w), int(c_out), _vp(_stream(stream)))
    _check(rc, "qconv_unroll")
    return out


def few_channel_plan(d: dict, c_out: int, fold: str = "rows") -> dict:
    """How a few-channel layer ``d`` (8-bit) runs as an unrolled one.

    fold="all": every filter tap goes into the channels, leaving a 1x1
    convolution over c_out >= R*S*C channels; fold="rows": the filter columns
    and groups of stride_h rows go into the channels, leaving a
    ceil(R/stride_h) x 1 convolution at stride 1 over c_out >= stride_h*S*C
    channels.  Returns the unroll arguments of the input (``x``) and of the
    filters (``w``, given as K x C x R x S) and the descriptor (``desc``) of the
    equivalent convolution; its output is the layer's output.
    """
    r, s_, sh = d["r"], d["s"], d["stride_h"]
    p = (d["h"] + 2 * d["pad_h"] - r) // sh + 1
    q = (d["w"] + 2 * d["pad_w"] - s_) // d["stride_w"] + 1
    if p < 1 or q < 1:
        raise QConvError(EINVAL, "the filter is larger than the padded input")
    if fold == "all":
        x = dict(taps_h=r, stride_h=sh, pad_h=d["pad_h"], out_h=p)
        w = dict(taps_h=r, stride_h=1, pad_h=0, out_h=1)
        rr, hh = 1, p
    elif fold == "rows":
        rr = -(-r // sh)
        x = dict(taps_h=sh, stride_h=sh, pad_h=d["pad_h"], out_h=p + rr - 1)
        w = dict(taps_h=sh, stride_h=sh, pad_h=0, out_h=rr)
        hh = p + rr - 1
    else:
        raise QConvError(EINVAL, f"fold must be 'rows' or 'all', not {fold!r}")
    x.update(taps_w=s_, stride_w=d["stride_w"], pad_w=d["pad_w"])
    w.update(taps_w=s_, stride_w=1, pad_w=0)
    desc = dict(d, h=hh, w=q, c=c_out, r=rr, s=1, stride_h=1, stride_w=1, pad_h=0, pad_w=0)
    return {"x": x, "w": w, "desc": desc}


def conv2d(d: dict, x: torch.Tensor, w: torch.Tensor, *, requant: bool = False, mult: torch.Tensor | None = None,
           shift: int = 20, relu: bool = True, clamp: tuple = (0, 15), out: torch.Tensor | None = None,
           tile: int = -1, workspace: torch.Tensor | None = None, stream=None,
           prepared: bool = False, splits: int = 1, bias: torch.Tensor | None = None,
           residual: torch.Tensor | None = None, residual_signed: bool = False,
           noalloc: bool = False) -> torch.Tensor:
    """The convolution with its fused epilogue; returns the output tensor.

    Raw mode: int32 N x P x Q x K accumulators.  Requant mode: the packed
    b-bit output (the next layer's input layout).  With ``prepared`` the
    filters `w` come from :func:`prepare_filters` for the same `tile`; with
    ``noalloc`` as well, the call goes through qconv2d_prepared_noalloc (a
    split-K uses the library's device scratch instead of `workspace`).
    """
    desc = make_desc(d)
    info = layout(d)
    bits = desc.bits
    if out is None:
        if requant:
            out = torch.empty(packed_shape(desc.n, info["p"], info["q"], desc.k, bits, desc.nb),
                              dtype=packed_dtype(bits), device=x.device)
        else:
            out = torch.empty(raw_shape(desc, info), dtype=torch.int32, device=x.device)
    epi = QConvEpilogue()
    if requant:
        if mult is None or mult.dtype != torch.int32 or mult.numel() != desc.k:
            raise QConvError(EINVAL, "requant needs an int32 multiplier per output channel")
        epi.mode, epi.mult = OUT_REQUANT, _dev_ptr(mult, "mult", 4 * desc.k)
        epi.shift, epi.relu, epi.clamp_lo, epi.clamp_hi = int(shift), int(bool(relu)), int(clamp[0]), int(clamp[1])
        _epilogue_extras(epi, desc, info["y_packed_bytes"], bias, residual, residual_signed)
    else:
        epi.mode = OUT_RAW_I32
    ws_ptr, ws_bytes = (None, 0) if workspace is None else (_dev_ptr(workspace, "workspace"),
                                                           workspace.numel() * workspace.element_size())
    y_bytes = info["y_packed_bytes"] if requant else info["y_raw_bytes"]
    if noalloc:
        if not prepared or workspace is not None:
            raise QConvError(EINVAL, "noalloc runs prepared filters and takes no workspace")
        wb = prepared_filter_bytes(d, tile)
        rc = lib().qconv2d_prepared_noalloc(ctypes.byref(desc), _dev_ptr(x, "x", info["x_bytes"]),
                                            _dev_ptr(w, "w", wb), w.numel() * w.element_size(), ctypes.byref(epi),
                                            _dev_ptr(out, "y", y_bytes), int(tile), int(splits), _vp(_stream(stream)))
        _check(rc, "qconv2d_prepared_noalloc")
        return out
    if prepared:
        wb = prepared_filter_bytes(d, tile)
        rc = lib().qconv2d_prepared(ctypes.byref(desc), _dev_ptr(x, "x", info["x_bytes"]), _dev_ptr(w, "w", wb),
                                    w.numel() * w.element_size(), ctypes.byref(epi), _dev_ptr(out, "y", y_bytes),
                                    int(tile), int(splits), ws_ptr, ws_bytes, _vp(_stream(stream)))
        _check(rc, "qconv2d_prepared")
        return out
    rc = lib().qconv2d(ctypes.byref(desc), _dev_ptr(x, "x", info["x_bytes"]), _dev_ptr(w, "w", info["w_bytes"]),
                       ctypes.byref(epi), _dev_ptr(out, "y", y_bytes), ws_ptr, ws_bytes, int(tile),
                       _vp(_stream(stream)))
    _check(rc, "qconv2d")
    return out


class PackCall:
    """A qconv_pack call with its arguments marshalled once; ``()`` enqueues it."""

    def __init__(self, src: torch.Tensor, bits: int, is_signed: bool, out: torch.Tensor | None = None, stream=None):
        if src.dtype != torch.int8 or src.dim() != 4:
            raise QConvError(EINVAL, "pack expects a 4-d int8 tensor")
        n, c, h, w = src.shape
        if out is None:
            out = torch.empty(packed_shape(n, h, w, c, bits), dtype=packed_dtype(bits), device=src.device)
        self.src, self.out = src, out
        self._args = (_dev_ptr(src, "src"), _dev_ptr(out, "dst", n * c * h * w * bits // 8), n, c, h, w, int(bits),
                      int(bool(is_signed)), _vp(_stream(stream)))
        self._fn = lib().qconv_pack

    def __call__(self) -> torch.Tensor:
        _check(self._fn(*self._args), "qconv_pack")
        return self.out


class Conv2dCall:
    """A qconv2d call with its arguments marshalled once; ``()`` enqueues it.

    Tensors are held so their memory outlives the call object.
    """

    def __init__(self, d: dict, x: torch.Tensor, w: torch.Tensor, *, requant: bool = False,
                 mult: torch.Tensor | None = None, shift: int = 20, relu: bool = True, clamp: tuple = (0, 15),
                 out: torch.Tensor | None = None, tile: int = -1, stream=None, prepared: bool = False,
                 splits: int = 1, workspace: torch.Tensor | None = None, schedule: dict | None = None,
                 bias: torch.Tensor | None = None, residual: torch.Tensor | None = None,
                 residual_signed: bool = False):
        """With `schedule` (a dict of qconv_schedule knobs; `w` prepared for its
        tile) the call goes through qconv2d_scheduled."""
        if schedule is not None:
            prepared = True
            tile = int(schedule.get("tile_id", tile))
            splits = int(schedule.get("splits", 1))
        self.desc = make_desc(d)
        info = layout(d)
        bits = self.desc.bits
        if out is None:
            shape = (packed_shape(self.desc.n, info["p"], info["q"], self.desc.k, bits, self.desc.nb) if requant
                     else raw_shape(self.desc, info))
            out = torch.empty(shape, dtype=packed_dtype(bits) if requant else torch.int32, device=x.device)
        self.epi = QConvEpilogue()
        if requant:
            if mult is None or mult.dtype != torch.int32 or mult.numel() != self.desc.k:
                raise QConvError(EINVAL, "requant needs an int32 multiplier per output channel")
            self.epi.mode, self.epi.mult = OUT_REQUANT, _dev_ptr(mult, "mult", 4 * self.desc.k)
            self.epi.shift, self.epi.relu = int(shift), int(bool(relu))
            self.epi.clamp_lo, self.epi.clamp_hi = int(clamp[0]), int(clamp[1])
            _epilogue_extras(self.epi, self.desc, info["y_packed_bytes"], bias, residual, residual_signed)
        else:
            self.epi.mode = OUT_RAW_I32
        y_bytes = info["y_packed_bytes"] if requant else info["y_raw_bytes"]
        self.x, self.w, self.mult, self.out, self.info = x, w, mult, out, info
        self.bias, self.residual = bias, residual
        self.tile = default_tile(d) if tile == -1 else int(tile)
        self.prepared = prepared
        self.splits = int(splits)
        if prepared:
            wb = prepared_filter_bytes(d, self.tile)
            if workspace is None and self.splits > 1:
                workspace = make_workspace(d, self.tile, self.splits, x.device)
            self.workspace = workspace
            ws_ptr, ws_bytes = (None, 0) if workspace is None else (_dev_ptr(workspace, "workspace"),
                                                                   workspace.numel() * workspace.element_size())
            if schedule is not None:
                self.schedule = make_schedule(dict(schedule, tile_id=self.tile, splits=self.splits))
                self._args = (ctypes.byref(self.desc), _dev_ptr(x, "x", info["x_bytes"]), _dev_ptr(w, "w", wb),
                              w.numel() * w.element_size(), ctypes.byref(self.epi), _dev_ptr(out, "y", y_bytes),
                              ctypes.byref(self.schedule), ws_ptr, ws_bytes, _vp(_stream(stream)))
                self._fn = lib().qconv2d_scheduled
            else:
                self._args = (ctypes.byref(self.desc), _dev_ptr(x, "x", info["x_bytes"]), _dev_ptr(w, "w", wb),
                              w.numel() * w.element_size(), ctypes.byref(self.epi), _dev_ptr(out, "y", y_bytes),
                              self.tile, self.splits, ws_ptr, ws_bytes, _vp(_stream(stream)))
                self._fn = lib().qconv2d_prepared
        else:
            self._args = (ctypes.byref(self.desc), _dev_ptr(x, "x", info["x_bytes"]), _dev_ptr(w, "w", info["w_bytes"]),
                          ctypes.byref(self.epi), _dev_ptr(out, "y", y_bytes), None, 0, self.tile,
                          _vp(_stream(stream)))
            self._fn = lib().qconv2d

    def __call__(self) -> torch.Tensor:
        _check(self._fn(*self._args), "qconv2d")
        return self.out


def proj_default_tile(d: dict) -> int:
    """The built-in tile for a 3x3 layer with a fused 1x1 projection."""
    return _check(lib().qconv_proj_default_tile(ctypes.byref(make_desc(d))), "qconv_proj_default_tile")


def proj_tile_status(d: dict, tile_id: int) -> int:
    """QCONV_OK if `tile_id` can run the 3x3 layer `d` with a fused projection."""
    return lib().qconv_proj_tile_check(ctypes.byref(make_desc(d)), int(tile_id))


def proj_workspace_bytes(d: dict, tile: int = -1, splits: int = 1) -> int:
    """Split-K workspace bytes of the fused projection launch; 0 without a split."""
    n = ctypes.c_size_t(0)
    _check(lib().qconv_proj_workspace_bytes(ctypes.byref(make_desc(d)), int(tile), int(splits), ctypes.byref(n)),
           "qconv_proj_workspace_bytes")
    return int(n.value)


def proj_desc(d: dict) -> dict:
    """The 1x1 projection a 3x3 layer can carry: same input, channels and stride, no padding."""
    return dict(d, r=1, s=1, pad_h=0, pad_w=0)


def prepare_filters_proj(d: dict, w_packed: torch.Tensor, w_proj_packed: torch.Tensor, tile: int = -1,
                         out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Packed 3x3 filters and packed 1x1 projection filters -> one prepared image
    for `tile` (the projection as its tenth tap)."""
    desc = make_desc(d)
    n = ctypes.c_size_t(0)
    _check(lib().qconv_prepared_proj_filter_bytes(ctypes.byref(desc), int(tile), ctypes.byref(n)),
           "qconv_prepared_proj_filter_bytes")
    nbytes = int(n.value)
    info = layout(d)
    if out is None:
        out = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=w_packed.device)
    rc = lib().qconv_prepare_filters_proj(ctypes.byref(desc), _dev_ptr(w_packed, "w_packed", info["w_bytes"]),
                                          _dev_ptr(w_proj_packed, "w_proj_packed", info["w_bytes"] // (desc.r * desc.s)),
                                          int(tile), _dev_ptr(out, "w_prepared", nbytes),
                                          out.numel() * out.element_size(), _vp(_stream(stream)))
    _check(rc, "qconv_prepare_filters_proj")
    return out


def _requant_epilogue(desc: QConvDesc, info: dict, mult, shift, relu, clamp, bias=None) -> QConvEpilogue:
    epi = QConvEpilogue()
    if mult is None or mult.dtype != torch.int32 or mult.numel() != desc.k:
        raise QConvError(EINVAL, "requant needs an int32 multiplier per output channel")
    epi.mode, epi.mult = OUT_REQUANT, _dev_ptr(mult, "mult", 4 * desc.k)
    epi.shift, epi.relu, epi.clamp_lo, epi.clamp_hi = int(shift), int(bool(relu)), int(clamp[0]), int(clamp[1])
    _epilogue_extras(epi, desc, info["y_packed_bytes"], bias, None, False)
    return epi


class ProjConv2dCall:
    """A qconv2d_proj call (a 3x3 layer with its 1x1 projection fused in) with
    its arguments marshalled once; ``()`` enqueues it and returns (y, y_proj).

    `w_prepared` comes from :func:`prepare_filters_proj` for `tile`.  Raw mode
    (requant=False) gives both int32 accumulator tensors; requant mode takes
    each output's own multipliers, shift, ReLU, clamp and optional bias
    (``proj`` holds the projection's: dict(mult=, shift=, relu=, clamp=, bias=)).
    `splits` > 1 is split-K, with a zero-filled `workspace` of
    :func:`proj_workspace_bytes` (made here when not given).
    """

    def __init__(self, d: dict, x: torch.Tensor, w_prepared: torch.Tensor, *, tile: int = -1, requant: bool = False,
                 mult: torch.Tensor | None = None, shift: int = 20, relu: bool = True, clamp: tuple = (0, 15),
                 bias: torch.Tensor | None = None, proj: dict | None = None, out: torch.Tensor | None = None,
                 out_proj: torch.Tensor | None = None, splits: int = 1, workspace: torch.Tensor | None = None,
                 stream=None):
        self.desc = make_desc(d)
        info = layout(d)
        bits = self.desc.bits
        shape = (packed_shape(self.desc.n, info["p"], info["q"], self.desc.k, bits) if requant
                 else raw_shape(self.desc, info))
        dtype = packed_dtype(bits) if requant else torch.int32
        out = torch.empty(shape, dtype=dtype, device=x.device) if out is None else out
        out_proj = torch.empty(shape, dtype=dtype, device=x.device) if out_proj is None else out_proj
        if requant:
            pj = proj or {}
            self.epi = _requant_epilogue(self.desc, info, mult, shift, relu, clamp, bias)
            self.epi_proj = _requant_epilogue(self.desc, info, pj.get("mult"), pj.get("shift", 20),
                                              pj.get("relu", True), pj.get("clamp", (0, 15)), pj.get("bias"))
        else:
            self.epi, self.epi_proj = QConvEpilogue(), QConvEpilogue()
            self.epi.mode = self.epi_proj.mode = OUT_RAW_I32
        self.tile = proj_default_tile(d) if tile == -1 else int(tile)
        n = ctypes.c_size_t(0)
        _check(lib().qconv_prepared_proj_filter_bytes(ctypes.byref(self.desc), self.tile, ctypes.byref(n)),
               "qconv_prepared_proj_filter_bytes")
        y_bytes = info["y_packed_bytes"] if requant else info["y_raw_bytes"]
        self.x, self.w, self.out, self.out_proj, self.info = x, w_prepared, out, out_proj, info
        self.keep = (mult, bias, proj)
        self.splits = int(splits)
        if workspace is None and self.splits > 1:
            nws = proj_workspace_bytes(d, self.tile, self.splits)
            workspace = torch.zeros(nws, dtype=torch.uint8, device=x.device) if nws else None
        self.workspace = workspace
        ws_ptr, ws_bytes = (None, 0) if workspace is None else (_dev_ptr(workspace, "workspace"),
                                                               workspace.numel() * workspace.element_size())
        self._args = (ctypes.byref(self.desc), _dev_ptr(x, "x", info["x_bytes"]),
                      _dev_ptr(w_prepared, "w", int(n.value)), w_prepared.numel() * w_prepared.element_size(),
                      ctypes.byref(self.epi), _dev_ptr(out, "y", y_bytes), ctypes.byref(self.epi_proj),
                      _dev_ptr(out_proj, "y_proj", y_bytes), self.tile, self.splits, ws_ptr, ws_bytes,
                      _vp(_stream(stream)))
        self._fn = lib().qconv2d_proj

    def __call__(self):
        _check(self._fn(*self._args), "qconv2d_proj")
        return self.out, self.out_proj


class PackingConv2dCall:
    """A qconv2d_packing call (the pack fused into the convolution) with its
    arguments marshalled once; ``()`` enqueues it and returns y.  `x` is the
    int8 N x C x H x W activations, `w_prepared` the filters prepared for
    `tile`; with ``x_packed`` (a tensor, or True to allocate one) the packed
    input is written too."""

    def __init__(self, d: dict, x: torch.Tensor, w_prepared: torch.Tensor, *, tile: int, requant: bool = True,
                 mult: torch.Tensor | None = None, shift: int = 20, relu: bool = True, clamp: tuple = (0, 15),
                 out: torch.Tensor | None = None, x_packed=None, stream=None):
        if x.dtype != torch.int8 or x.dim() != 4:
            raise QConvError(EINVAL, "the fused pack reads a 4-d int8 tensor")
        self.desc = make_desc(d)
        info = layout(d)
        bits = self.desc.bits
        if out is None:
            shape = (packed_shape(self.desc.n, info["p"], info["q"], self.desc.k, bits) if requant
                     else raw_shape(self.desc, info))
            out = torch.empty(shape, dtype=packed_dtype(bits) if requant else torch.int32, device=x.device)
        if x_packed is True:
            x_packed = torch.empty(packed_shape(self.desc.n, self.desc.h, self.desc.w, self.desc.c, bits),
                                   dtype=packed_dtype(bits), device=x.device)
        self.epi = QConvEpilogue()
        if requant:
            if mult is None or mult.dtype != torch.int32 or mult.numel() != self.desc.k:
                raise QConvError(EINVAL, "requant needs an int32 multiplier per output channel")
            self.epi.mode, self.epi.mult = OUT_REQUANT, _dev_ptr(mult, "mult", 4 * self.desc.k)
            self.epi.shift, self.epi.relu = int(shift), int(bool(relu))
            self.epi.clamp_lo, self.epi.clamp_hi = int(clamp[0]), int(clamp[1])
        else:
            self.epi.mode = OUT_RAW_I32
        y_bytes = info["y_packed_bytes"] if requant else info["y_raw_bytes"]
        self.x, self.w, self.mult, self.out, self.x_packed = x, w_prepared, mult, out, x_packed
        self.tile = int(tile)
        wb = prepared_filter_bytes(d, self.tile)
        xp_ptr = None if x_packed is None else _dev_ptr(x_packed, "x_packed", info["x_bytes"])
        self._args = (ctypes.byref(self.desc), _dev_ptr(x, "x", x.numel()), xp_ptr, _dev_ptr(w_prepared, "w", wb),
                      w_prepared.numel() * w_prepared.element_size(), ctypes.byref(self.epi),
                      _dev_ptr(out, "y", y_bytes), self.tile, _vp(_stream(stream)))
        self._fn = lib().qconv2d_packing

    def __call__(self) -> torch.Tensor:
        _check(self._fn(*self._args), "qconv2d_packing")
        return self.out
