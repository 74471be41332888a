"""Chained layers: each layer's packed output buffer is the next layer's input.

The requantising epilogue writes the output in the same channel-packed NHWC
layout the next convolution reads (Sec. 3.3), so a network is a list of
qconv2d calls with no relayout between them.  A forward pass can
be replayed as a HIP graph to take host launch cost out of the loop.
"""
from __future__ import annotations

from dataclasses import dataclass

import torch

from . import qconv, sweep


@dataclass
class LayerSpec:
    """One convolution of a chain.  ``src`` is the index of the layer whose output
    it reads (-1: the network input)."""
    desc: dict
    w_packed: torch.Tensor
    mult: torch.Tensor
    shift: int
    relu: bool
    clamp: tuple
    src: int = -1
    tile: int = -1
    splits: int = 0        # split-K factor; 0: the tuned choice (else 1)
    bias: torch.Tensor | None = None   # int32 per output channel (accumulator units)
    residual_src: int | None = None    # layer whose output is added before ReLU (-1: the input); None: none
    residual_signed: bool = False


def projection_pairs(layers) -> dict[int, int]:
    """Layers that can run as one launch: a 3x3 layer with padding 1 and a 1x1
    layer without padding that read the same input at the same stride with the
    same channels and operand types (a residual stage's first convolution and
    its shortcut projection).  Returns {3x3 layer: 1x1 layer}; the 1x1 layer
    must come later in the chain and neither may take a residual."""
    pairs, used = {}, set()
    for i, A in enumerate(layers):
        d = A.desc
        if not (d["r"] == 3 and d["s"] == 3 and d["pad_h"] == 1 and d["pad_w"] == 1) or A.residual_src is not None:
            continue
        if int(d.get("nb", 0)) > 1:
            continue
        for j in range(i + 1, len(layers)):
            B = layers[j]
            e = B.desc
            if j in used or B.src != A.src or B.residual_src is not None:
                continue
            if (e["r"], e["s"], e["pad_h"], e["pad_w"]) != (1, 1, 0, 0):
                continue
            if all(e[f] == d[f] for f in ("n", "h", "w", "c", "k", "stride_h", "stride_w", "bits", "x_signed",
                                         "w_signed")):
                pairs[i] = j
                used.add(j)
                break
    return pairs


def branch_plan(layers) -> tuple[list[bool], list[list[int]]]:
    """Which layers of a chain run on the second stream, and the layers on the
    other stream each one must wait for.

    A layer goes to the second stream when it does not read the output of the
    layer just before it and the layer just after it reads that output
    instead, so the main line of layers steps over it: in a residual network,
    the strided 1x1 projection, which reads the block input beside the block's
    first 3x3 and is added only at the block's end.
    """
    n = len(layers)
    on_side = [0 < i < n - 1 and L.src != i - 1 and layers[i + 1].src == i - 1 for i, L in enumerate(layers)]
    waits = []
    for i, L in enumerate(layers):
        deps = {d for d in (L.src, L.residual_src) if d is not None and d >= 0}
        waits.append(sorted(d for d in deps if on_side[d] != on_side[i]))
    return on_side, waits


class Chain:
    """Layers on one stream; filters are prepared once for each layer's tile.

    With ``fuse_projections`` (the default), a strided 3x3 layer and the 1x1
    projection that reads the same input (:func:`projection_pairs`) run as one
    launch (qconv2d_proj): the projection's products ride on the 3x3 layer's
    staged input band, and its output goes to its own buffer.

    With ``branches`` (which turns the fusion off), a layer that the main line
    of layers steps over (a strided 1x1 projection beside the block's first
    3x3) runs on a second stream instead, so the two convolutions share the
    chip; events order it after its input and before the layers that read its
    output, and every forward pass starts and ends with the two streams joined.
    """

    def __init__(self, layers: list[LayerSpec], x_packed: torch.Tensor, stream=None, branches: bool = False,
                 fuse_projections: bool = True):
        self.layers = layers
        self.x = x_packed
        self.filters = []
        self.main = stream if stream is not None else torch.cuda.current_stream(x_packed.device)
        self.on_side, self.waits = branch_plan(layers) if branches else ([False] * len(layers),
                                                                          [[] for _ in layers])
        self.pairs = projection_pairs(layers) if fuse_projections and not branches else {}
        fused_into = {j: i for i, j in self.pairs.items()}
        self.side = torch.cuda.Stream(device=x_packed.device) if any(self.on_side) else None
        needed = {d for w in self.waits for d in w}
        self.events = [torch.cuda.Event() if i in needed else None for i in range(len(layers))]
        # one factory per launch: factory(stream) builds the call for that stream;
        # layers fused into an earlier launch have none
        self.factories = []
        proj_out = {}   # 3x3 layer -> the output buffer of the projection fused into its launch
        outs = []
        for i, L in enumerate(layers):
            if i in fused_into:
                outs.append(proj_out[fused_into[i]])
                self.factories.append(None)
                continue
            inp = self.x if L.src < 0 else outs[L.src]
            if i in self.pairs:
                P = layers[self.pairs[i]]
                tile, splits = L.tile, L.splits
                if tile == -1:
                    tile, tuned_splits = sweep.tuned_proj_config(L.desc)
                    splits = splits or tuned_splits
                splits = splits or 1
                wprep = qconv.prepare_filters_proj(L.desc, L.w_packed, P.w_packed, tile)
                nws = qconv.proj_workspace_bytes(L.desc, tile, splits)
                ws = torch.zeros(nws, dtype=torch.uint8, device=x_packed.device) if nws else None
                first = qconv.ProjConv2dCall(L.desc, inp, wprep, tile=tile, requant=True, mult=L.mult,
                                             shift=L.shift, relu=L.relu, clamp=L.clamp, bias=L.bias,
                                             proj=dict(mult=P.mult, shift=P.shift, relu=P.relu, clamp=P.clamp,
                                                       bias=P.bias), splits=splits, workspace=ws)
                y, yp = first.out, first.out_proj

                def make(stream, L=L, P=P, inp=inp, wprep=wprep, tile=tile, splits=splits, ws=ws, y=y, yp=yp):
                    return qconv.ProjConv2dCall(L.desc, inp, wprep, tile=tile, requant=True, mult=L.mult,
                                                shift=L.shift, relu=L.relu, clamp=L.clamp, bias=L.bias,
                                                proj=dict(mult=P.mult, shift=P.shift, relu=P.relu, clamp=P.clamp,
                                                          bias=P.bias), out=y, out_proj=yp, splits=splits,
                                                workspace=ws, stream=stream)
                proj_out[i] = yp
                self.filters.append(wprep)
                outs.append(y)
                self.factories.append(make)
                continue
            tile, splits = L.tile, L.splits
            if tile == -1:
                tile, tuned_splits = sweep.tuned_config(L.desc)
                splits = splits or tuned_splits
            splits = splits or 1
            wprep = qconv.prepare_filters(L.desc, L.w_packed, tile)
            self.filters.append(wprep)
            res = None
            if L.residual_src is not None:
                res = self.x if L.residual_src < 0 else outs[L.residual_src]
            ws = qconv.make_workspace(L.desc, tile, splits, x_packed.device) if splits > 1 else None
            first = qconv.Conv2dCall(L.desc, inp, wprep, requant=True, mult=L.mult, shift=L.shift, relu=L.relu,
                                     clamp=L.clamp, tile=tile, prepared=True, splits=splits, workspace=ws,
                                     bias=L.bias, residual=res, residual_signed=L.residual_signed)

            def make(stream, L=L, inp=inp, wprep=wprep, tile=tile, splits=splits, ws=ws, res=res, y=first.out):
                return qconv.Conv2dCall(L.desc, inp, wprep, requant=True, mult=L.mult, shift=L.shift, relu=L.relu,
                                        clamp=L.clamp, tile=tile, prepared=True, splits=splits, workspace=ws,
                                        bias=L.bias, residual=res, residual_signed=L.residual_signed, out=y,
                                        stream=stream)
            outs.append(first.out)
            self.factories.append(make)
        self.outputs = outs
        self.calls = [f(self._stream_of(i, self.main)) if f else None for i, f in enumerate(self.factories)]
        self.launches = sum(1 for c in self.calls if c is not None)
        self.graph = None

    def _stream_of(self, i: int, main):
        return self.side if self.on_side[i] else main

    def _run(self, calls, main) -> None:
        if self.side is not None:
            self.side.wait_stream(main)
        for i, c in enumerate(calls):
            if c is None:
                continue
            s = self._stream_of(i, main)
            for d in self.waits[i]:
                s.wait_event(self.events[d])
            c()
            if self.events[i] is not None:
                self.events[i].record(s)
        if self.side is not None:
            main.wait_stream(self.side)

    def forward(self) -> list[torch.Tensor]:
        self._run(self.calls, self.main)
        return self.outputs

    def capture(self) -> None:
        """Record one forward pass as a graph (the library allocates and memsets nothing)."""
        s = torch.cuda.Stream()
        s.wait_stream(self.main)
        with torch.cuda.stream(s):
            # calls marshal the stream at construction: rebuild them for the capture stream
            calls = [f(self._stream_of(i, s)) if f else None for i, f in enumerate(self.factories)]
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                self._run(calls, s)
        self.main.wait_stream(s)
        self.graph = g

    def replay(self) -> list[torch.Tensor]:
        self.graph.replay()
        return self.outputs
