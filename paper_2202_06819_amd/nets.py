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

    With ``branches``, a layer that the main line of layers steps over (a
    strided 1x1 projection beside the block's first 3x3) runs on a second
    stream, so the two convolutions share the chip; events order it
    after its input and before the layers that read its output, and every
    forward pass starts and ends with the two streams joined.
    """

    def __init__(self, layers: list[LayerSpec], x_packed: torch.Tensor, stream=None, branches: bool = False):
        self.layers = layers
        self.x = x_packed
        self.calls = []
        self.filters = []
        self.main = stream if stream is not None else torch.cuda.current_stream(x_packed.device)
        self.on_side, self.waits = branch_plan(layers) if branches else ([False] * len(layers),
                                                                          [[] for _ in layers])
        self.side = torch.cuda.Stream(device=x_packed.device) if any(self.on_side) else None
        needed = {d for w in self.waits for d in w}
        self.events = [torch.cuda.Event() if i in needed else None for i in range(len(layers))]
        outs = []
        for i, L in enumerate(layers):
            inp = self.x if L.src < 0 else outs[L.src]
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
            call = qconv.Conv2dCall(L.desc, inp, wprep, requant=True, mult=L.mult, shift=L.shift,
                                    relu=L.relu, clamp=L.clamp, tile=tile, stream=self._stream_of(i, self.main),
                                    prepared=True, splits=splits, bias=L.bias, residual=res,
                                    residual_signed=L.residual_signed)
            outs.append(call.out)
            self.calls.append(call)
        self.outputs = outs
        self.graph = None

    def _stream_of(self, i: int, main):
        return self.side if self.on_side[i] else main

    def _run(self, calls, main) -> None:
        if self.side is not None:
            self.side.wait_stream(main)
        for i, c in enumerate(calls):
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
            calls = [qconv.Conv2dCall(c.desc, c.x, c.w, requant=True, mult=c.mult, shift=c.epi.shift,
                                      relu=bool(c.epi.relu), clamp=(c.epi.clamp_lo, c.epi.clamp_hi), out=c.out,
                                      tile=c.tile, stream=self._stream_of(i, s), prepared=c.prepared,
                                      splits=c.splits, workspace=getattr(c, "workspace", None), bias=c.bias,
                                      residual=c.residual, residual_signed=bool(c.epi.residual_signed))
                     for i, c in enumerate(self.calls)]
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                self._run(calls, s)
        self.main.wait_stream(s)
        self.graph = g

    def replay(self) -> list[torch.Tensor]:
        self.graph.replay()
        return self.outputs
