"""Chained layers: each layer's packed output buffer is the next layer's input.

The requantising epilogue writes the output in the same channel-packed NHWC
layout the next convolution reads (Sec. 3.3), so a network is a list of
qconv2d calls on one stream with no relayout between them.  A forward pass can
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


class Chain:
    """Layers on one stream; filters are prepared once for each layer's tile."""

    def __init__(self, layers: list[LayerSpec], x_packed: torch.Tensor, stream=None):
        self.layers = layers
        self.x = x_packed
        self.calls = []
        self.filters = []
        outs = []
        for L in layers:
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
                                    relu=L.relu, clamp=L.clamp, tile=tile, stream=stream, prepared=True,
                                    splits=splits, bias=L.bias, residual=res, residual_signed=L.residual_signed)
            outs.append(call.out)
            self.calls.append(call)
        self.outputs = outs
        self.graph = None

    def forward(self) -> list[torch.Tensor]:
        for c in self.calls:
            c()
        return self.outputs

    def capture(self) -> None:
        """Record one forward pass as a graph (the library allocates and memsets nothing)."""
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            # calls marshal the stream at construction: rebuild them for the capture stream
            calls = [qconv.Conv2dCall(c.desc, c.x, c.w, requant=True, mult=c.mult, shift=c.epi.shift,
                                      relu=bool(c.epi.relu), clamp=(c.epi.clamp_lo, c.epi.clamp_hi), out=c.out,
                                      tile=c.tile, stream=s, prepared=c.prepared, splits=c.splits,
                                      workspace=getattr(c, "workspace", None), bias=c.bias,
                                      residual=c.residual, residual_signed=bool(c.epi.residual_signed))
                     for c in self.calls]
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s):
                for c in calls:
                    c()
        torch.cuda.current_stream().wait_stream(s)
        self.graph = g

    def replay(self) -> list[torch.Tensor]:
        self.graph.replay()
        return self.outputs
