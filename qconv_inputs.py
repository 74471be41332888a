"""Seeded synthetic inputs and workload shapes for the quantised convolution path.

This module holds no arithmetic of the method: it only draws integers and
names shapes.  It is the one module both the GPU path's tests/benchmark and the
CPU oracle's callers use, so that both sides see the same bytes.

Every tensor of layer ``layer_id`` in workload ``workload_id`` is drawn from
``numpy.random.default_rng([workload_id, layer_id, tensor_id])`` with tensor_id
0 = activations (int8, N x C x H x W), 1 = filters (int8, K x C x R x S),
2 = per-output-channel multipliers (int32, K).

Workloads (the shapes of the paper's evaluation, Sec. 4.1 / Table 1: the 3x3
convolutions of ResNet stages, 4-bit; plus the other layers of the same
networks):

  0  one 4-bit 3x3 layer, N=1, 56x56, C=K=64, stride 1, pad 1, raw int32 output
  1  the same layer at N=8 with the fused requantising epilogue (this is the
     stage-2 workload of Table 1: 2*N*P*Q*K*C*R*S = 1,849,688,064 ops)
  2  ResNet-18 convolution stack after the stem, 4-bit, N=16, chained
  3  the ResNet-18 layer list in 8-bit, N=16
  4  ResNet-50 bottleneck layers, 4-bit, N=64, all stride 1
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import numpy as np

U4 = (0, 15)        # unsigned 4-bit activations
S4 = (-8, 7)        # signed 4-bit filters
S8 = (-128, 127)    # signed 8-bit activations and filters
MULT = (1 << 14, 1 << 15)   # per-channel multiplier range [2^14, 2^15)
SHIFT = 20


@dataclass(frozen=True)
class Epilogue:
    shift: int = SHIFT
    relu: bool = True
    lo: int = 0
    hi: int = 15
    mult_range: tuple = MULT


@dataclass(frozen=True)
class Layer:
    name: str
    n: int
    h: int
    w: int
    c: int
    k: int
    r: int
    s: int
    stride: int = 1
    pad: int = 0
    bits: int = 4
    x_signed: bool = False
    w_signed: bool = True
    x_range: tuple = U4
    w_range: tuple = S4
    epilogue: Epilogue | None = field(default_factory=Epilogue)
    src: int = -1          # chained networks: index of the layer whose output this one reads

    @property
    def p(self) -> int:
        return (self.h + 2 * self.pad - self.r) // self.stride + 1

    @property
    def q(self) -> int:
        return (self.w + 2 * self.pad - self.s) // self.stride + 1

    @property
    def macs(self) -> int:
        return self.n * self.p * self.q * self.k * self.c * self.r * self.s

    @property
    def ops(self) -> int:
        return 2 * self.macs

    def desc(self) -> dict:
        return dict(n=self.n, h=self.h, w=self.w, c=self.c, k=self.k, r=self.r, s=self.s,
                    stride_h=self.stride, stride_w=self.stride, pad_h=self.pad, pad_w=self.pad,
                    bits=self.bits, x_signed=int(self.x_signed), w_signed=int(self.w_signed))


def rng(workload_id: int, layer_id: int, tensor_id: int) -> np.random.Generator:
    return np.random.default_rng([workload_id, layer_id, tensor_id])


def draw_int8(g: np.random.Generator, shape, lo: int, hi: int) -> np.ndarray:
    """Uniform integers in [lo, hi] as int8."""
    return g.integers(lo, hi + 1, size=shape, dtype=np.int64).astype(np.int8)


def layer_tensors(workload_id: int, layer_id: int, layer: Layer) -> dict:
    """x (N,C,H,W) int8, w (K,C,R,S) int8 and mult (K,) int32 for one layer."""
    x = draw_int8(rng(workload_id, layer_id, 0), (layer.n, layer.c, layer.h, layer.w), *layer.x_range)
    w = draw_int8(rng(workload_id, layer_id, 1), (layer.k, layer.c, layer.r, layer.s), *layer.w_range)
    out = {"x": x, "w": w, "mult": None}
    if layer.epilogue is not None:
        lo, hi = layer.epilogue.mult_range
        out["mult"] = rng(workload_id, layer_id, 2).integers(lo, hi, size=layer.k, dtype=np.int64).astype(np.int32)
    return out


# --------------------------------------------------------------------------- workloads

def workload0() -> list[Layer]:
    return [Layer("c0_56x56_64to64_3x3", 1, 56, 56, 64, 64, 3, 3, 1, 1, epilogue=None)]


def workload1() -> list[Layer]:
    return [Layer("c1_56x56_64to64_3x3_n8", 8, 56, 56, 64, 64, 3, 3, 1, 1)]


def table1_stages() -> list[Layer]:
    """The four 3x3 convolutions of Table 1 (ResNet-50 stages 2-5: 56x56 64->64,
    28x28 128->128, 14x14 256->256, 7x7 512->512, stride 1, pad 1), at batch 8,
    where each has exactly the table's 1,849,688,064 ops."""
    return [Layer(f"t1_stage{i + 2}_{h}x{h}_{c}to{c}_3x3_n8", 8, h, h, c, c, 3, 3, 1, 1)
            for i, (h, c) in enumerate(((56, 64), (28, 128), (14, 256), (7, 512)))]


def _resnet18(n: int, bits: int) -> list[Layer]:
    """The 19 convolutions of ResNet-18 after the 7x7 stem, in forward order.

    The 1x1 downsample of a stage reads the block input (the same tensor as the
    strided 3x3).  Residual additions, pooling, stem and classifier are not
    part of the stack.
    """
    if bits == 4:
        kw = {}
    else:
        kw = dict(bits=8, x_signed=True, w_signed=True, x_range=S8, w_range=S8,
                  epilogue=Epilogue(relu=False, lo=-128, hi=127))
    layers: list[Layer] = []

    def add(name, h, c, k, r, stride, pad, src):
        layers.append(Layer(name, n, h, h, c, k, r, r, stride, pad, src=src, **kw))
        return len(layers) - 1

    prev = -1
    for b in range(2):
        prev = add(f"l1.{b}.conv1", 56, 64, 64, 3, 1, 1, prev)
        prev = add(f"l1.{b}.conv2", 56, 64, 64, 3, 1, 1, prev)
    h, c = 56, 64
    for stage in (2, 3, 4):
        k = c * 2
        block_in = prev
        a = add(f"l{stage}.0.conv1", h, c, k, 3, 2, 1, block_in)
        b2 = add(f"l{stage}.0.conv2", h // 2, k, k, 3, 1, 1, a)
        add(f"l{stage}.0.downsample", h, c, k, 1, 2, 0, block_in)
        a = add(f"l{stage}.1.conv1", h // 2, k, k, 3, 1, 1, b2)
        prev = add(f"l{stage}.1.conv2", h // 2, k, k, 3, 1, 1, a)
        h, c = h // 2, k
    return layers


def workload2() -> list[Layer]:
    return _resnet18(16, 4)


def workload3() -> list[Layer]:
    return _resnet18(16, 8)


def distinct(layers: list[Layer]) -> list[Layer]:
    """One layer per distinct shape, first occurrence kept (10 for ResNet-18)."""
    seen, out = set(), []
    for L in layers:
        key = (L.h, L.c, L.k, L.r, L.stride)
        if key not in seen:
            seen.add(key)
            out.append(L)
    return out


BOTTLENECK_REPEATS = {56: 3, 28: 4, 14: 6, 7: 3}


def workload4() -> list[Layer]:
    """ResNet-50 bottleneck layers at N=64 (1x1 reduce, 3x3, 1x1 expand per stage), stride 1."""
    out = []
    for h, c_in, mid in ((56, 256, 64), (28, 512, 128), (14, 1024, 256), (7, 2048, 512)):
        out.append(Layer(f"b{h}.reduce_1x1_{c_in}to{mid}", 64, h, h, c_in, mid, 1, 1, 1, 0))
        out.append(Layer(f"b{h}.3x3_{mid}to{mid}", 64, h, h, mid, mid, 3, 3, 1, 1))
        out.append(Layer(f"b{h}.expand_1x1_{mid}to{4 * mid}", 64, h, h, mid, 4 * mid, 1, 1, 1, 0))
    return out


WORKLOADS = {0: workload0, 1: workload1, 2: workload2, 3: workload3, 4: workload4}


def table1_layers(n: int = 8) -> list[Layer]:
    """The four 3x3 convolutions of Table 1 (ResNet-50 stages 2-5) at batch n."""
    return [Layer(f"stage{i + 2}_{h}x{h}_{c}", n, h, h, c, c, 3, 3, 1, 1)
            for i, (h, c) in enumerate(((56, 64), (28, 128), (14, 256), (7, 512)))]


def scaled(layer: Layer, **kw) -> Layer:
    return replace(layer, **kw)
