"""Network descriptions of the parareal networks (structure only, no arithmetic).

A parareal network (Sec. 3, eq. (barf)) is described by its parts:

* ``pre[j]``    -- preprocessing operator C^j : X -> X_{j-1}           (eq. (xjyj))
* ``fine[j]``   -- parallel sub-network g^j : X_{j-1} -> X_j            (Sec. 3.1)
* ``coarse[j]`` -- coarse block F^j : X_j -> X_{j+1}, j = 1..N-1        (eq. (tilderk))
* ``head``      -- postprocessing h: global average pool + linear layer (Tables vgg / resnet)

Each part is a *segment*: a small list of nodes over numbered tensor slots.  Slot 0 is the
segment input, ``out`` the segment output.  Nodes are listed in a valid evaluation order.

Node kinds (all tensors NHWC):

``conv``     dst = conv_{k,stride,pad}(A) [+ slot ``res``];  A = ReLU(BN_b(src)) when ``bn`` >= 0
             (pre-activation prologue), else A = src.  Convolution is cross-correlation with zero
             padding and no bias; filters are stored [c_out][k][k][c_in].
``bnact``    dst = pool(ReLU(BN_b(src))) [+ slot ``res``];  pool = 2x2/2 max pool when ``pool`` == 2.
``maxpool3`` dst = 3x3, stride 2, pad 1 max pool of src (padding never wins).

A BN instance b normalises one slot (``bns[b]``) with batch statistics; every consumer that names
b sees the same activation ReLU(BN_b(slot)).

This module is shared input data: it holds no part of the method's arithmetic.
"""
from __future__ import annotations

import math

import numpy as np
from dataclasses import dataclass, field
from typing import List, Optional, Tuple


@dataclass
class Node:
    op: str
    src: int
    dst: int
    bn: int = -1
    pool: int = 0
    k: int = 1
    stride: int = 1
    pad: int = 0
    cout: int = 0
    res: int = -1


@dataclass
class Segment:
    in_shape: Tuple[int, int, int]          # (H, W, C) of slot 0
    nodes: List[Node] = field(default_factory=list)
    bns: List[int] = field(default_factory=list)   # slot normalised by each BN instance
    out: int = 0

    @property
    def n_slots(self) -> int:
        m = 0
        for n in self.nodes:
            m = max(m, n.dst, n.src, n.res)
        return m + 1


@dataclass
class Net:
    name: str
    dtype: str                 # "f32" or "bf16": storage / MFMA operand type of the GPU path
    batch: int
    in_shape: Tuple[int, int, int]   # image (H, W, C)
    classes: int
    pre: List[Segment]
    fine: List[Segment]
    coarse: List[Segment]
    head_cin: int
    seeds: Tuple[int, int, int]      # (weights, input, labels)
    input_layout: str = "nchw->nhwc"
    bn_init: str = "unit"            # "unit": gamma = 1, beta = 0; "random": seeded gamma, beta

    @property
    def n_sub(self) -> int:
        return len(self.fine)


class _SegBuilder:
    """Small helper that allocates slots and BN instances while a segment is written."""

    def __init__(self, in_shape):
        self.seg = Segment(in_shape=tuple(in_shape))
        self.next_slot = 1
        self.bn_of_slot = {}

    def new_slot(self):
        s = self.next_slot
        self.next_slot += 1
        return s

    def bn(self, slot):
        if slot not in self.bn_of_slot:
            self.bn_of_slot[slot] = len(self.seg.bns)
            self.seg.bns.append(slot)
        return self.bn_of_slot[slot]

    def conv(self, src, cout, k, stride=1, pad=None, preact=False, res=-1):
        if pad is None:
            pad = (k - 1) // 2
        dst = self.new_slot()
        self.seg.nodes.append(Node("conv", src, dst, self.bn(src) if preact else -1, 0,
                                   k, stride, pad, cout, res))
        return dst

    def bnact(self, src, pool=0, res=-1):
        dst = self.new_slot()
        self.seg.nodes.append(Node("bnact", src, dst, self.bn(src), pool, res=res))
        return dst

    def maxpool3(self, src):
        dst = self.new_slot()
        self.seg.nodes.append(Node("maxpool3", src, dst, k=3, stride=2, pad=1))
        return dst

    def done(self, out):
        self.seg.out = out
        return self.seg


# ----------------------------------------------------------------------------------------------
# building blocks
# ----------------------------------------------------------------------------------------------

def _bottleneck(b: _SegBuilder, x, cin, cout, stride):
    """Pre-activation bottleneck residual unit (Fig. ru; x_l = H_l(x_{l-1}) + x_{l-1}).

    1x1 squeeze to cout/4, 3x3 (carrying the stride), 1x1 expand to cout, each preceded by
    BN + ReLU.  When the channel count or resolution changes, a 1x1 convolution (same stride)
    on the pre-activated input replaces the identity skip."""
    mid = cout // 4
    z1 = b.conv(x, mid, 1, 1, 0, preact=True)
    if cin != cout or stride != 1:
        sk = b.conv(x, cout, 1, stride, 0, preact=True)
    else:
        sk = x
    z2 = b.conv(z1, mid, 3, stride, 1, preact=True)
    return b.conv(z2, cout, 1, 1, 0, preact=True, res=sk)


def _coarse_ru_paper(b: _SegBuilder, x, cin, cout, stride):
    """Coarse RU of the paper (Sec. 4.2.1): two 3x3 convolutions and a skip connection; the first
    convolution takes stride 2 when downsampling.  Pre-activation form with a 1x1 projection on
    the skip when the shape changes."""
    z1 = b.conv(x, cout, 3, stride, 1, preact=True)
    sk = b.conv(x, cout, 1, stride, 0, preact=True) if (cin != cout or stride != 1) else x
    return b.conv(z1, cout, 3, 1, 1, preact=True, res=sk)


def _pre_pool_conv(img_shape, target_shape, wide_img_ok=False):
    """C^j for j > 1 (Sec. 4.1.1, 4.2.1): 3x3/2 max pools down to the target resolution, then a
    1x1 convolution to the target channel count (bias free, no normalisation)."""
    H, W, C = img_shape
    th, tw, tc = target_shape
    b = _SegBuilder(img_shape)
    s = 0
    h = H
    while h > th:
        s = b.maxpool3(s)
        h = (h + 2 - 3) // 2 + 1
    assert h == th, (H, th)
    s = b.conv(s, tc, 1, 1, 0)
    return b.done(s)


# ----------------------------------------------------------------------------------------------
# ResNet-1001 (Table resnet)
# ----------------------------------------------------------------------------------------------

RESNET_UNITS_PER_STAGE = 111
RESNET_WIDTHS = (64, 128, 256)          # output widths of the three stages (mid = width / 4)


def resnet_units(img_hw, units_per_stage=RESNET_UNITS_PER_STAGE, widths=RESNET_WIDTHS, stem=16):
    """The residual units of ResNet-1001 (3 x 111) as (cin, cout, stride, out_hw)."""
    units = []
    cin, hw = stem, img_hw
    for s, cout in enumerate(widths):
        for u in range(units_per_stage):
            stride = 2 if (s > 0 and u == 0) else 1
            hw = hw // stride
            units.append((cin, cout, stride, hw))
            cin = cout
    return units


def partition_units(n_units, n_sub):
    """Contiguous chunks of ceil(n_units / N) units, the remainder to the last sub-network."""
    size = math.ceil(n_units / n_sub)
    bounds = []
    start = 0
    for j in range(n_sub):
        end = min(n_units, start + size) if j < n_sub - 1 else n_units
        bounds.append((start, end))
        start = end
    assert all(e > s for s, e in bounds), "empty sub-network"
    return bounds


def unit_cost(unit, kind="bytes"):
    """Cost of one residual unit (cin, cout, stride, out_hw) for partitioning: "flops" = forward
    multiply-adds of its convolutions, "bytes" = elements its convolutions read and write (what
    bounds a layer-at-a-time schedule on a bandwidth-bound device).  Per image."""
    cin, cout, stride, hw = unit
    hin, mid = hw * stride, cout // 4
    convs = [(hin, cin, hin, mid, 1), (hin, mid, hw, mid, 3), (hw, mid, hw, cout, 1)]   # (in_hw, cin, out_hw, cout, k)
    if cin != cout or stride != 1:
        convs.append((hin, cin, hw, cout, 1))
    if kind == "flops":
        return float(sum(o * o * co * ci * k * k for (i, ci, o, co, k) in convs))
    return float(sum(i * i * ci + o * o * co for (i, ci, o, co, k) in convs) + hw * hw * cout)


def partition_balanced(costs, n_sub):
    """Contiguous split of units with costs ``costs`` into ``n_sub`` non-empty sub-networks that
    minimises the largest sub-network cost (the decomposition by computational cost the paper
    suggests in the Remark after Table grad).  Exact dynamic programme over prefix sums; ties go to
    the earliest cut."""
    n = len(costs)
    assert 1 <= n_sub <= n
    S = np.concatenate([[0.0], np.cumsum(np.asarray(costs, dtype=np.float64))])
    INF = np.inf
    best = np.full((n_sub + 1, n + 1), INF)
    arg = np.zeros((n_sub + 1, n + 1), dtype=np.int64)
    best[0, 0] = 0.0
    for k in range(1, n_sub + 1):
        for i in range(k, n - (n_sub - k) + 1):
            j = np.arange(k - 1, i)
            v = np.maximum(best[k - 1, j], S[i] - S[j])
            a = int(np.argmin(v))
            best[k, i] = v[a]
            arg[k, i] = j[a]
    bounds = []
    i = n
    for k in range(n_sub, 0, -1):
        j = int(arg[k, i])
        bounds.append((j, i))
        i = j
    return bounds[::-1]


def partition_per_stage(units_per_stage, n_stages, n_sub):
    """The paper's split for N = 3 N_0 (Sec. 4.2.1): every stage cut into N_0 sub-networks of
    ceil(111 / N_0) units, the remainder to the stage's last one, so X_j is constant per stage."""
    assert n_sub % n_stages == 0
    n0 = n_sub // n_stages
    bounds = []
    for st in range(n_stages):
        sub = partition_units(units_per_stage, n0)
        bounds += [(st * units_per_stage + a, st * units_per_stage + b) for a, b in sub]
    return bounds


def resnet_parareal(name, batch, img_hw, n_sub, classes, dtype, seeds, coarse="config",
                    units_per_stage=RESNET_UNITS_PER_STAGE, widths=RESNET_WIDTHS, stem=16,
                    partition="contiguous"):
    """Parareal ResNet-N (Sec. 4.2.1).  ``units_per_stage`` / ``widths`` / ``stem`` give smaller
    nets of the same form for tests.  ``partition``: "contiguous" chunks of ceil(333/N) units
    (any N), the paper's "per_stage" split (N a multiple of 3), or "balanced" / "balanced_flops":
    equal cost per sub-network by unit_cost "bytes" / "flops"."""
    units = resnet_units(img_hw, units_per_stage, widths, stem)
    if partition == "per_stage":
        bounds = partition_per_stage(units_per_stage, len(widths), n_sub)
    elif partition in ("balanced", "balanced_flops"):
        kind = "flops" if partition == "balanced_flops" else "bytes"
        bounds = partition_balanced([unit_cost(u, kind) for u in units], n_sub)
    else:
        bounds = partition_units(len(units), n_sub)
    # X_0 = stem output (``stem`` channels at full resolution), X_j = shape after g^j
    X = [(img_hw, img_hw, stem)]
    for (s, e) in bounds:
        cin, cout, stride, hw = units[e - 1]
        X.append((hw, hw, cout))
    img = (img_hw, img_hw, 3)
    pre = []
    for j in range(n_sub):
        if j == 0:
            b = _SegBuilder(img)
            pre.append(b.done(b.conv(0, stem, 3, 1, 1)))
        else:
            pre.append(_pre_pool_conv(img, X[j]))
    fine = []
    for j, (s, e) in enumerate(bounds):
        b = _SegBuilder(X[j])
        x = 0
        for (cin, cout, stride, hw) in units[s:e]:
            x = _bottleneck(b, x, cin, cout, stride)
        fine.append(b.done(x))
    crs = []
    for j in range(1, n_sub):
        xin, xout = X[j], X[j + 1]
        stride = xin[0] // xout[0]
        b = _SegBuilder(xin)
        if coarse == "config":
            y = _bottleneck(b, 0, xin[2], xout[2], stride)
        else:  # the paper's coarse network: ceil(12/N) coarse RUs per F^j
            nc = math.ceil(12 / n_sub)
            y = 0
            c = xin[2]
            for r in range(nc):
                y = _coarse_ru_paper(b, y, c, xout[2], stride if r == 0 else 1)
                c = xout[2]
        crs.append(b.done(y))
    return Net(name, dtype, batch, img, classes, pre, fine, crs, X[-1][2], seeds)


# ----------------------------------------------------------------------------------------------
# VGG-16 (Table vgg), Parareal VGG-16-4 split of Sec. 4.1.1
# ----------------------------------------------------------------------------------------------

# sub-network j of the paper's split: list of (channels, ...) conv layers, a 2x2/2 max pool after
# the last one of every block.  g^1 = [64]+mp, [128,128]+mp ; g^2 = [256]x3+mp ; g^3, g^4 = [512]x3+mp
VGG_SPLIT = [[[64], [128, 128]], [[256, 256, 256]], [[512, 512, 512]], [[512, 512, 512]]]


def vgg_parareal(name, batch, img_hw, classes, dtype, seeds, coarse="config", split=VGG_SPLIT,
                 stem=64):
    """Parareal VGG-16-4 (Sec. 4.1.1); ``split`` / ``stem`` give smaller nets for tests."""
    img = (img_hw, img_hw, 3)
    X = [(img_hw, img_hw, stem)]
    fine = []
    for blocks in split:
        H, W, C = X[-1]
        b = _SegBuilder(X[-1])
        s = 0
        act = True          # slot s is already an activation (no BN/ReLU to apply)
        for blk in blocks:
            for i, c in enumerate(blk):
                s = b.conv(s, c, 3, 1, 1, preact=not act)
                act = False
                C = c
            s = b.bnact(s, pool=2)
            act = True
            H //= 2
            W //= 2
        fine.append(b.done(s))
        X.append((H, W, C))
    n_sub = len(fine)
    pre = []
    b = _SegBuilder(img)
    pre.append(b.done(b.bnact(b.conv(0, stem, 3, 1, 1))))
    for j in range(1, n_sub):
        pre.append(_pre_pool_conv(img, X[j]))
    crs = []
    for j in range(1, n_sub):
        b = _SegBuilder(X[j])
        if coarse == "config":          # one 3x3 convolution (+ BN, ReLU, 2x2 max pool)
            y = b.bnact(b.conv(0, X[j + 1][2], 3, 1, 1), pool=2)
        else:                           # the paper: two 3x3 convolutions and a max pool
            z = b.conv(0, X[j + 1][2], 3, 1, 1)
            z = b.conv(z, X[j + 1][2], 3, 1, 1, preact=True)
            y = b.bnact(z, pool=2)
        crs.append(b.done(y))
    return Net(name, dtype, batch, img, classes, pre, fine, crs, X[-1][2], seeds)


# ----------------------------------------------------------------------------------------------
# tiny fp32 network: N = 2 pre-activation basic blocks at 16 channels
# ----------------------------------------------------------------------------------------------

def tiny_parareal(name="tiny-basic-n2", batch=4, hw=32, ch=16, n_sub=2, classes=10, dtype="f32",
                  seeds=(1001, 1002, 1003)):
    shape = (hw, hw, ch)
    pre = []
    for j in range(n_sub):
        b = _SegBuilder(shape)
        pre.append(b.done(0 if j == 0 else b.conv(0, ch, 1, 1, 0)))
    fine = []
    for j in range(n_sub):
        b = _SegBuilder(shape)
        z = b.conv(0, ch, 3, 1, 1, preact=True)
        fine.append(b.done(b.conv(z, ch, 3, 1, 1, preact=True, res=0)))
    crs = []
    for j in range(1, n_sub):
        b = _SegBuilder(shape)
        crs.append(b.done(b.conv(0, ch, 3, 1, 1)))
    return Net(name, dtype, batch, shape, classes, pre, fine, crs, ch, seeds,
               input_layout="nchw->nhwc")


# ----------------------------------------------------------------------------------------------
# the five workloads
# ----------------------------------------------------------------------------------------------

def config(idx: int, batch: Optional[int] = None, coarse: str = "config", partition: str = "contiguous") -> Net:
    """Workload ``idx`` (0..5); ``batch`` overrides the batch size (smaller parity cases);
    ``coarse="paper"`` replaces the coarse blocks F^j of the VGG / ResNet workloads by the paper's
    own coarse networks (ResNet: ceil(12/N) two-3x3 residual units per F^j, Sec. 4.2.1; VGG: two
    3x3 convolutions and a max pool, Sec. 4.1.1); ``partition`` splits the ResNet units
    (resnet_parareal)."""
    sfx = ("" if coarse == "config" else "-papercoarse") + ("" if partition == "contiguous" else "-" + partition)
    if idx == 0:
        return tiny_parareal(batch=batch or 4)
    if idx == 1:
        return vgg_parareal("vgg16-parareal-n4" + sfx, batch or 128, 32, 10, "bf16", (2001, 2002, 2003),
                            coarse=coarse)
    if idx == 2:
        return resnet_parareal("resnet1001-parareal-n4" + sfx, batch or 64, 32, 4, 100, "bf16",
                               (3001, 3002, 3003), coarse=coarse, partition=partition)
    if idx == 3:
        return resnet_parareal("resnet1001-parareal-n16" + sfx, batch or 128, 32, 16, 100, "bf16",
                               (4001, 4002, 4003), coarse=coarse, partition=partition)
    if idx == 4:
        return resnet_parareal("resnet1001-parareal-n8-64px" + sfx, batch or 128, 64, 8, 200, "bf16",
                               (5001, 5002, 5003), coarse=coarse, partition=partition)
    if idx == 5:
        # ImageNet-shaped Parareal VGG-16-4 (Sec. 4.1.1, Table gradvgg): 224x224x3, 1000 classes,
        # the paper's coarse blocks
        return vgg_parareal("vgg16-parareal-n4-224px", batch or 128, 224, 1000, "bf16",
                            (6001, 6002, 6003), coarse="paper")
    raise ValueError(idx)


CONFIG_NAMES = [config(i, 1).name for i in range(6)]
