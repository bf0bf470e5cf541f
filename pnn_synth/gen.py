"""Seeded synthetic inputs for the parareal networks: images, labels and initial parameters.

Everything here is random-number generation and storage-type rounding of *inputs*; nothing of the
method's arithmetic.  Values are returned as float64 numpy arrays that are exactly representable
in the storage type the GPU path uses (bf16 or fp32), so that both sides consume identical numbers.

* image  x  ~ N(0, 1), drawn as [B, C, H, W] and stored NHWC;
* labels    ~ U{0 .. classes-1};
* conv filters: He-normal, std sqrt(2 / fan_in), fan_in = c_in * k * k (Sec. 4: initialisation of
  He et al.), drawn directly in [c_out][k][k][c_in] order;
* BN: gamma = 1, beta = 0 (``net.bn_init == "unit"``, the initial state of training), or, with
  ``net.bn_init == "random"``, gamma ~ U(0.5, 1.5) and beta ~ N(0, 0.2^2) drawn from their own
  PCG64 stream (seed: the weight seed + 7919), as BN parameters look once training has moved them;
  linear head: He-normal weight [classes][C], bias 0 (``"random"``: bias ~ N(0, 0.1^2)).

Tensors are drawn from one PCG64 stream per config in a fixed order: pre segments j = 1..N,
fine segments j = 1..N, coarse segments j = 1..N-1, then the head.
"""
from __future__ import annotations

import numpy as np

from .nets import Net, Segment


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """float64 -> nearest float32 -> nearest-even bfloat16, returned as float64."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_to_bf16(a)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def segment_shapes(seg: Segment):
    """(H, W, C) of every slot of a segment, inferred from the node list."""
    shapes = {0: tuple(seg.in_shape)}
    for n in seg.nodes:
        H, W, C = shapes[n.src]
        if n.op == "conv":
            Ho = (H + 2 * n.pad - n.k) // n.stride + 1
            Wo = (W + 2 * n.pad - n.k) // n.stride + 1
            shapes[n.dst] = (Ho, Wo, n.cout)
        elif n.op == "bnact":
            shapes[n.dst] = (H // 2, W // 2, C) if n.pool == 2 else (H, W, C)
        elif n.op == "maxpool3":
            shapes[n.dst] = ((H + 2 - 3) // 2 + 1, (W + 2 - 3) // 2 + 1, C)
        else:
            raise ValueError(n.op)
    return shapes


def init_segment(seg: Segment, rng: np.random.Generator, dtype: str, bn_rng=None):
    """Parameters of one segment: {'conv': [W per conv node or None], 'gamma': [...], 'beta': [...]}.
    ``bn_rng``: generator of random BN parameters (None: gamma = 1, beta = 0)."""
    shapes = segment_shapes(seg)
    conv = []
    for n in seg.nodes:
        if n.op == "conv":
            cin = shapes[n.src][2]
            std = np.sqrt(2.0 / (cin * n.k * n.k))
            w = rng.standard_normal((n.cout, n.k, n.k, cin)) * std
            conv.append(to_storage(w, dtype))
        else:
            conv.append(None)
    if bn_rng is None:
        gamma = [np.ones(shapes[s][2]) for s in seg.bns]
        beta = [np.zeros(shapes[s][2]) for s in seg.bns]
    else:
        gamma, beta = [], []
        for s in seg.bns:
            C = shapes[s][2]
            gamma.append(to_storage(bn_rng.uniform(0.5, 1.5, C), "f32"))
            beta.append(to_storage(0.2 * bn_rng.standard_normal(C), "f32"))
    return {"conv": conv, "gamma": gamma, "beta": beta}


def init_params(net: Net):
    rng = np.random.Generator(np.random.PCG64(net.seeds[0]))
    if net.bn_init == "random":
        bn_rng = np.random.Generator(np.random.PCG64(net.seeds[0] + 7919))
    elif net.bn_init == "unit":
        bn_rng = None
    else:
        raise ValueError(net.bn_init)
    p = {
        "pre": [init_segment(s, rng, net.dtype, bn_rng) for s in net.pre],
        "fine": [init_segment(s, rng, net.dtype, bn_rng) for s in net.fine],
        "coarse": [init_segment(s, rng, net.dtype, bn_rng) for s in net.coarse],
    }
    w = rng.standard_normal((net.classes, net.head_cin)) * np.sqrt(2.0 / net.head_cin)
    b = np.zeros(net.classes) if bn_rng is None else to_storage(0.1 * bn_rng.standard_normal(net.classes), "f32")
    p["head"] = {"w": to_storage(w, "f32"), "b": b}
    return p


def make_input(net: Net):
    rng = np.random.Generator(np.random.PCG64(net.seeds[1]))
    H, W, C = net.in_shape
    x = rng.standard_normal((net.batch, C, H, W)).transpose(0, 2, 3, 1)
    return to_storage(np.ascontiguousarray(x), net.dtype)


def make_labels(net: Net):
    rng = np.random.Generator(np.random.PCG64(net.seeds[2]))
    return rng.integers(0, net.classes, size=net.batch).astype(np.int32)


def make_all(net: Net):
    return make_input(net), make_labels(net), init_params(net)
