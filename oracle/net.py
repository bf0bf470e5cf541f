"""Test infrastructure: the CPU oracle of the parareal neural network, fp64.

ONLY tests, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg may import this
module.  It shares no code with the GPU path.

What it computes is the network f-bar of eq. (barf) and its exact gradient:

  forward (Alg. para2, eqs. (xjyj), (rk), (tilderk), (tildey))
      x_j = C^j(x),  y_j = g^j(x_j)                     j = 1..N
      r_j = y_j - x_{j+1} (j < N),  r_N = 0
      rt_1 = r_1,  rt_{j+1} = r_{j+1} + F^j(rt_j)        j = 1..N-1
      ytilde = y_N + rt_N,  logits = h(ytilde),  L = mean softmax cross-entropy
  backward (Alg. para3, eqs. (ingredient1)-(deltaj))
      D_N = dL/dytilde,  D_0 = 0
      D_j = D_{j+1} . dF^j/drt_j,   dL/deta_j = D_{j+1} . dF^j/deta_j     j = N-1..1
      dL/dphi_j = D_j . dg^j/dphi_j          (dL/dy_j = D_j)
      dL/dx_j   = D_j . dg^j/dx_j - D_{j-1}  (then dL/ddelta_j through C^j)

Each segment (C^j, g^j, F^j) is evaluated node by node (see ``pnn_synth.nets``) and
differentiated by the chain rule written out per layer: convolution, BN (training mode, biased
variance, eps = 1e-5), ReLU (derivative 0 at 0), max pool (gradient to the first maximum).

Storage model.  With ``bf16=True`` every value the GPU path stores in bfloat16 is rounded to the
nearest bfloat16 at the point it is stored; arithmetic stays fp64.  Those points are: conv and
bnact outputs (after the residual / external addend), pre-activated conv operands ReLU(BN(z)),
the interface residuals r_j, D_N, the BN-backward input dL/d(BN output), every slot gradient,
and dL/dx_j after the combine.  BN statistics are taken from the stored (rounded) tensors.
With ``bf16=False`` nothing is rounded: the plain fp64 definition.
"""
from __future__ import annotations

import numpy as np

from . import prim as P

BN_EPS = 1e-5


# ------------------------------------------------------------------------------------------------
# node-level definitions (one layer of a segment)
# ------------------------------------------------------------------------------------------------

def bn_batch_stats(z):
    """Training-mode BN statistics of a stored tensor: per-channel mean and 1/sqrt(var + eps),
    biased variance over (n, h, w)."""
    C = z.shape[-1]
    mean, var = P.bn_stats(z.reshape(-1, C))
    return mean, 1.0 / np.sqrt(var + BN_EPS)


def bn_relu(z, gamma, beta, stats):
    """(ReLU(BN(z)), BN(z)) without rounding."""
    mean, invstd = stats
    y = (z - mean) * invstd * gamma + beta
    return np.maximum(y, 0.0), y


def node_forward(n, w, gamma, beta, src, res, ext, st, stats=None):
    """Value a node stores: conv_{k,stride,pad}(A) or pool(ReLU(BN(src))) or a 3x3/2 max pool,
    plus the residual and external addends, rounded to storage once."""
    if n.op == "conv":
        a = st(bn_relu(src, gamma, beta, stats)[0]) if n.bn >= 0 else src
        y = P.conv_fwd(a, w, n.stride, n.pad)
    elif n.op == "bnact":
        y = bn_relu(src, gamma, beta, stats)[0]
        if n.pool == 2:
            y = P.maxpool_fwd(y, 2, 2, 0)
    elif n.op == "maxpool3":
        y = P.maxpool_fwd(src, 3, 2, 1)
    else:
        raise ValueError(n.op)
    if res is not None:
        y = y + res
    if ext is not None:
        y = y + ext
    return st(y)


def conv_node_backward(n, w, a, g):
    """dL/dW and dL/dA of conv node n from dL/d(output) = g; A is the operand it consumed."""
    return (P.conv_bwd_weight(a, g, n.k, n.stride, n.pad),
            P.conv_bwd_data(g, w, a.shape, n.stride, n.pad))


def bnact_node_backward(n, act, g):
    """dL/d(ReLU(BN(src))) of a bnact node: the 2x2 pool routes g to the first maximum."""
    return P.maxpool_bwd(act, g, 2, 2, 0) if n.pool == 2 else g


def bn_input_grad(z, gamma, stats, dbn):
    """BN backward from dbn = dL/d(BN output): (dL/dz, dgamma, dbeta), batch statistics."""
    C = z.shape[-1]
    M = z.size // C
    mean, invstd = stats
    xhat = (z - mean) * invstd
    sdb, sdbx = P.colsum2(dbn.reshape(-1, C), xhat.reshape(-1, C))
    gx = gamma * invstd / M * (M * dbn - sdb - xhat * sdbx)
    return gx, sdbx, sdb


def bn_backward(z, gamma, stats, ybn, dA, st):
    """BN + ReLU backward from dA = dL/d(ReLU(BN(z))).  Returns (dbn, dL/dz, dgamma, dbeta) with
    dbn = dL/d(BN output) as stored."""
    dbn = st(dA * (ybn > 0.0))
    gx, dgamma, dbeta = bn_input_grad(z, gamma, stats, dbn)
    return dbn, gx, dgamma, dbeta


# ------------------------------------------------------------------------------------------------
# segments (C^j, g^j, F^j)
# ------------------------------------------------------------------------------------------------

class SegmentRun:
    """Forward state of one segment kept for its backward pass."""

    def __init__(self, seg, prm):
        self.seg = seg
        self.prm = prm
        self.slots = {}
        self.bn = {}

    def stats(self, b):
        if b not in self.bn:
            self.bn[b] = bn_batch_stats(self.slots[self.seg.bns[b]])
        return self.bn[b]

    def bn_forward(self, b):
        """(ReLU(BN_b(z)), BN_b(z)) without rounding; statistics from the stored slot."""
        return bn_relu(self.slots[self.seg.bns[b]], self.prm["gamma"][b], self.prm["beta"][b],
                       self.stats(b))


def seg_forward(seg, prm, x, st, ext=None):
    """Evaluate a segment on input ``x``; ``ext`` is added to the last node's result before it
    is stored (the coarse blocks' r_{j+1} or y_N addend)."""
    run = SegmentRun(seg, prm)
    run.slots[0] = x
    last = len(seg.nodes) - 1
    for i, n in enumerate(seg.nodes):
        g_b = prm["gamma"][n.bn] if n.bn >= 0 else None
        b_b = prm["beta"][n.bn] if n.bn >= 0 else None
        run.slots[n.dst] = node_forward(
            n, prm["conv"][i], g_b, b_b, run.slots[n.src],
            run.slots[n.res] if n.res >= 0 else None, ext if i == last else None, st,
            run.stats(n.bn) if n.bn >= 0 else None)
    if ext is not None and not seg.nodes:
        run.slots[0] = st(x + ext)
    return run.slots[seg.out], run


def seg_backward(run, gout, st):
    """Gradients of a segment from dL/d(output) = ``gout``.

    Returns (dL/d(input), {'conv': [dW per node], 'gamma': [...], 'beta': [...]})."""
    seg, prm = run.seg, run.prm
    G = {}          # gradient accumulated per slot
    dA = {}         # gradient w.r.t. ReLU(BN_b(.)) accumulated per BN instance (before pooling)
    grads = {"conv": [None] * len(seg.nodes),
             "gamma": [None] * len(seg.bns), "beta": [None] * len(seg.bns)}
    G[seg.out] = gout

    def finish(s):
        """All consumers of slot s are done: add its BN path and store its gradient."""
        g = G.get(s)
        if s in seg.bns:
            b = seg.bns.index(s)
            if b in dA:
                _, ybn = run.bn_forward(b)
                dbn, gx, grads["gamma"][b], grads["beta"][b] = bn_backward(
                    run.slots[s], prm["gamma"][b], run.stats(b), ybn, dA[b], st)
                g = gx if g is None else g + gx
        if g is None:
            g = np.zeros_like(run.slots[s])
        G[s] = st(g)
        return G[s]

    def add(s, v):
        G[s] = v if s not in G else G[s] + v

    for i in range(len(seg.nodes) - 1, -1, -1):
        n = seg.nodes[i]
        g = finish(n.dst)
        if n.res >= 0:
            add(n.res, g)
        if n.op == "conv":
            a = st(run.bn_forward(n.bn)[0]) if n.bn >= 0 else run.slots[n.src]
            grads["conv"][i], da = conv_node_backward(n, prm["conv"][i], a, g)
            if n.bn >= 0:
                dA[n.bn] = da if n.bn not in dA else dA[n.bn] + da
            else:
                add(n.src, da)
        elif n.op == "bnact":
            d = bnact_node_backward(n, run.bn_forward(n.bn)[0], g)
            dA[n.bn] = d if n.bn not in dA else dA[n.bn] + d
        elif n.op == "maxpool3":
            add(n.src, P.maxpool_bwd(run.slots[n.src], g, 3, 2, 1))
    return finish(0), grads


class ParaRealOracle:
    """The parareal network f-bar of one ``pnn_synth.Net`` with given parameters."""

    def __init__(self, net, params, bf16=None):
        self.net = net
        self.p = params
        self.bf16 = (net.dtype == "bf16") if bf16 is None else bf16

    def st(self, a):
        return P.round_bf16(a) if self.bf16 else a

    # -- postprocessing h: global average pool + linear layer, softmax cross-entropy ------------
    def head(self, yt, labels):
        hp = self.p["head"]
        B, H, W, C = yt.shape
        pooled = yt.mean(axis=(1, 2))
        logits = pooled @ hp["w"].T + hp["b"]
        zmax = logits.max(axis=1, keepdims=True)
        lse = zmax[:, 0] + np.log(np.exp(logits - zmax).sum(axis=1))
        loss = float(np.mean(lse - logits[np.arange(B), labels]))
        prob = np.exp(logits - lse[:, None])
        dlogits = prob.copy()
        dlogits[np.arange(B), labels] -= 1.0
        dlogits /= B
        dW = dlogits.T @ pooled
        db = dlogits.sum(axis=0)
        dpooled = dlogits @ hp["w"]
        D_N = self.st(np.broadcast_to(dpooled[:, None, None, :] / (H * W), yt.shape).copy())
        return {"logits": logits, "loss": loss, "D_N": D_N, "dw": dW, "db": db}

    # -- Alg. para2 ---------------------------------------------------------------------------
    def forward(self, x, exact_interfaces=False):
        net, st = self.net, self.st
        N = net.n_sub
        out = {"x": [], "y": [], "r": [], "rt": [], "pre_run": [], "fine_run": [], "coarse_run": []}
        for j in range(N):
            if exact_interfaces and j > 0:
                xj = out["y"][j - 1]           # x_{j+1} := y_j  (interfaces already exact)
                out["pre_run"].append(None)
            else:
                xj, run = seg_forward(net.pre[j], self.p["pre"][j], x, st)
                out["pre_run"].append(run)
            yj, run = seg_forward(net.fine[j], self.p["fine"][j], xj, st)
            out["x"].append(xj)
            out["y"].append(yj)
            out["fine_run"].append(run)
        for j in range(N - 1):                  # r_j = y_j - x_{j+1}
            out["r"].append(st(out["y"][j] - out["x"][j + 1]))
        if N == 1:
            out["ytilde"] = out["y"][0]
            return out
        out["rt"].append(out["r"][0])          # rt_1 = r_1
        for j in range(N - 1):                  # rt_{j+1} = r_{j+1} + F^j(rt_j); ytilde = y_N + rt_N
            ext = out["r"][j + 1] if j + 1 < N - 1 else out["y"][N - 1]
            v, run = seg_forward(net.coarse[j], self.p["coarse"][j], out["rt"][j], st, ext=ext)
            out["coarse_run"].append(run)
            if j + 1 < N - 1:
                out["rt"].append(v)
            else:
                out["ytilde"] = v
        return out

    # -- Alg. para3 ---------------------------------------------------------------------------
    def backward(self, fwd, hd):
        net, st = self.net, self.st
        N = net.n_sub
        D = [None] * N
        D[N - 1] = hd["D_N"]
        deta = [None] * (N - 1)
        for j in range(N - 2, -1, -1):          # D_j = D_{j+1} . dF^j/drt_j
            D[j], deta[j] = seg_backward(fwd["coarse_run"][j], D[j + 1], st)
        dxg, dphi = [], []
        for j in range(N):                      # dL/dy_j = D_j
            g, gr = seg_backward(fwd["fine_run"][j], D[j], st)
            dxg.append(g)
            dphi.append(gr)
        dx = [dxg[0]] + [st(dxg[j] - D[j - 1]) for j in range(1, N)]   # - D_{j-1} (eq. (deltaj))
        ddelta = []
        dimg = None
        for j in range(N):
            run = fwd["pre_run"][j]
            if run is None:
                ddelta.append(None)
                continue
            gimg, gr = seg_backward(run, dx[j], st)
            ddelta.append(gr)
            dimg = gimg if dimg is None else dimg + gimg
        return {"D": D, "deta": deta, "dx_fine": dxg, "dx": dx, "dphi": dphi, "ddelta": ddelta,
                "dimage": dimg}

    def step(self, x, labels):
        fwd = self.forward(x)
        hd = self.head(fwd["ytilde"], labels)
        bwd = self.backward(fwd, hd)
        return fwd, hd, bwd

    # -- the original network f = h o g^N o ... o g^1 o C^1 (sequential) ---------------------
    def sequential(self, x, labels=None):
        """Output of g^N o ... o g^1 o C^1; with ``labels`` also the head and dL/dx."""
        runs = []
        v, run = seg_forward(self.net.pre[0], self.p["pre"][0], x, self.st)
        runs.append(run)
        for j in range(self.net.n_sub):
            v, run = seg_forward(self.net.fine[j], self.p["fine"][j], v, self.st)
            runs.append(run)
        if labels is None:
            return v
        hd = self.head(v, labels)
        g = hd["D_N"]
        for run in reversed(runs):
            g, _ = seg_backward(run, g, self.st)
        return v, hd, g


def param_count(net, coarse=True, bn=True):
    """Trainable parameter counts {pre, fine[j], coarse[j], head} from the node lists."""
    from pnn_synth.gen import segment_shapes

    def seg_count(seg):
        sh = segment_shapes(seg)
        c = 0
        for n in seg.nodes:
            if n.op == "conv":
                c += n.cout * n.k * n.k * sh[n.src][2]
        if bn:
            c += sum(2 * sh[s][2] for s in seg.bns)
        return c

    return {"pre": [seg_count(s) for s in net.pre], "fine": [seg_count(s) for s in net.fine],
            "coarse": [seg_count(s) for s in net.coarse],
            "head": net.classes * net.head_cin + net.classes}


def receptive_field(seg):
    """Receptive field (pixels per side) of the segment output along its main path: the chain of
    ``src`` inputs from the output back to slot 0 (skip connections do not widen it)."""
    by_dst = {n.dst: n for n in seg.nodes}
    chain = []
    s = seg.out
    while s != 0:
        n = by_dst[s]
        chain.append(n)
        s = n.src
    rf, jump = 1, 1
    for n in reversed(chain):
        if n.op in ("conv", "maxpool3"):
            rf += (n.k - 1) * jump
            jump *= n.stride
        elif n.op == "bnact" and n.pool == 2:
            rf += jump
            jump *= 2
    return rf
