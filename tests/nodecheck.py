"""Teacher-forced, node-level parity of a GPU training step.

After one step on the GPU, every checked node of a segment is recomputed by the oracle's node-level
definitions (``oracle.net``) from the GPU's OWN stored inputs (layer inputs, BN statistics inputs,
output gradients), and compared with what the GPU stored.  Each comparison therefore isolates one
kernel invocation: its error is only rounding (fp32 accumulation vs fp64, occasional bf16 rounding
flips), not the amplification of earlier differences through a deep network.

At full sizes the convolutions (forward, data gradient, weight gradient) are evaluated at sampled
output positions; BN statistics / backward and the combine / head checks use whole tensors.
"""
from __future__ import annotations

import numpy as np

from pnn_synth.gen import segment_shapes
from oracle import prim as P
from oracle.net import (bn_batch_stats, bn_input_grad, bn_relu, bnact_node_backward,
                        conv_node_backward, node_forward)  # noqa: F401


def rel_inf(a, ref):
    a, ref = np.asarray(a), np.asarray(ref)
    return float(np.abs(a - ref).max() / max(np.abs(ref).max(), 1e-30)) if ref.size else 0.0


def rel_2(a, ref):
    a, ref = np.asarray(a), np.asarray(ref)
    return float(np.linalg.norm((a - ref).ravel()) / max(np.linalg.norm(ref.ravel()), 1e-30)) if ref.size else 0.0


class SegView:
    """The GPU tensors of one segment after a step: slot values, slot gradients, BN data."""

    def __init__(self, g, part, j, dx_fine=None):
        import torch
        self.torch = torch
        self.g = g
        net = g.net
        self.part, self.j = part, j
        self.seg = [net.pre, net.fine, net.coarse][part][j]
        self.shapes = segment_shapes(self.seg)
        self.B = net.batch
        N = net.n_sub
        self.ext_add = None
        self.gin = None
        if part == 1:
            self.ext_in, self.ext_out, self.gout = g.x[j], g.y[j], g.D[j]
            self.gin = dx_fine[j] if dx_fine is not None else None
        elif part == 2:
            last = j == N - 2
            self.ext_in = g.rt[j]
            self.ext_out = g.ytilde if last else g.rt[j + 1]
            self.ext_add = g.y[N - 1] if last else g.r[j + 1]
            self.gout, self.gin = g.D[j + 1], g.D[j]
        else:
            self.ext_in, self.ext_out, self.gout = g.image, g.x[j], g.dx[j]
        self._cache = {}

    def _ws(self, buf, off, n, dtype):
        t = buf[off:off + n * (2 if dtype == self.torch.bfloat16 else 4)]
        return t.view(dtype)

    def _np(self, t, shape):
        return t.float().cpu().numpy().astype(np.float64).reshape(shape)

    def full_shape(self, s):
        return (self.B,) + tuple(self.shapes[s])

    def value(self, s):
        key = ("v", s)
        if key not in self._cache:
            sh = self.full_shape(s)
            if s == 0:
                v = self._np(self.ext_in, sh)
            elif s == self.seg.out:
                v = self._np(self.ext_out, sh)
            else:
                off = self.g.plan.inspect(self.part, self.j, 0, s)
                v = self._np(self._ws(self.g.saved, off, int(np.prod(sh)), self.g.sdt), sh)
            self._cache[key] = v
        return self._cache[key]

    def grad(self, s):
        """dL/d(slot s) as the GPU holds it, or None."""
        key = ("g", s)
        if key not in self._cache:
            sh = self.full_shape(s)
            if s == self.seg.out:
                v = self._np(self.gout, sh)
            elif s == 0:
                v = None if self.gin is None else self._np(self.gin, sh)
            else:
                off = self.g.plan.inspect(self.part, self.j, 1, s)
                if off is not None:
                    v = self._np(self._ws(self.g.scratch, off, int(np.prod(sh)), self.g.sdt), sh)
                else:
                    # a slot read only by a residual addition has its consumer's gradient
                    cons = [n for n in self.seg.nodes if n.src == s]
                    resc = [n for n in self.seg.nodes if n.res == s]
                    v = self.grad(resc[0].dst) if (resc and not cons) else None
            self._cache[key] = v
        return self._cache[key]

    def dbn(self, b):
        """dL/d(BN output) of BN instance b masked by ReLU', as stored by the library, or None when
        the library forms it inside its BN-apply pass instead of storing it."""
        sh = self.full_shape(self.seg.bns[b])
        off = self.g.plan.inspect(self.part, self.j, 2, b)
        if off is None:
            return None
        return self._np(self._ws(self.g.scratch, off, int(np.prod(sh)), self.g.sdt), sh)

    def stats(self, b):
        C = self.shapes[self.seg.bns[b]][2]
        off = self.g.plan.inspect(self.part, self.j, 3, b)
        return self._np(self._ws(self.g.saved, off, 4 * C, self.torch.float32), (4, C))


def check_segment(view, prm, grads, st, metric, nodes=None, sample=None, seed=0):
    """{check name: error} for the nodes ``nodes`` (all by default) of one segment.

    ``prm``: the segment's parameters (host values uploaded to the GPU); ``grads``: the GPU's
    parameter gradients of the segment (``ParaRealGPU.unpack_grads``); ``st``: storage rounding;
    ``sample``: number of sampled output positions per convolution (None: whole tensors)."""
    seg = view.seg
    rng = np.random.default_rng(seed)
    err = {}
    nodes = list(range(len(seg.nodes))) if nodes is None else list(nodes)
    ostats = {}

    def stats_o(b):
        if b not in ostats:
            ostats[b] = bn_batch_stats(view.value(seg.bns[b]))
        return ostats[b]

    def act(b, rounded=True):
        a = bn_relu(view.value(seg.bns[b]), prm["gamma"][b], prm["beta"][b], stats_o(b))[0]
        return st(a) if rounded else a

    def pick(size):
        return None if sample is None or size <= sample else rng.integers(0, size, sample)

    # BN statistics of every BN a checked node reads
    for b in sorted({seg.nodes[i].bn for i in nodes if seg.nodes[i].bn >= 0}):
        gs = view.stats(b)
        mo, io = stats_o(b)
        err[f"bn{b}.mean"] = float(np.max(np.abs(gs[0] - mo) * io))     # in units of the std
        err[f"bn{b}.invstd"] = rel_inf(gs[1], io)

    # forward values
    for i in nodes:
        n = seg.nodes[i]
        src = view.value(n.src)
        res = view.value(n.res) if n.res >= 0 else None
        ext = view.ext_add if (n.dst == seg.out and view.ext_add is not None) else None
        ext = None if ext is None else view._np(ext, view.full_shape(n.dst))
        got = view.value(n.dst)
        idx = pick(got.size) if n.op == "conv" else None
        if idx is None:
            ref = node_forward(n, prm["conv"][i], prm["gamma"][n.bn] if n.bn >= 0 else None,
                               prm["beta"][n.bn] if n.bn >= 0 else None, src, res, ext, st,
                               stats_o(n.bn) if n.bn >= 0 else None)
            err[f"n{i}.fwd"] = metric(got, ref)
        else:
            a = act(n.bn) if n.bn >= 0 else src
            ref = P.conv_fwd_at(a, prm["conv"][i], n.stride, n.pad, idx)
            if res is not None:
                ref = ref + res.ravel()[idx]
            if ext is not None:
                ref = ref + ext.ravel()[idx]
            err[f"n{i}.fwd"] = metric(got.ravel()[idx], st(ref))

    # weight gradients
    for i in nodes:
        n = seg.nodes[i]
        if n.op != "conv":
            continue
        g = view.grad(n.dst)
        a = act(n.bn) if n.bn >= 0 else view.value(n.src)
        dw = grads["conv"][i]
        idx = pick(dw.size)
        if idx is None:
            ref = conv_node_backward(n, prm["conv"][i], a, g)[0]
            err[f"n{i}.dW"] = metric(dw, ref)
        else:
            err[f"n{i}.dW"] = metric(dw.ravel()[idx], P.conv_bwd_weight_at(a, g, n.k, n.stride, n.pad, idx))

    # data gradients of every slot a checked node reads
    slots = sorted({seg.nodes[i].src for i in nodes})
    for s in slots:
        cons = [k for k, n in enumerate(seg.nodes) if n.src == s and n.op != "maxpool3"]
        resc = [k for k, n in enumerate(seg.nodes) if n.res == s]
        if not cons:
            continue
        z = view.value(s)
        idx = pick(z.size)
        bn = seg.bns.index(s) if s in seg.bns and any(seg.nodes[k].bn >= 0 for k in cons) else None
        need_dx = bn is not None or view.grad(s) is not None
        if not need_dx:
            continue
        da = 0.0
        for k in cons:
            n = seg.nodes[k]
            g = view.grad(n.dst)
            if n.op == "conv":
                if idx is None:
                    d = P.conv_bwd_data(g, prm["conv"][k], z.shape, n.stride, n.pad)
                else:
                    d = P.conv_bwd_data_at(g, prm["conv"][k], z.shape, n.stride, n.pad, idx)
            else:
                d = bnact_node_backward(n, act(n.bn, rounded=False), g)
                d = d if idx is None else d.ravel()[idx]
            da = da + d
        skip = view.grad(seg.nodes[resc[0]].dst) if resc else None
        gs = view.grad(s)
        if bn is not None:
            ybn = bn_relu(z, prm["gamma"][bn], prm["beta"][bn], stats_o(bn))[1]
            dbn_gpu = view.dbn(bn)
            if dbn_gpu is not None:
                mask = (ybn > 0.0) if idx is None else (ybn.ravel()[idx] > 0.0)
                got = dbn_gpu if idx is None else dbn_gpu.ravel()[idx]
                err[f"s{s}.dbn"] = metric(got, st(da * mask))
                dbn_t = dbn_gpu
            else:
                # not held by the library (its only consumer is a 1x1 convolution, whose data
                # gradient is cheap in full): the BN backward below starts from the oracle's dbn
                assert len(cons) == 1 and seg.nodes[cons[0]].op == "conv" and seg.nodes[cons[0]].k == 1
                n = seg.nodes[cons[0]]
                da_full = P.conv_bwd_data(view.grad(n.dst), prm["conv"][cons[0]], z.shape, n.stride, n.pad)
                dbn_t = st(da_full * (ybn > 0.0))
            gx, dgamma, dbeta = bn_input_grad(z, prm["gamma"][bn], stats_o(bn), dbn_t)
            if dbn_gpu is not None:
                err[f"bn{bn}.dgamma"] = metric(grads["gamma"][bn], dgamma)
                err[f"bn{bn}.dbeta"] = metric(grads["beta"][bn], dbeta)
            else:
                # the GPU's sums run over its own dbn, which differs from the oracle's in the
                # rounding of single elements: the error of a sum is measured against the sum of
                # the magnitudes of its terms, per channel
                C = z.shape[-1]
                mean, invstd = stats_o(bn)
                ab = np.abs(dbn_t.reshape(-1, C))
                abx = np.abs(dbn_t.reshape(-1, C) * ((z.reshape(-1, C) - mean) * invstd))
                err[f"bn{bn}.dgamma"] = float(np.linalg.norm(grads["gamma"][bn] - dgamma)
                                              / np.linalg.norm(abx.sum(0)))
                err[f"bn{bn}.dbeta"] = float(np.linalg.norm(grads["beta"][bn] - dbeta)
                                             / np.linalg.norm(ab.sum(0)))
            if gs is not None:
                err[f"s{s}.grad"] = metric(gs, st(gx + (skip if skip is not None else 0.0)))
        elif gs is not None:
            ref = da + (0.0 if skip is None else (skip if idx is None else skip.ravel()[idx]))
            got = gs if idx is None else gs.ravel()[idx]
            err[f"s{s}.grad"] = metric(got, st(ref))
    return err


def check_combine_and_head(g, labels, st, metric, dx_fine):
    """Interfaces r_j = y_j - x_{j+1}, dL/dx_j = dx_j - D_{j-1} and the head, teacher-forced."""
    from oracle.net import ParaRealOracle
    to = g.to_np
    N = g.net.n_sub
    err = {}
    for j in range(N - 1):
        err[f"r{j}"] = metric(to(g.r[j]), st(to(g.y[j]) - to(g.x[j + 1])))
    for j in range(1, N):
        err[f"dx{j}.combine"] = metric(to(g.dx[j]), st(to(dx_fine[j]) - to(g.D[j - 1])))
    o = ParaRealOracle(g.net, {"head": {"w": to(g.eps)[:g.net.classes * to(g.ytilde).shape[-1]]
                                        .reshape(g.net.classes, -1), "b": to(g.eps)[-g.net.classes:]}},
                       bf16=g.net.dtype == "bf16")
    hd = o.head(to(g.ytilde), labels)
    err["loss"] = abs(float(g.loss.item()) - hd["loss"]) / abs(hd["loss"])
    err["logits"] = metric(to(g.logits), hd["logits"])
    err["D_N"] = metric(to(g.D[N - 1]), hd["D_N"])
    K = g.net.classes
    dW = to(g.deps)
    err["head.dw"] = metric(dW[:-K], hd["dw"].ravel())
    err["head.db"] = metric(dW[-K:], hd["db"])
    return err
