"""Independent library cross-check of the oracle: the same parareal network written with PyTorch
CPU float64 operators (conv2d, batch_norm in training mode, max_pool2d, linear, cross_entropy)
and differentiated by autograd.  Used only by the CPU pin tests."""
import numpy as np
import torch
import torch.nn.functional as F


def _t(a, grad=False):
    return torch.tensor(np.asarray(a), dtype=torch.float64, requires_grad=grad)


class TorchParaReal:
    def __init__(self, net, params):
        self.net = net
        self.leaves = {}

        def seg_params(tag, seg, prm):
            out = {"conv": [], "gamma": [], "beta": []}
            for i, w in enumerate(prm["conv"]):
                if w is None:
                    out["conv"].append(None)
                else:    # [o][r][s][c] -> [o][c][r][s]
                    t = _t(np.transpose(w, (0, 3, 1, 2)), True)
                    self.leaves[(tag, "conv", i)] = t
                    out["conv"].append(t)
            for b in range(len(seg.bns)):
                g, be = _t(prm["gamma"][b], True), _t(prm["beta"][b], True)
                self.leaves[(tag, "gamma", b)] = g
                self.leaves[(tag, "beta", b)] = be
                out["gamma"].append(g)
                out["beta"].append(be)
            return out

        self.pre = [seg_params(("pre", j), s, p) for j, (s, p) in enumerate(zip(net.pre, params["pre"]))]
        self.fine = [seg_params(("fine", j), s, p) for j, (s, p) in enumerate(zip(net.fine, params["fine"]))]
        self.coarse = [seg_params(("coarse", j), s, p)
                       for j, (s, p) in enumerate(zip(net.coarse, params["coarse"]))]
        self.hw = _t(params["head"]["w"], True)
        self.hb = _t(params["head"]["b"], True)

    @staticmethod
    def segment(seg, prm, x):
        slots = {0: x}
        for i, n in enumerate(seg.nodes):
            def act():
                z = slots[n.src]
                y = F.batch_norm(z, None, None, prm["gamma"][n.bn], prm["beta"][n.bn],
                                 training=True, eps=1e-5)
                return F.relu(y)
            if n.op == "conv":
                a = act() if n.bn >= 0 else slots[n.src]
                y = F.conv2d(a, prm["conv"][i], stride=n.stride, padding=n.pad)
            elif n.op == "bnact":
                y = act()
                if n.pool == 2:
                    y = F.max_pool2d(y, 2, 2)
            else:
                y = F.max_pool2d(slots[n.src], 3, 2, 1)
            if n.res >= 0:
                y = y + slots[n.res]
            slots[n.dst] = y
        return slots[seg.out]

    def loss(self, x_nhwc, labels):
        net = self.net
        N = net.n_sub
        x = _t(np.transpose(x_nhwc, (0, 3, 1, 2)))
        xs = [self.segment(net.pre[j], self.pre[j], x) for j in range(N)]
        ys = [self.segment(net.fine[j], self.fine[j], xs[j]) for j in range(N)]
        if N == 1:
            yt = ys[0]
        else:
            r = [ys[j] - xs[j + 1] for j in range(N - 1)] + [torch.zeros_like(ys[N - 1])]
            rt = r[0]
            for j in range(N - 1):
                rt = r[j + 1] + self.segment(net.coarse[j], self.coarse[j], rt)
            yt = ys[N - 1] + rt
        logits = F.linear(yt.mean(dim=(2, 3)), self.hw, self.hb)
        return F.cross_entropy(logits, torch.tensor(labels, dtype=torch.long)), logits
