"""One training step of a parareal network on the GPU: the libpnn entry points in the order of
Alg. para2 (forward) and Alg. para3 (backward), on device buffers allocated through PyTorch.

PyTorch provides device memory, host<->device copies of inputs / results and the stream; every
step of the network itself runs in libpnn's kernels.
"""
from __future__ import annotations

import numpy as np

from . import binding as B


def _torch():
    import torch
    return torch


def bf16_bits(f):
    """float32 array -> bfloat16 bit patterns (uint16), rounded to nearest even; NaN stays NaN."""
    u = np.ascontiguousarray(f, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        r[nan] = 0x7FC0
    return r


class ParaRealGPU:
    """Device state of one parareal network (``pnn_synth.Net``) and its training step."""

    def __init__(self, net, params=None, device="cuda"):
        torch = _torch()
        if not torch.cuda.is_available():
            raise RuntimeError("ParaRealGPU needs a GPU (HIP device)")
        self.net = net
        self.plan = B.Plan(net)
        B.pnn_set_streams(self.plan, 4)   # the fine sub-network groups on up to 4 streams
        self.coarse_chain_all = True      # coarse_bwd_all (deferred coarse weight gradients)
        self.overlap_bwd = False          # parareal_bwd: the coarse chain overlapped with the fine backward
        self.coarse_fwd_chain = True      # coarse_fwd_all (input BN sums from the previous block)
        self.dev = torch.device(device)
        self.sdt = torch.bfloat16 if net.dtype == "bf16" else torch.float32
        N, Bt = net.n_sub, net.batch
        u8 = dict(dtype=torch.uint8, device=self.dev)
        f32 = dict(dtype=torch.float32, device=self.dev)
        act = dict(dtype=self.sdt, device=self.dev)

        def pbuf(part, j, grad):
            _, tot = self.plan.param_layout(part, j, grad)
            return torch.zeros(max(tot, 256), **u8)

        self.delta = [pbuf(0, j, 0) for j in range(N)]
        self.phi = [pbuf(1, j, 0) for j in range(N)]
        self.eta = [pbuf(2, j, 0) for j in range(N - 1)]
        self.ddelta = [pbuf(0, j, 1) for j in range(N)]
        self.dphi = [pbuf(1, j, 1) for j in range(N)]
        self.deta = [pbuf(2, j, 1) for j in range(N - 1)]
        xs = [self.plan.tensor_shape(0, j) for j in range(N)]
        ys = [self.plan.tensor_shape(1, j) for j in range(N)]
        self.x = [torch.zeros((Bt,) + s, **act) for s in xs]
        self.y = [torch.zeros((Bt,) + s, **act) for s in ys]
        self.r = [torch.zeros((Bt,) + ys[j], **act) for j in range(N - 1)]
        # rt_0 = r_0 (eq. (tilderk)); rt_j for 1 <= j <= N-2; ytilde in X_N
        self.rt = ([self.r[0]] if N > 1 else []) + [torch.zeros((Bt,) + ys[j], **act) for j in range(1, N - 1)]
        self.ytilde = torch.zeros((Bt,) + ys[N - 1], **act) if N > 1 else self.y[0]
        self.D = [torch.zeros((Bt,) + ys[j], **act) for j in range(N)]
        self.dx = [torch.zeros((Bt,) + s, **act) for s in xs]
        self.rnorm2 = torch.zeros(max(N - 1, 1), **f32)
        C = ys[N - 1][2]
        K = net.classes
        self.eps = torch.zeros(K * C + K, **f32)
        self.deps = torch.zeros(K * C + K, **f32)
        self.loss = torch.zeros(1, **f32)
        self.logits = torch.zeros((Bt, K), **f32)
        self.image = torch.zeros((Bt,) + tuple(net.in_shape), **act)
        self.labels = torch.zeros(Bt, dtype=torch.int32, device=self.dev)
        self.saved = torch.zeros(max(self.plan.workspace_size(B.PNN_WS_SAVED), 256), **u8)
        self.scratch = torch.zeros(max(self.plan.workspace_size(B.PNN_WS_SCRATCH), 256), **u8)
        if params is not None:
            self.load_params(params)

    # -- marshalling -----------------------------------------------------------------------------
    def _pack(self, part, j, seg, prm):
        offs, tot = self.plan.param_layout(part, j, 0)
        buf = np.zeros(max(tot, 256), dtype=np.uint8)
        n = len(seg.nodes)
        for i, w in enumerate(prm["conv"]):
            if w is None:
                continue
            f = np.ascontiguousarray(w, dtype=np.float32)
            raw = bf16_bits(f).tobytes() if self.net.dtype == "bf16" else f.tobytes()
            buf[offs[i]:offs[i] + len(raw)] = np.frombuffer(raw, dtype=np.uint8)
        for b in range(len(seg.bns)):
            for k, key in enumerate(("gamma", "beta")):
                raw = np.ascontiguousarray(prm[key][b], dtype=np.float32).tobytes()
                o = offs[n + 2 * b + k]
                buf[o:o + len(raw)] = np.frombuffer(raw, dtype=np.uint8)
        return buf

    def load_params(self, params):
        torch = _torch()
        net = self.net
        for part, segs, dst in ((0, net.pre, self.delta), (1, net.fine, self.phi), (2, net.coarse, self.eta)):
            key = ("pre", "fine", "coarse")[part]
            for j, seg in enumerate(segs):
                dst[j].copy_(torch.from_numpy(self._pack(part, j, seg, params[key][j])))
        h = params["head"]
        self.eps.copy_(torch.from_numpy(np.concatenate([h["w"].ravel(), h["b"]]).astype(np.float32)))

    def load_input(self, x, labels):
        torch = _torch()
        self.image.copy_(torch.from_numpy(np.asarray(x, dtype=np.float32)).to(self.sdt))
        self.labels.copy_(torch.from_numpy(np.asarray(labels, dtype=np.int32)))

    def unpack_grads(self, part, j):
        """{'conv': [dW or None], 'gamma': [...], 'beta': [...]} of one segment, float64."""
        net = self.net
        seg = [net.pre, net.fine, net.coarse][part][j]
        buf = [self.ddelta, self.dphi, self.deta][part][j].cpu().numpy()
        offs, _ = self.plan.param_layout(part, j, 1)
        from pnn_synth.gen import segment_shapes
        sh = segment_shapes(seg)
        out = {"conv": [], "gamma": [], "beta": []}
        n = len(seg.nodes)
        for i, nd in enumerate(seg.nodes):
            if nd.op != "conv":
                out["conv"].append(None)
                continue
            cnt = nd.cout * nd.k * nd.k * sh[nd.src][2]
            a = buf[offs[i]:offs[i] + 4 * cnt].view(np.float32).astype(np.float64)
            out["conv"].append(a.reshape(nd.cout, nd.k, nd.k, sh[nd.src][2]))
        for b, s in enumerate(seg.bns):
            C = sh[s][2]
            for k, key in enumerate(("gamma", "beta")):
                o = offs[n + 2 * b + k]
                out[key].append(buf[o:o + 4 * C].view(np.float32).astype(np.float64))
        return out

    @staticmethod
    def to_np(t):
        return t.detach().float().cpu().numpy().astype(np.float64)

    # -- the step ----------------------------------------------------------------------------------
    def stream(self):
        return _torch().cuda.current_stream().cuda_stream

    def forward(self, s=None, rnorm=False, fine_events=None, coarse_events=None):
        """Alg. para2 and the head (loss, D_N).  ``fine_events`` / ``coarse_events``: pairs of
        torch.cuda.Event recorded (on torch's current stream) around parareal_fine_fwd / the
        coarse chain."""
        s = self.stream() if s is None else s
        p, N = self.plan, self.net.n_sub
        B.pnn_pre_fwd(p, self.image, self.x, self.delta, self.saved, self.scratch, s)
        if fine_events:
            fine_events[0].record()
        B.parareal_fine_fwd(p, self.x, self.phi, self.y, self.saved, self.scratch, s)
        if fine_events:
            fine_events[1].record()
        if N > 1:
            B.parareal_combine_fwd(p, self.y, self.x, self.r, self.rnorm2 if rnorm else None,
                                   self.scratch, s)
            if coarse_events:
                coarse_events[0].record()
            self._coarse_forward(s)
            if coarse_events:
                coarse_events[1].record()
        B.pnn_head_fwd_bwd(p, self.ytilde, self.eps, self.labels, self.logits, self.loss,
                           self.D[N - 1], self.deps, self.scratch, s)

    def _coarse_forward(self, s):
        """The coarse chain rt_{j+1} = add_j + F^j(rt_j), j = 0..N-2 (ytilde last)."""
        p, N = self.plan, self.net.n_sub
        adds = [self.r[j + 1] for j in range(N - 2)] + [self.y[N - 1]]
        outs = [self.rt[j + 1] for j in range(N - 2)] + [self.ytilde]
        if self.coarse_fwd_chain:
            B.coarse_fwd_all(p, [self.rt[0]] + outs, self.eta, adds, self.saved, self.scratch, s)
        else:
            for j in range(N - 1):
                B.coarse_fwd(p, j, self.rt[j], self.eta[j], adds[j], outs[j], self.saved, self.scratch, s)

    def backward(self, s=None, fine_events=None, coarse_events=None):
        """Alg. para3.  ``fine_events`` / ``coarse_events`` as in ``forward``, around
        parareal_fine_bwd / the coarse chain."""
        self.backward_coarse_fine(s, fine_events, coarse_events)
        self.backward_pre(s)

    def backward_coarse_fine(self, s=None, fine_events=None, coarse_events=None):
        """The coarse chain D_j (j = N-1..1) and the fine sub-networks' gradients.  With
        ``overlap_bwd`` (and N > 1) both run in one parareal_bwd call, which starts each group of
        fine sub-networks as soon as the chain has produced its D_j; ``fine_events`` then bracket
        that call and ``coarse_events`` are not recorded."""
        s = self.stream() if s is None else s
        p, N = self.plan, self.net.n_sub
        if self.overlap_bwd and N > 1:
            if fine_events:
                fine_events[0].record()
            B.parareal_bwd(p, self.D, self.rt, self.eta, self.deta, self.x, self.phi, self.dx, self.dphi,
                           self.saved, self.scratch, s)
            if fine_events:
                fine_events[1].record()
            return
        if coarse_events:
            coarse_events[0].record()
        if N > 1 and self.coarse_chain_all:
            B.coarse_bwd_all(p, self.D, self.rt, self.eta, self.saved, self.deta, self.scratch, s)
        else:
            for j in range(N - 2, -1, -1):
                B.coarse_bwd(p, j, self.D[j + 1], self.rt[j], self.eta[j], self.saved, self.D[j],
                             self.deta[j], self.scratch, s)
        if coarse_events:
            coarse_events[1].record()
        if fine_events:
            fine_events[0].record()
        B.parareal_fine_bwd(p, self.D, self.x, self.phi, self.saved, self.dx, self.dphi, self.scratch, s)
        if fine_events:
            fine_events[1].record()

    def backward_pre(self, s=None):
        """dL/dx_j -= D_{j-1}, then the preprocessing operators' gradients."""
        s = self.stream() if s is None else s
        p = self.plan
        B.parareal_combine_bwd(p, self.dx, self.D, s)
        B.pnn_pre_bwd(p, self.image, self.dx, self.delta, self.saved, self.ddelta, self.scratch, s)

    def step(self, s=None):
        self.forward(s)
        self.backward(s)

    # -- HIP graphs ---------------------------------------------------------------------------
    def _parts(self):
        """The step's library calls in order, as parts that are captured one graph each (so that
        the fine and coarse parts can still be timed between replays)."""
        p, N = self.plan, self.net.n_sub
        st = self.stream

        def coarse_fwd():
            self._coarse_forward(st())

        def coarse_bwd():
            if self.coarse_chain_all:
                B.coarse_bwd_all(p, self.D, self.rt, self.eta, self.saved, self.deta, self.scratch, st())
            else:
                for j in range(N - 2, -1, -1):
                    B.coarse_bwd(p, j, self.D[j + 1], self.rt[j], self.eta[j], self.saved, self.D[j],
                                 self.deta[j], self.scratch, st())

        parts = {
            "pre_fwd": lambda: B.pnn_pre_fwd(p, self.image, self.x, self.delta, self.saved, self.scratch, st()),
            "fine_fwd": lambda: B.parareal_fine_fwd(p, self.x, self.phi, self.y, self.saved, self.scratch, st()),
            "combine_fwd": lambda: B.parareal_combine_fwd(p, self.y, self.x, self.r, None, self.scratch, st()),
            "coarse_fwd": coarse_fwd,
            "head": lambda: B.pnn_head_fwd_bwd(p, self.ytilde, self.eps, self.labels, self.logits, self.loss,
                                               self.D[N - 1], self.deps, self.scratch, st()),
            "coarse_bwd": coarse_bwd,
            "fine_bwd": lambda: B.parareal_fine_bwd(p, self.D, self.x, self.phi, self.saved, self.dx, self.dphi,
                                                    self.scratch, st()),
            "pre_bwd": lambda: self.backward_pre(st()),
        }
        if N == 1:
            for k in ("combine_fwd", "coarse_fwd", "coarse_bwd"):
                del parts[k]
        return parts

    def capture(self, whole=False):
        """Capture one training step (forward and backward, as ``forward`` + ``backward`` run it)
        into HIP graphs (no eager step is needed first: the library's calls create nothing).  A
        replay repeats the step on what the buffers hold then.  ``whole=False``: one graph per part
        (the fine and coarse parts can be timed between replays; the backward's calls separate);
        ``whole=True``: the forward as one graph and the backward as another, the backward as
        ``overlap_bwd`` makes it (the coarse chain overlapped with the fine backward, its fork and
        join across the plan's side streams captured with it)."""
        torch = _torch()
        self.graphs = {}
        self.whole = whole
        parts = {"fwd": self.forward, "bwd": self.backward} if whole else self._parts()
        for name, fn in parts.items():
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                fn()
            self.graphs[name] = g
        torch.cuda.synchronize()

    def replay_forward(self, fine_events=None, coarse_events=None):
        """``forward`` from the captured graphs; the events as in ``forward`` (whole-step graphs:
        none)."""
        G = self.graphs
        if getattr(self, "whole", False):
            G["fwd"].replay()
            return
        G["pre_fwd"].replay()
        if fine_events:
            fine_events[0].record()
        G["fine_fwd"].replay()
        if fine_events:
            fine_events[1].record()
        if "coarse_fwd" in G:
            G["combine_fwd"].replay()
            if coarse_events:
                coarse_events[0].record()
            G["coarse_fwd"].replay()
            if coarse_events:
                coarse_events[1].record()
        G["head"].replay()

    def replay_backward(self, fine_events=None, coarse_events=None):
        """``backward`` from the captured graphs; the events as in ``backward`` (whole-step graphs:
        none)."""
        G = self.graphs
        if getattr(self, "whole", False):
            G["bwd"].replay()
            return
        if coarse_events:
            coarse_events[0].record()
        if "coarse_bwd" in G:
            G["coarse_bwd"].replay()
        if coarse_events:
            coarse_events[1].record()
        if fine_events:
            fine_events[0].record()
        G["fine_bwd"].replay()
        if fine_events:
            fine_events[1].record()
        G["pre_bwd"].replay()

    # -- parameter update (SGD with momentum; include/pnn.h pnn_sgd_step) -------------------------
    def sgd_init(self, master=True):
        """Zeroed momentum buffers laid out like the gradient buffers; for bf16 networks (with
        ``master``) also fp32 master copies of the filters, filled from the stored filters by the
        first step."""
        torch = _torch()
        self.mom = [[torch.zeros_like(b, dtype=torch.uint8) for b in bufs]
                    for bufs in (self.ddelta, self.dphi, self.deta)]
        self.mom.append([torch.zeros_like(self.deps)])
        self.master = None
        if master and self.net.dtype == "bf16":
            self.master = [[torch.zeros_like(b, dtype=torch.uint8) for b in bufs]
                           for bufs in (self.ddelta, self.dphi, self.deta)]
        self._master_fresh = True

    def sgd_step(self, lr, mu=0.9, weight_decay=1e-4, nesterov=True, s=None):
        s = self.stream() if s is None else s
        if not hasattr(self, "mom"):
            self.sgd_init()
        parts = ((self.delta, self.ddelta), (self.phi, self.dphi), (self.eta, self.deta), ([self.eps], [self.deps]))
        for part, (pb, gb) in enumerate(parts):
            if not pb:
                continue
            m = self.master[part] if (self.master is not None and part < 3) else None
            B.pnn_sgd_step(self.plan, part, pb, gb, self.mom[part], lr, mu, weight_decay, nesterov, s,
                           master=m, master_init=self._master_fresh)
        self._master_fresh = False
