"""GPU parity of the parameter update (pnn_sgd_step through the C ABI) against the fp64 oracle
(oracle/sgd.py), teacher-forced per call: every tensor of every part, two Nesterov steps in a row
(the second reads the momentum the first wrote) and one plain-momentum step.

Bar: the fp32 evaluation's rounding bound, 8 * 2^-24 times the magnitude of the terms that form
each result (|mu v| + |g| + wd |w| for the momentum, |w| + lr |update| for the parameter), and for
bf16 parameters half a bf16 ulp more (round to nearest even of the fp32 result)."""
import numpy as np
import pytest

import pnn_synth as S

pytestmark = pytest.mark.gpu


def _tensors(g, part, j):
    """(param offset, grad offset, count, stored as float) of every tensor of one segment."""
    net = g.net
    if part == 3:
        return [(0, 0, g.eps.numel(), True)]
    seg = [net.pre, net.fine, net.coarse][part][j]
    sh = S.segment_shapes(seg)
    po, _ = g.plan.param_layout(part, j, 0)
    go, _ = g.plan.param_layout(part, j, 1)
    out = []
    n = len(seg.nodes)
    for i, nd in enumerate(seg.nodes):
        if nd.op == "conv":
            out.append((po[i], go[i], nd.cout * nd.k * nd.k * sh[nd.src][2], net.dtype == "f32"))
    for b, s in enumerate(seg.bns):
        for k in range(2):
            out.append((po[n + 2 * b + k], go[n + 2 * b + k], sh[s][2], True))
    return out


def _bufs(g, part):
    if part == 3:
        return [g.eps], [g.deps]
    return [(g.delta, g.ddelta), (g.phi, g.dphi), (g.eta, g.deta)][part]


def _f32(buf, off, cnt):
    return buf[off:off + 4 * cnt].view(np.float32).astype(np.float64)


def _param(buf, off, cnt, f32):
    if f32:
        return _f32(buf, off, cnt)
    raw = buf[off:off + 2 * cnt].view(np.uint16).astype(np.uint32) << 16
    return raw.view(np.float32).astype(np.float64)


def _bf16_ulp(x):
    e = np.floor(np.log2(np.maximum(np.abs(x), 1e-38)))
    return 2.0 ** (e - 7)


def _check_step(g, lr, mu, wd, nesterov):
    import torch
    from oracle.sgd import sgd_step
    host = lambda t: t.detach().cpu().numpy().view(np.uint8).copy()
    before = {}
    for part in range(4):
        pb, gb = _bufs(g, part)
        before[part] = [(host(pb[j]), host(gb[j]), host(g.mom[part][j])) for j in range(len(pb))]
    g.sgd_step(lr, mu, wd, nesterov)
    torch.cuda.synchronize()
    worst = 0.0
    for part in range(4):
        pb, _ = _bufs(g, part)
        for j in range(len(pb)):
            p0, g0, v0 = before[part][j]
            p1, v1 = host(pb[j]), host(g.mom[part][j])
            for (po, go, cnt, f32) in _tensors(g, part, j):
                w0, g0_, v0_ = _param(p0, po, cnt, f32), _f32(g0, go, cnt), _f32(v0, go, cnt)
                w_ref, v_ref = sgd_step(w0, g0_, v0_, lr, mu, wd, nesterov)
                w_got, v_got = _param(p1, po, cnt, f32), _f32(v1, go, cnt)
                m_d = np.abs(g0_) + wd * np.abs(w0)
                m_v = mu * np.abs(v0_) + m_d
                m_w = np.abs(w0) + lr * ((m_d + mu * m_v) if nesterov else m_v)
                eps = 8 * 2.0 ** -24
                assert np.all(np.abs(v_got - v_ref) <= eps * m_v + 1e-30), (part, j, po)
                bound = eps * m_w + 1e-30
                if not f32:
                    bound = bound + 0.5 * _bf16_ulp(w_ref)
                err = np.abs(w_got - w_ref)
                assert np.all(err <= bound), (part, j, po, float(np.max(err / bound)))
                worst = max(worst, float(np.max(err / bound)))
    return worst


@pytest.mark.parametrize("idx,batch", [(0, 2), (2, 2)])
def test_sgd_step_matches_oracle(idx, batch):
    import torch
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    g.load_input(x, labels)
    g.forward()
    g.backward()
    g.sgd_init()
    gen = torch.Generator(device="cuda").manual_seed(11)
    for bufs in g.mom:                   # non-zero momentum: the first step exercises mu * v too
        for b in bufs:
            f = b.view(torch.float32) if b.dtype == torch.uint8 else b
            f.copy_(torch.randn(f.shape, generator=gen, device="cuda") * 1e-3)
    wd = 1e-4 if idx else 5e-4
    print(f"[sgd] {net.name}: worst error / bound",
          [_check_step(g, 0.1, 0.9, wd, True), _check_step(g, 0.1, 0.9, wd, True),
           _check_step(g, 0.05, 0.9, wd, False)], flush=True)
