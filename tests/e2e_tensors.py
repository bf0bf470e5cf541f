"""Names of the tensors of one training step, taken from the oracle's results or from the GPU's
buffers, so that whole steps can be compared tensor by tensor (tests/test_gpu_e2e_bf16.py) and the
oracle can be compared with itself (tests/golden/conditioning.py)."""
from __future__ import annotations

import numpy as np


def rel_2(a, ref):
    a, ref = np.asarray(a), np.asarray(ref)
    return float(np.linalg.norm((a - ref).ravel()) / max(np.linalg.norm(ref.ravel()), 1e-30)) if ref.size else 0.0


def rel_inf(a, ref):
    a, ref = np.asarray(a), np.asarray(ref)
    return float(np.abs(a - ref).max() / max(np.abs(ref).max(), 1e-30)) if ref.size else 0.0


def family(name):
    """Tensor family of a compared tensor: forward values, D_j, dL/dx_j, the head's gradients, and
    the parameter gradients by part (pre / fine / coarse) and kind (conv filters / BN gamma, beta)."""
    if name in ("loss", "logits", "ytilde") or name[0] in "xyr":
        return "forward"
    if name.startswith("D"):
        return "D"
    if name.startswith("dx"):
        return "dx"
    if name.startswith("head"):
        return "head"
    part, key = name.split(".", 1)
    kind = "conv" if key.startswith("conv") else "bn"
    return part.rstrip("0123456789") + "." + kind


def grad_named(name, j, grads):
    """{name: array} of one segment's parameter gradients ({'conv': [...], 'gamma': [...], ...})."""
    out = {}
    for key in ("conv", "gamma", "beta"):
        for i, a in enumerate(grads[key]):
            if a is not None:
                out[f"{name}{j}.{key}{i}"] = a
    return out


def oracle_tensors(net, fwd, hd, bwd):
    """{name: array} of one oracle step (``ParaRealOracle.step``)."""
    N = net.n_sub
    t = {"logits": hd["logits"], "ytilde": fwd["ytilde"]}
    for j in range(N):
        t[f"x{j}"], t[f"y{j}"] = fwd["x"][j], fwd["y"][j]
        t[f"D{j}"], t[f"dx{j}"] = bwd["D"][j], bwd["dx"][j]
    for j in range(N - 1):
        t[f"r{j}"] = fwd["r"][j]
    for j in range(1, N - 1):
        t[f"rt{j}"] = fwd["rt"][j]
    t["head.dw"], t["head.db"] = hd["dw"], hd["db"]
    for name, ref in (("pre", bwd["ddelta"]), ("fine", bwd["dphi"]), ("coarse", bwd["deta"])):
        for j, r in enumerate(ref):
            if r is not None:
                t.update(grad_named(name, j, r))
    return t


def gpu_tensors(g):
    """{name: array} of the GPU's buffers after one step (``ParaRealGPU``), float64."""
    net, to = g.net, g.to_np
    N = net.n_sub
    t = {"logits": to(g.logits), "ytilde": to(g.ytilde)}
    for j in range(N):
        t[f"x{j}"], t[f"y{j}"] = to(g.x[j]), to(g.y[j])
        t[f"D{j}"], t[f"dx{j}"] = to(g.D[j]), to(g.dx[j])
    for j in range(N - 1):
        t[f"r{j}"] = to(g.r[j])
    for j in range(1, N - 1):
        t[f"rt{j}"] = to(g.rt[j])
    dW = to(g.deps)
    K = net.classes
    t["head.dw"], t["head.db"] = dW[:-K].reshape(K, -1), dW[-K:]
    for part, name in ((0, "pre"), (1, "fine"), (2, "coarse")):
        for j in range(len([net.pre, net.fine, net.coarse][part])):
            gr = g.unpack_grads(part, j)
            if any(a is not None for a in gr["conv"]) or gr["gamma"]:
                t.update(grad_named(name, j, gr))
    return t


def compare(got, ref):
    """{name: (e_2, e_inf)} over the names of ``ref`` (both dicts of arrays)."""
    return {k: (rel_2(got[k], ref[k]), rel_inf(got[k], ref[k])) for k in ref}


def bf16_ulp_up(v):
    """The next bfloat16 value above each (bf16-representable, finite) element of v."""
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(v)                      # v = m 2^e, 0.5 <= |m| < 1: one ulp is 2^(e - 8)
    step = np.ldexp(1.0, e - 8)
    step = np.where((v < 0) & (m == -0.5), step / 2, step)   # -2^k: the spacing above is finer
    return np.where(v == 0.0, 2.0 ** -133, v + step)


def perturb_ulp(a, count, seed):
    """Copy of the bf16-valued array ``a`` with ``count`` seeded elements moved up by one bf16 ulp."""
    rng = np.random.default_rng(seed)
    b = np.array(a, dtype=np.float64, copy=True)
    idx = rng.choice(b.size, size=count, replace=False)
    flat = b.reshape(-1)
    flat[idx] = bf16_ulp_up(flat[idx])
    return b
