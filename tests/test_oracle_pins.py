"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU needed).

Each test names the pin it implements; together they are meant to catch a dropped term, a wrong
sign or index, or a transposed operand anywhere in the oracle.
"""
import copy
import json
import math
import os

import numpy as np
import pytest

import pnn_synth as S
from pnn_synth.nets import Net, _SegBuilder, resnet_parareal, vgg_parareal, tiny_parareal
from oracle import prim as P
from oracle.net import ParaRealOracle, param_count, receptive_field, seg_forward

GOLD = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(12345)


# ----------------------------------------------------------------------------------------------
# small networks of every form the configs use
# ----------------------------------------------------------------------------------------------

def mini_resnet(n_sub=3, batch=2, hw=8, seeds=(11, 12, 13)):
    return resnet_parareal("mini-resnet", batch, hw, n_sub, 5, "f32", seeds,
                           units_per_stage=2, widths=(8, 16, 32), stem=4)


def mini_vgg(batch=2, seeds=(21, 22, 23)):
    return vgg_parareal("mini-vgg", batch, 16, 5, "f32", seeds,
                        split=[[[4], [8, 8]], [[8, 8]], [[16]]], stem=4)


def mini_tiny(batch=2, seeds=(31, 32, 33)):
    return tiny_parareal("mini-tiny", batch, 8, 4, 3, 5, "f32", seeds)


MINIS = {"resnet": mini_resnet, "vgg": mini_vgg, "tiny": mini_tiny}


# ----------------------------------------------------------------------------------------------
# P1: convolution against a matrix product, an identity kernel and a shift; adjoint identities
# ----------------------------------------------------------------------------------------------

def test_p1_conv1x1_is_matmul():
    x = rng.standard_normal((2, 5, 7, 6))
    w = rng.standard_normal((4, 1, 1, 6))
    y = P.conv_fwd(x, w, 1, 0)
    np.testing.assert_allclose(y, (x.reshape(-1, 6) @ w[:, 0, 0, :].T).reshape(2, 5, 7, 4), rtol=1e-13)
    y2 = P.conv_fwd(x, w, 2, 0)          # stride 2 = subsample then matmul
    xs = x[:, ::2, ::2, :]
    np.testing.assert_allclose(y2, (xs.reshape(-1, 6) @ w[:, 0, 0, :].T).reshape(xs.shape[:3] + (4,)),
                               rtol=1e-13)


def test_p1_identity_and_shift_kernels():
    x = rng.standard_normal((2, 6, 5, 3))
    w = np.zeros((3, 3, 3, 3))
    for c in range(3):
        w[c, 1, 1, c] = 1.0
    np.testing.assert_array_equal(P.conv_fwd(x, w, 1, 1), x)
    # single tap at (r, s) = (0, 2): y[p, q] = x[p - 1, q + 1] with zero fill (cross-correlation)
    w = np.zeros((3, 3, 3, 3))
    for c in range(3):
        w[c, 0, 2, c] = 1.0
    y = P.conv_fwd(x, w, 1, 1)
    ref = np.zeros_like(x)
    ref[:, 1:, :-1, :] = x[:, :-1, 1:, :]
    np.testing.assert_array_equal(y, ref)


@pytest.mark.parametrize("k,st,pad,H", [(3, 1, 1, 7), (3, 2, 1, 8), (1, 2, 0, 8), (3, 2, 1, 7), (1, 1, 0, 5)])
def test_p1_conv_backward_adjoints(k, st, pad, H):
    """<conv(x, w), g> = <x, dgrad(g, w)> = <w, wgrad(x, g)> (bilinearity, exact up to rounding)."""
    x = rng.standard_normal((2, H, H + 1, 5))
    w = rng.standard_normal((6, k, k, 5))
    y = P.conv_fwd(x, w, st, pad)
    g = rng.standard_normal(y.shape)
    lhs = float((y * g).sum())
    np.testing.assert_allclose(float((x * P.conv_bwd_data(g, w, x.shape, st, pad)).sum()), lhs, rtol=1e-12)
    np.testing.assert_allclose(float((w * P.conv_bwd_weight(x, g, k, st, pad)).sum()), lhs, rtol=1e-12)


@pytest.mark.parametrize("k,st,pad,H", [(3, 1, 1, 7), (3, 2, 1, 8), (1, 2, 0, 8)])
def test_sampled_conv_primitives_match_full(k, st, pad, H):
    """The sampled-output evaluations equal the full definitions at the sampled indices."""
    x = rng.standard_normal((2, H, H, 5))
    w = rng.standard_normal((6, k, k, 5))
    y = P.conv_fwd(x, w, st, pad)
    g = rng.standard_normal(y.shape)
    for full, f in ((y, lambda i: P.conv_fwd_at(x, w, st, pad, i)),
                    (P.conv_bwd_data(g, w, x.shape, st, pad), lambda i: P.conv_bwd_data_at(g, w, x.shape, st, pad, i)),
                    (P.conv_bwd_weight(x, g, k, st, pad), lambda i: P.conv_bwd_weight_at(x, g, k, st, pad, i))):
        idx = rng.integers(0, full.size, 50)
        np.testing.assert_array_equal(f(idx), full.ravel()[idx])


def test_maxpool_definition_and_tie_rule():
    x = np.array([[1.0, 3.0, 3.0, 0.0], [2.0, 3.0, -1.0, 5.0]]).reshape(1, 2, 4, 1)
    y = P.maxpool_fwd(x, 2, 2, 0)
    np.testing.assert_array_equal(y.ravel(), [3.0, 5.0])
    gx = P.maxpool_bwd(x, np.array([10.0, 20.0]).reshape(1, 1, 2, 1), 2, 2, 0)
    ref = np.zeros(8)
    ref[1] = 10.0          # first maximum in row-major window order
    ref[7] = 20.0
    np.testing.assert_array_equal(gx.ravel(), ref)
    # 3x3 / 2 / pad 1: padding never wins even when every value is negative
    x = -1.0 - rng.random((1, 4, 4, 2))
    y = P.maxpool_fwd(x, 3, 2, 1)
    assert y.shape == (1, 2, 2, 2)
    np.testing.assert_array_equal(y[0, 0, 0], x[0, :2, :2].reshape(-1, 2).max(0))
    np.testing.assert_array_equal(y[0, 1, 1], x[0, 1:4, 1:4].reshape(-1, 2).max(0))


# ----------------------------------------------------------------------------------------------
# P2 / P3: batch normalisation closed form and backward invariants
# ----------------------------------------------------------------------------------------------

def _bnact_segment(shape):
    b = _SegBuilder(shape)
    return b.done(b.bnact(0))


def test_p2_bn_forward_moments():
    C = 5
    z = 3.0 + 2.0 * rng.standard_normal((4, 6, 6, C))
    gamma, beta = rng.random(C) + 0.5, rng.standard_normal(C)
    seg = _bnact_segment((6, 6, C))
    run = seg_forward(seg, {"conv": [None], "gamma": [gamma], "beta": [beta]}, z, lambda a: a)[1]
    _, ybn = run.bn_forward(0)
    zz = z.reshape(-1, C)
    var = zz.var(axis=0)
    np.testing.assert_allclose(ybn.reshape(-1, C).mean(0), beta, atol=1e-12)
    np.testing.assert_allclose(ybn.reshape(-1, C).var(0), gamma ** 2 * var / (var + 1e-5), rtol=1e-12)


def test_bn_statistics_of_a_large_mean_tensor():
    """Batch statistics of a channel whose mean is 1e6 times its spread: values 1e6 + k / 8 for
    k = 0..7 (exact in fp64) have mean 1e6 + 7/16 and biased variance (63/12) / 64 = 21/256 in closed
    form; the two-pass statistics reproduce them to fp64 rounding (a one-pass E[z^2] - mean^2 in
    fp64 would lose about 12 of its 16 digits here)."""
    from oracle.net import bn_batch_stats
    z = (1e6 + np.arange(8) / 8.0).reshape(2, 2, 2, 1)
    mean, invstd = bn_batch_stats(z)
    assert mean[0] == 1e6 + 7.0 / 16.0
    np.testing.assert_allclose(1.0 / invstd[0] ** 2 - 1e-5, 21.0 / 256.0, rtol=1e-9)


def test_p3_bn_backward_invariants():
    """For x -> BN(x) (ReLU not reached): sum dx = 0 and, with eps > 0,
    sum dx * xhat = gamma * invstd * dgamma * eps / (var + eps)  (0 in the eps -> 0 limit)."""
    from oracle.net import seg_backward
    C = 4
    z = rng.standard_normal((3, 5, 5, C))
    seg = _bnact_segment((5, 5, C))
    prm = {"conv": [None], "gamma": [np.ones(C)], "beta": [np.full(C, 50.0)]}   # ReLU is identity
    out, run = seg_forward(seg, prm, z, lambda a: a)
    g = rng.standard_normal(out.shape)
    dx, grads = seg_backward(run, g, lambda a: a)
    var = z.reshape(-1, C).var(0)
    xhat = (z - z.reshape(-1, C).mean(0)) / np.sqrt(var + 1e-5)
    np.testing.assert_allclose(dx.reshape(-1, C).sum(0), 0.0, atol=1e-11)
    dgamma = (g * xhat).reshape(-1, C).sum(0)
    np.testing.assert_allclose(grads["gamma"][0], dgamma, rtol=1e-12)
    np.testing.assert_allclose((dx * xhat).reshape(-1, C).sum(0),
                               dgamma / np.sqrt(var + 1e-5) * 1e-5 / (var + 1e-5), rtol=1e-6, atol=1e-13)
    np.testing.assert_allclose(grads["beta"][0], g.reshape(-1, C).sum(0), rtol=1e-12)


# ----------------------------------------------------------------------------------------------
# P4: softmax cross-entropy closed form
# ----------------------------------------------------------------------------------------------

@pytest.mark.parametrize("classes,lnC", [(10, 2.302585093), (100, 4.605170186), (200, 5.298317367)])
def test_p4_ce_uniform_logits(classes, lnC):
    net = mini_tiny()
    net.classes = classes
    x, _, p = S.make_all(net)
    p["head"] = {"w": np.zeros((classes, net.head_cin)), "b": np.zeros(classes)}
    o = ParaRealOracle(net, p)
    labels = np.arange(net.batch) % classes
    hd = o.head(o.forward(x)["ytilde"], labels)
    assert abs(hd["loss"] - lnC) < 1e-9
    assert abs(hd["db"].sum()) < 1e-15        # every dlogits row sums to 0
    np.testing.assert_array_equal(hd["D_N"], 0.0)


# ----------------------------------------------------------------------------------------------
# P5 / P7: special cases that reduce the parareal network to the original one
# ----------------------------------------------------------------------------------------------

def test_p5_single_subnetwork_is_original():
    net = mini_resnet(n_sub=1)
    x, labels, p = S.make_all(net)
    o = ParaRealOracle(net, p)
    fwd = o.forward(x)
    np.testing.assert_array_equal(fwd["ytilde"], o.sequential(x))
    assert fwd["r"] == [] and fwd["rt"] == []


@pytest.mark.parametrize("kind", ["resnet", "vgg", "tiny"])
def test_p7_exact_interfaces(kind):
    """x_{j+1} := y_j makes every r_j = 0; with F^j(0) = 0 then every rt_j = 0 and
    ytilde = g^N o ... o g^1 o C^1 (x)."""
    net = MINIS[kind]()
    x, labels, p = S.make_all(net)
    o = ParaRealOracle(net, p)
    fwd = o.forward(x, exact_interfaces=True)
    for r in fwd["r"] + fwd["rt"]:
        np.testing.assert_array_equal(r, 0.0)
    np.testing.assert_array_equal(fwd["ytilde"], o.sequential(x))


# ----------------------------------------------------------------------------------------------
# P6: Proposition (Consistency) -- linear f and F^j = g^{j+1} give f-bar = f
# ----------------------------------------------------------------------------------------------

def linear_net(N=4, hw=8, ch=4, B=2):
    shape = (hw, hw, ch)
    pre, fine, crs = [], [], []
    for j in range(N):
        b = _SegBuilder(shape)
        pre.append(b.done(0 if j == 0 else b.conv(0, ch, 1, 1, 0)))
        b = _SegBuilder(shape)
        z = b.conv(0, ch, 3, 1, 1)
        fine.append(b.done(b.conv(z, ch, 3, 1, 1, res=0)))
    for j in range(1, N):
        crs.append(copy.deepcopy(fine[j]))
    return Net("linear", "f32", B, shape, 5, pre, fine, crs, ch, (41, 42, 43))


@pytest.mark.parametrize("N", [2, 3, 4])
def test_p6_consistency_proposition(N):
    net = linear_net(N)
    x, labels, p = S.make_all(net)
    for j in range(N - 1):
        p["coarse"][j] = copy.deepcopy(p["fine"][j + 1])          # F^j := g^{j+1}
    o = ParaRealOracle(net, p)
    fwd, hd, bwd = o.step(x, labels)
    yseq, hseq, dseq = o.sequential(x, labels)
    scale = np.abs(yseq).max()
    np.testing.assert_allclose(fwd["ytilde"], yseq, atol=1e-12 * scale)
    assert abs(hd["loss"] - hseq["loss"]) < 1e-12
    # f-bar = f for all x, hence dL/dx agree; this exercises the -D_{j-1} term of eq. (deltaj)
    np.testing.assert_allclose(bwd["dimage"], dseq, atol=1e-12 * np.abs(dseq).max())
    # and the proposition fails as soon as F^j differs from g^{j+1}
    p2 = copy.deepcopy(p)
    p2["coarse"][0]["conv"][0] = p2["coarse"][0]["conv"][0] * 1.01
    y2 = ParaRealOracle(net, p2).forward(x)["ytilde"]
    assert np.abs(y2 - yseq).max() > 1e-6 * scale


# ----------------------------------------------------------------------------------------------
# P8 / P9: central finite differences on tiny nets, every parameter group and the interfaces
# ----------------------------------------------------------------------------------------------

def _loss(net, p, x, labels):
    o = ParaRealOracle(net, p)
    return o.head(o.forward(x)["ytilde"], labels)["loss"]


def _param_refs(net, p, bwd, hd):
    """(getter path, analytic gradient) for every parameter array of f-bar (eq. (barf))."""
    refs = []
    for part, grads in (("pre", bwd["ddelta"]), ("fine", bwd["dphi"]), ("coarse", bwd["deta"])):
        for j, gr in enumerate(grads):
            if gr is None:
                continue
            for i, g in enumerate(gr["conv"]):
                if g is not None:
                    refs.append(((part, j, "conv", i), g))
            for b in range(len(gr["gamma"])):
                refs.append(((part, j, "gamma", b), gr["gamma"][b]))
                refs.append(((part, j, "beta", b), gr["beta"][b]))
    refs.append((("head", "w"), hd["dw"]))
    refs.append((("head", "b"), hd["db"]))
    return refs


def _get(p, path):
    if path[0] == "head":
        return p["head"][path[1]]
    part, j, kind, i = path
    return p[part][j][kind][i]


@pytest.mark.parametrize("kind", ["resnet", "vgg", "tiny"])
def test_p8_finite_differences_all_parameter_groups(kind):
    net = MINIS[kind]()
    x, labels, p = S.make_all(net)
    # non-trivial BN affine parameters so that gamma / beta gradients are generic
    lr = np.random.default_rng(7)
    for part in ("pre", "fine", "coarse"):
        for sp in p[part]:
            sp["gamma"] = [1.0 + 0.3 * lr.standard_normal(g.shape) for g in sp["gamma"]]
            sp["beta"] = [0.2 * lr.standard_normal(b.shape) for b in sp["beta"]]
    o = ParaRealOracle(net, p)
    fwd, hd, bwd = o.step(x, labels)
    refs = _param_refs(net, p, bwd, hd)
    groups = {r[0][0] for r in refs}
    assert groups == {"pre", "fine", "coarse", "head"} or (kind == "tiny" and "pre" in groups)
    pick = np.random.default_rng(99)
    checked = 0
    worst = 0.0
    for path, g in refs:
        arr = _get(p, path)
        for _ in range(2):
            idx = tuple(pick.integers(0, s) for s in arr.shape)
            old = arr[idx]
            h = 1e-6 * max(1.0, abs(old))
            arr[idx] = old + h
            lp = _loss(net, p, x, labels)
            arr[idx] = old - h
            lm = _loss(net, p, x, labels)
            arr[idx] = old
            fd = (lp - lm) / (2 * h)
            err = abs(fd - g[idx]) / max(abs(g[idx]), 1e-4)
            worst = max(worst, err)
            checked += 1
    assert checked >= 20
    assert worst < 1e-5, worst


@pytest.mark.parametrize("kind", ["resnet", "vgg"])
def test_p9_interface_gradients_are_D(kind):
    """dL/dy_j = D_j for every j (eq. (ingredient1), Alg. para3), by finite differences on y_j."""
    net = MINIS[kind]()
    x, labels, p = S.make_all(net)
    o = ParaRealOracle(net, p)
    fwd, hd, bwd = o.step(x, labels)
    N = net.n_sub

    def loss_from(ys):
        r = [ys[j] - fwd["x"][j + 1] for j in range(N - 1)]
        rt = r[0]
        for j in range(N - 1):
            ext = r[j + 1] if j + 1 < N - 1 else ys[N - 1]
            rt, _ = seg_forward(net.coarse[j], p["coarse"][j], rt, lambda a: a, ext=ext)
        return o.head(rt, labels)["loss"]

    pick = np.random.default_rng(5)
    for j in range(N):
        for _ in range(3):
            ys = [y.copy() for y in fwd["y"]]
            idx = tuple(pick.integers(0, s) for s in ys[j].shape)
            h = 1e-6
            ys[j][idx] += h
            lp = loss_from(ys)
            ys[j][idx] -= 2 * h
            lm = loss_from(ys)
            fd = (lp - lm) / (2 * h)
            d = bwd["D"][j][idx]
            assert abs(fd - d) <= 1e-6 * abs(d) + 5e-9, (j, fd, d)   # FD rounding ~ 1e-16 * L / h


# ----------------------------------------------------------------------------------------------
# P10 / P11: the paper's parameter counts and receptive field pin the network descriptions
# ----------------------------------------------------------------------------------------------

def _gold():
    with open(os.path.join(GOLD, "param_counts.json")) as f:
        return json.load(f)


def _close(count, printed_M):
    """The paper prints parameter counts in millions with one decimal (rounded or truncated):
    accept a count within 0.06 M of the printed value."""
    return abs(count / 1e6 - printed_M) <= 0.06


def test_p10_resnet_parameter_counts():
    g = _gold()
    net1 = resnet_parareal("p", 1, 32, 1, 100, "f32", (1, 2, 3))
    pc = param_count(net1)
    assert _close(pc["pre"][0] + sum(pc["fine"]) + pc["head"], g["resnet1001_total_M"]["value"])
    body = sum(pc["fine"])
    for N in (3, 6, 12, 18):
        net = resnet_parareal("p", 1, 32, N, 100, "f32", (1, 2, 3), coarse="paper", partition="per_stage")
        pcn = param_count(net, bn=False)
        pcf = param_count(net)
        assert _close(sum(pcn["coarse"]), g["parareal_resnet_coarse_M"]["value"][str(N)]), N
        assert sum(pcf["fine"]) == body
        assert _close(body / N, g["parareal_resnet_subnet_M"]["value"][str(N)]), N
        total = sum(pcf["pre"]) + sum(pcf["fine"]) + sum(pcf["coarse"]) + pcf["head"]
        if str(N) in g["parareal_resnet_total_M"]["value"]:
            assert _close(total, g["parareal_resnet_total_M"]["value"][str(N)]), N


def test_p10_vgg_parameter_counts():
    g = _gold()
    net = vgg_parareal("v", 1, 224, 1000, "f32", (1, 2, 3), coarse="paper")
    pcn = param_count(net, bn=False)
    assert _close(sum(pcn["coarse"]), g["parareal_vgg16_4_coarse_M"]["value"])
    assert _close(sum(pcn["fine"]) / 4, g["parareal_vgg16_4_subnet_M"]["value"])
    # the split of Sec. 4.1.1: X_j of 56/28/14/7 pixels with 128/256/512/512 channels
    assert [S.segment_shapes(f)[f.out] for f in net.fine] == [(56, 56, 128), (28, 28, 256),
                                                              (14, 14, 512), (7, 7, 512)]


def test_p11_coarse_receptive_field():
    g = _gold()
    net = resnet_parareal("p", 1, 32, 3, 100, "f32", (1, 2, 3), coarse="paper", partition="per_stage")
    assert receptive_field(net.coarse[0]) == g["coarse_ru4_receptive_field"]["value"]


def test_config_partitions():
    """Contiguous chunks of ceil(333/N) units for the N = 4, 16, 8 workloads."""
    shapes = lambda net: [S.segment_shapes(f)[f.out] for f in net.fine]
    assert shapes(S.config(2, 1)) == [(32, 32, 64), (16, 16, 128), (8, 8, 256), (8, 8, 256)]
    n4 = S.config(3, 1)
    assert shapes(n4) == [(32, 32, 64)] * 5 + [(16, 16, 128)] * 5 + [(8, 8, 256)] * 6
    assert [sum(1 for n in f.nodes if n.op == "conv" and n.res >= 0) for f in n4.fine] == [21] * 15 + [18]
    n5 = S.config(4, 1)
    assert shapes(n5) == [(64, 64, 64)] * 2 + [(32, 32, 128)] * 3 + [(16, 16, 256)] * 3


# ----------------------------------------------------------------------------------------------
# P12: whole-network library cross-check (PyTorch CPU float64 autograd)
# ----------------------------------------------------------------------------------------------

@pytest.mark.parametrize("kind", ["resnet", "vgg", "tiny"])
def test_p12_torch_autograd_cross_check(kind):
    torch = pytest.importorskip("torch")
    from tests.torch_ref import TorchParaReal
    net = MINIS[kind]()
    x, labels, p = S.make_all(net)
    o = ParaRealOracle(net, p)
    fwd, hd, bwd = o.step(x, labels)
    tr = TorchParaReal(net, p)
    loss, logits = tr.loss(x, labels)
    loss.backward()
    assert abs(loss.item() - hd["loss"]) < 1e-12
    np.testing.assert_allclose(logits.detach().numpy(), hd["logits"], rtol=1e-11, atol=1e-12)
    n = 0
    for path, g in _param_refs(net, p, bwd, hd):
        if path[0] == "head":
            t = tr.hw if path[1] == "w" else tr.hb
        else:
            part, j, kind_, i = path
            t = tr.leaves[((part, j), kind_, i)]
        tg = t.grad.numpy()
        if path[0] != "head" and path[2] == "conv":
            tg = np.transpose(tg, (0, 2, 3, 1))
        np.testing.assert_allclose(g, tg, rtol=1e-9, atol=1e-12 * max(1.0, np.abs(tg).max()),
                                   err_msg=str(path))
        n += 1
    assert n > 10


# ----------------------------------------------------------------------------------------------
# storage model: bfloat16 rounding
# ----------------------------------------------------------------------------------------------

def test_bf16_rounding_matches_library():
    torch = pytest.importorskip("torch")
    v = np.concatenate([rng.standard_normal(20000).astype(np.float32),
                        np.float32([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 2 ** -120 * 1.5])])
    ref = torch.tensor(v).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(P.round_bf16(v.astype(np.float64)), ref)
    np.testing.assert_array_equal(S.gen.round_to_bf16(v.astype(np.float64)), ref)


def test_bf16_storage_model():
    """The bf16 storage model is the fp64 network with rounding at the storage points.

    (a) every tensor it stores is exactly bf16-representable;
    (b) its forward output stays within 2e-2 (normwise) of plain fp64;
    (c) its gradients do NOT: moving activations by bf16 storage flips ReLU masks, and the
        gradients of a deep BN/ReLU network move by far more than 2e-2.  Rounding only the
        backward quantities moves them by < 2e-2.  This is why GPU gradients are compared with
        the oracle evaluated under the same storage model."""
    net = mini_resnet(batch=8)
    x, labels, p = S.make_all(net)
    x = S.gen.round_to_bf16(x)
    f64 = ParaRealOracle(net, p, bf16=False)
    b16 = ParaRealOracle(net, p, bf16=True)
    fa, ha, ba = f64.step(x, labels)
    fb, hb, bb = b16.step(x, labels)
    for run in fb["fine_run"] + fb["coarse_run"]:
        for k, v in run.slots.items():
            if k != 0:
                np.testing.assert_array_equal(P.round_bf16(v), v)
    for v in fb["r"] + bb["dx"] + bb["D"]:
        np.testing.assert_array_equal(P.round_bf16(v), v)
    rel = lambda a, b: np.linalg.norm(a - b) / np.linalg.norm(a)
    assert rel(fa["ytilde"], fb["ytilde"]) < 2e-2
    assert max(rel(a, b) for a, b in zip(ba["dx"], bb["dx"])) > 2e-2
    bc = b16.backward(fa, f64.head(fa["ytilde"], labels))     # exact forward, rounded backward
    assert max(rel(a, b) for a, b in zip(ba["dx"], bc["dx"])) < 2e-2


# ------------------------------------------------------------------------------------------------
# parameter update (Sec. 4 training setup): SGD with momentum and weight decay
# ------------------------------------------------------------------------------------------------

def test_sgd_plain_descent_on_a_quadratic():
    """mu = 0 on f(w) = a w^2 / 2 with decay wd: w_k = (1 - lr (a + wd))^k w_0 (closed form)."""
    from oracle.sgd import sgd_step
    a, lr, wd = 3.0, 0.05, 1e-2
    w0 = np.array([1.5, -2.0, 0.25])
    w, v = w0.copy(), np.zeros(3)
    for k in range(1, 8):
        w, v = sgd_step(w, a * w, v, lr, 0.0, wd, nesterov=True)
        assert np.allclose(w, (1 - lr * (a + wd)) ** k * w0, rtol=1e-14, atol=0)


@pytest.mark.parametrize("nesterov", [True, False])
def test_sgd_momentum_decay_without_gradient(nesterov):
    """Zero gradient and decay: v_k = mu^k v_0 and w_k = w_0 - lr c mu (1 - mu^k) / (1 - mu) v_0 with
    c = mu (Nesterov's look-ahead) or 1 (closed form of the geometric series)."""
    from oracle.sgd import sgd_step
    lr, mu = 0.1, 0.9
    v0 = np.array([0.5, -1.0])
    w0 = np.array([2.0, 3.0])
    w, v = w0.copy(), v0.copy()
    c = mu if nesterov else 1.0
    for k in range(1, 10):
        w, v = sgd_step(w, np.zeros(2), v, lr, mu, 0.0, nesterov)
        assert np.allclose(v, mu ** k * v0, rtol=1e-14)
        assert np.allclose(w, w0 - lr * c * mu * (1 - mu ** k) / (1 - mu) * v0, rtol=1e-13)


@pytest.mark.parametrize("nesterov", [True, False])
def test_sgd_matches_torch_optim(nesterov):
    """The same steps as torch.optim.SGD (momentum 0.9, weight decay, float64), an implementation
    written independently of this one."""
    import torch
    from oracle.sgd import sgd_step
    rng = np.random.default_rng(5)
    w0 = rng.standard_normal((7, 5))
    p = torch.nn.Parameter(torch.from_numpy(w0.copy()))
    opt = torch.optim.SGD([p], lr=0.03, momentum=0.9, weight_decay=5e-4, nesterov=nesterov)
    w, v = w0.copy(), np.zeros_like(w0)
    for _ in range(6):
        g = rng.standard_normal(w0.shape)
        p.grad = torch.from_numpy(g.copy())
        opt.step()
        w, v = sgd_step(w, g, v, 0.03, 0.9, 5e-4, nesterov)
        assert np.allclose(p.detach().numpy(), w, rtol=1e-13, atol=1e-15)


# ------------------------------------------------------------------------------------------------
# cost-balanced decomposition (Remark after Table grad): contiguous, min-max cost
# ------------------------------------------------------------------------------------------------

def _all_splits(n, k):
    """Every split of range(n) into k non-empty contiguous parts (brute force)."""
    import itertools
    for cuts in itertools.combinations(range(1, n), k - 1):
        b = (0,) + cuts + (n,)
        yield [(b[i], b[i + 1]) for i in range(k)]


@pytest.mark.parametrize("seed", range(6))
def test_balanced_partition_is_the_brute_force_optimum(seed):
    from pnn_synth.nets import partition_balanced
    rng = np.random.default_rng(seed)
    n, k = int(rng.integers(4, 11)), int(rng.integers(1, 5))
    costs = rng.uniform(0.1, 3.0, n)
    b = partition_balanced(costs, k)
    assert b[0][0] == 0 and b[-1][1] == n and all(e > s for s, e in b)
    assert all(b[i][1] == b[i + 1][0] for i in range(k - 1))
    got = max(costs[s:e].sum() for s, e in b)
    best = min(max(costs[s:e].sum() for s, e in sp) for sp in _all_splits(n, k))
    assert np.isclose(got, best, rtol=1e-12)


def test_balanced_partition_special_cases():
    """Equal costs give sizes differing by at most one; one sub-network takes everything; as many
    sub-networks as units gives one unit each; ResNet-1001's bottlenecks have (near) equal FLOPs, so
    the FLOP-balanced split of 333 units into 16 is 20-21 units each."""
    from pnn_synth.nets import partition_balanced, resnet_units, unit_cost
    for n, k in ((12, 4), (13, 4), (333, 16)):
        sizes = [e - s for s, e in partition_balanced(np.ones(n), k)]
        assert max(sizes) - min(sizes) <= 1 and sum(sizes) == n
    assert partition_balanced(np.ones(5), 1) == [(0, 5)]
    assert partition_balanced(np.arange(1.0, 6.0), 5) == [(i, i + 1) for i in range(5)]
    sizes = [e - s for s, e in partition_balanced([unit_cost(u, "flops") for u in resnet_units(32)], 16)]
    assert set(sizes) <= {20, 21, 22}
