"""GPU parity, end to end: one full training step (Alg. para2 + Alg. para3) through the C ABI against
the fp64 CPU oracle on the same seeded inputs.

Metric per checked tensor T (loss, logits, every x_j, y_j, r_j, ytilde, every D_j, dL/dx_j, every
parameter gradient of C^j, g^j, F^j and of the head):
  fp32 storage:  e_inf(T) = max|T_gpu - T_ref| / max|T_ref|  <= 1e-4
  bf16 storage:  e_2(T)   = ||T_gpu - T_ref||_2 / ||T_ref||_2, against the oracle evaluated with the
                 same bf16 storage points (its ``bf16=True`` mode).

End-to-end agreement is bounded by the network's own conditioning: the gradients of deep BN/ReLU
networks at initialisation move far more than the rounding that perturbs them (ReLU masks and
max-pool choices flip).  These tests therefore run every network form (tiny basic blocks, VGG,
pre-activation bottleneck ResNets with strided / projected units and sub-networks straddling
stages) at depths where fp32 agreement is exact to 1e-4; the full-depth workloads are checked node
by node, teacher-forced, in test_gpu_nodes.py.  Odd batches give ragged row tiles.
"""
import numpy as np
import pytest

import pnn_synth as S
from pnn_synth.nets import resnet_parareal, vgg_parareal

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def rel_inf(a, ref):
    return float(np.abs(a - ref).max() / max(np.abs(ref).max(), 1e-30))


def rel_2(a, ref):
    return float(np.linalg.norm((a - ref).ravel()) / max(np.linalg.norm(ref.ravel()), 1e-30))


def compare_step(g, net, fwd, hd, bwd, metric=None):
    """{tensor name: error} for every checked tensor of one step."""
    to = g.to_np
    err = {}
    m = metric or (rel_inf if net.dtype == "f32" else rel_2)
    N = net.n_sub
    err["loss"] = abs(float(g.loss.item()) - hd["loss"]) / abs(hd["loss"])
    err["logits"] = m(to(g.logits), hd["logits"])
    err["ytilde"] = m(to(g.ytilde), fwd["ytilde"])
    for j in range(N):
        err[f"y{j}"] = m(to(g.y[j]), fwd["y"][j])
        err[f"x{j}"] = m(to(g.x[j]), fwd["x"][j])
        err[f"D{j}"] = m(to(g.D[j]), bwd["D"][j])
        err[f"dx{j}"] = m(to(g.dx[j]), bwd["dx"][j])
    for j in range(N - 1):
        err[f"r{j}"] = m(to(g.r[j]), fwd["r"][j])
    for j in range(1, N - 1):
        err[f"rt{j}"] = m(to(g.rt[j]), fwd["rt"][j])
    dW = to(g.deps)
    K, C = hd["dw"].shape
    err["head.dw"] = m(dW[:K * C].reshape(K, C), hd["dw"])
    err["head.db"] = m(dW[K * C:], hd["db"])
    for part, name, ref in ((0, "pre", bwd["ddelta"]), (1, "fine", bwd["dphi"]), (2, "coarse", bwd["deta"])):
        for j, r in enumerate(ref):
            if r is None:
                continue
            got = g.unpack_grads(part, j)
            for key in ("conv", "gamma", "beta"):
                for i, (a, b) in enumerate(zip(got[key], r[key])):
                    if b is None:
                        continue
                    err[f"{name}{j}.{key}{i}"] = m(a, b)
    return err


def run_net(net, bf16_oracle=None):
    import torch
    from oracle.net import ParaRealOracle
    from paper_2103_08802_amd.step import ParaRealGPU
    _say(f"[parity] {net.name} dtype {net.dtype} batch {net.batch} N {net.n_sub}: GPU step")
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    g.load_input(x, labels)
    g.step()
    torch.cuda.synchronize()
    _say(f"[parity] {net.name}: oracle step")
    fwd, hd, bwd = ParaRealOracle(net, params, bf16=bf16_oracle).step(x, labels)
    err = compare_step(g, net, fwd, hd, bwd)
    worst = max(err, key=err.get)
    _say(f"[parity] {net.name}: {len(err)} tensors, worst {worst} = {err[worst]:.3e}")
    return err


def _assert_tol(err, tol):
    bad = {k: v for k, v in err.items() if not v <= tol}
    assert not bad, sorted(bad.items(), key=lambda kv: -kv[1])[:10]


def mini_resnet(n_sub, ups, batch, dtype="f32", hw=16, coarse="config", partition="contiguous"):
    return resnet_parareal(f"mini-resnet-u{ups}-n{n_sub}", batch, hw, n_sub, 10, dtype, (7, 8, 9),
                           units_per_stage=ups, widths=(64, 128, 256), stem=16, coarse=coarse,
                           partition=partition)


@pytest.mark.parametrize("bn_init", ["unit", "random"])
def test_tiny_workload_fp32(bn_init):
    """The tiny workload itself (N = 2 basic blocks, batch 4, fp32): every tensor to 1e-4; also with
    seeded non-trivial BN gamma / beta and head bias (the affine paths of the BN forward, the BN
    backward coefficients and the ReLU mask of the data-gradient epilogue)."""
    net = S.config(0)
    net.bn_init = bn_init
    _assert_tol(run_net(net), 1e-4)


@pytest.mark.parametrize("n_sub,ups,batch", [(1, 2, 2), (2, 2, 3), (3, 2, 2), (4, 4, 3), (5, 3, 2)])
def test_resnet_forms_fp32(n_sub, ups, batch):
    """Bottleneck ResNets with strided projected units, N not a multiple of 3 (sub-networks
    straddle stages), ragged tiles: every tensor to 1e-4."""
    _assert_tol(run_net(mini_resnet(n_sub, ups, batch)), 1e-4)


def test_resnet_forms_fp32_random_bn():
    """A bottleneck ResNet (N = 4, strided projected units, straddling sub-networks) with seeded
    non-trivial BN gamma / beta: every tensor to 1e-4."""
    net = mini_resnet(4, 4, 3)
    net.bn_init = "random"
    _assert_tol(run_net(net), 1e-4)


@pytest.mark.parametrize("n_sub,ups,batch", [(2, 2, 3), (3, 2, 2), (4, 4, 2)])
def test_resnet_paper_coarse_fp32(n_sub, ups, batch):
    """The paper's own coarse network (ceil(12/N) two-3x3 residual units per F^j, the first strided
    with a projection at stage changes, Sec. 4.2.1): every tensor to 1e-4."""
    _assert_tol(run_net(mini_resnet(n_sub, ups, batch, coarse="paper")), 1e-4)


@pytest.mark.parametrize("partition", ["balanced", "balanced_flops"])
def test_resnet_balanced_partition_fp32(partition):
    """Sub-networks of unequal unit counts from the cost-balanced decomposition: every tensor to
    1e-4."""
    _assert_tol(run_net(mini_resnet(4, 4, 2, partition=partition)), 1e-4)


def test_vgg_paper_coarse_fp32():
    """The VGG-16 workload with the paper's coarse blocks (two 3x3 convolutions and a max pool,
    Sec. 4.1.1) in fp32 at batch 3: every tensor to 1e-4."""
    net = S.config(1, 3, coarse="paper")
    net.dtype = "f32"
    _assert_tol(run_net(net), 1e-4)


def test_vgg_workload_structure_fp32():
    """The VGG-16 workload's network (all 13 convolutions, 2x2 pools, N = 4) in fp32 at batch 3.
    (With seeded non-trivial BN gamma / beta the same network has a 2x2 pool window in g^2 whose two
    largest activations differ by 7.7e-6 relative, within reach of fp32 rounding, so the pool's
    gradient routing can flip end to end; that form is checked node by node, teacher-forced, in
    test_gpu_nodes.py::test_random_bn_nodes.)"""
    net = S.config(1, 3)
    net.dtype = "f32"
    _assert_tol(run_net(net), 1e-4)


def test_vgg_workload_bf16_forward():
    """The VGG-16 workload in bf16 at batch 32: forward tensors (x_j, y_j, r_j, rt_j, ytilde,
    logits, loss) within 2e-2 of the bf16-storage oracle."""
    err = run_net(S.config(1, 32))
    fw = {k: v for k, v in err.items() if k[0] in "xyrl" or k == "ytilde"}
    _assert_tol(fw, 2e-2)


def test_coarse_bwd_all_equals_per_block_calls():
    """coarse_bwd_all (coarse weight gradients deferred into grouped launches) gives bit-identical
    D_j and deta_j to the N - 1 coarse_bwd calls."""
    import torch
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(2, 2)
    x, labels, params = S.make_all(net)
    out = []
    for chain_all in (False, True):
        g = ParaRealGPU(net, params)
        g.coarse_chain_all = chain_all
        g.load_input(x, labels)
        g.forward()
        g.backward_coarse_fine()
        torch.cuda.synchronize()
        out.append(([t.clone() for t in g.D], [t.clone() for t in g.deta]))
    for a, b in zip(out[0][0] + out[0][1], out[1][0] + out[1][1]):
        assert torch.equal(a, b)


@pytest.mark.gpu
@pytest.mark.parametrize("idx,batch", [(1, 2), (2, 2), (3, 4)])
def test_streams_do_not_change_results(idx, batch):
    """Running the fine sub-network groups on separate streams gives bit-identical loss, logits and
    parameter gradients to running every launch on the call's stream (also on a second step,
    which reuses the plan's streams and events)."""
    import torch
    from paper_2103_08802_amd import binding as B
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    out = []
    for streams in (1, 4):
        g = ParaRealGPU(net, params)
        B.pnn_set_streams(g.plan, streams)
        g.load_input(x, labels)
        res = []
        for _ in range(2):
            g.forward()
            g.backward()
            torch.cuda.synchronize()
            res += [t.clone() for t in [g.loss, g.logits, g.deps] + g.ddelta + g.dphi + g.deta]
        out.append(res)
    for a, b in zip(out[0], out[1]):
        assert torch.equal(a, b)


@pytest.mark.gpu
@pytest.mark.parametrize("idx,batch,streams,whole", [(2, 2, 4, False), (3, 4, 4, False), (3, 4, 1, False),
                                                     (2, 2, 4, True), (3, 4, 4, True)])
def test_graph_replay_matches_eager(idx, batch, streams, whole):
    """The step captured into HIP graphs (one per part, or with ``whole`` the forward and the
    overlapped backward as one graph each, its fork and join across the side streams captured
    with it; captured before any eager call) and replayed gives bit-identical loss, logits,
    parameter gradients and input gradients to the eager step, on every replay, with eager steps,
    output clearing and synchronisations in between."""
    import torch
    from paper_2103_08802_amd import binding as B
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    B.pnn_set_streams(g.plan, streams)
    g.load_input(x, labels)
    g.overlap_bwd = whole                # the eager reference runs the backward the graphs hold

    def outputs():
        return [t.clone() for t in [g.loss, g.logits, g.deps] + g.ddelta + g.dphi + g.deta + g.dx]

    g.capture(whole=whole)               # before any eager step: the library creates nothing in a call
    torch.cuda.synchronize()
    g.replay_forward()
    g.replay_backward()
    torch.cuda.synchronize()
    first = outputs()
    g.forward()
    g.backward()
    torch.cuda.synchronize()
    ref = outputs()
    for a, b in zip(first, ref):
        assert torch.equal(a, b)
    for _ in range(3):
        for t in [g.loss, g.logits, g.deps] + g.ddelta + g.dphi + g.deta + g.dx:
            t.zero_()                    # eager work between replays; the replay rewrites them
        torch.cuda.synchronize()
        g.replay_forward()
        g.replay_backward()
        torch.cuda.synchronize()
        for a, b in zip(outputs(), ref):
            assert torch.equal(a, b)
        g.forward()
        g.backward()
        torch.cuda.synchronize()
        for a, b in zip(outputs(), ref):
            assert torch.equal(a, b)


@pytest.mark.gpu
@pytest.mark.parametrize("idx,batch,streams", [(1, 2, 4), (2, 2, 4), (3, 4, 4), (3, 4, 1)])
def test_parareal_bwd_equals_separate_calls(idx, batch, streams):
    """parareal_bwd (coarse chain overlapped with the fine backward) gives bit-identical D_j,
    coarse and fine parameter gradients and input gradients to coarse_bwd_all followed by
    parareal_fine_bwd."""
    import torch
    from paper_2103_08802_amd import binding as B
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    out = []
    for overlap in (False, True, True):
        g = ParaRealGPU(net, params)
        B.pnn_set_streams(g.plan, streams)
        g.overlap_bwd = overlap
        g.load_input(x, labels)
        g.forward()
        g.backward()
        torch.cuda.synchronize()
        out.append([t.clone() for t in [g.loss, g.deps] + g.D + g.deta + g.dphi + g.ddelta + g.dx])
    for run in out[1:]:
        for a, b in zip(out[0], run):
            assert torch.equal(a, b)


@pytest.mark.gpu
def test_bench_configuration_full_size():
    """The launch configuration bench.py times (4 streams, coarse chain overlapped with the fine
    backward) at the full ResNet-1001 N=16 batch-128 workload gives bit-identical loss, logits and
    every parameter and input gradient to one stream with the separate calls (the path the
    node-level parity checks run at full size)."""
    import torch
    from paper_2103_08802_amd import binding as B
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(3)
    x, labels, params = S.make_all(net)
    out = []
    for streams, overlap in ((1, False), (4, True)):
        g = ParaRealGPU(net, params)
        B.pnn_set_streams(g.plan, streams)
        g.overlap_bwd = overlap
        g.load_input(x, labels)
        g.forward()
        g.backward()
        torch.cuda.synchronize()
        out.append([t.clone() for t in [g.loss, g.logits, g.deps] + g.ddelta + g.dphi + g.deta + g.dx])
        del g
        torch.cuda.empty_cache()
    assert torch.isfinite(out[0][0]).all()
    for a, b in zip(out[0], out[1]):
        assert torch.equal(a, b)


@pytest.mark.gpu
@pytest.mark.parametrize("idx,batch", [(0, 4), (1, 2), (3, 4)])
def test_combine_fwd_and_rnorm2(idx, batch):
    """parareal_combine_fwd: r_j = y_j - x_{j+1} rounded to storage, bit for bit (eq. (rk)), and the
    optional ||r_j||^2 equals the sum of squares of the stored r_j; whole and ragged tiles (the VGG
    workload at batch 2 has a 4096-element interface)."""
    import torch
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    g.load_input(x, labels)
    g.forward(rnorm=True)
    torch.cuda.synchronize()
    for j in range(net.n_sub - 1):
        ref = (g.y[j].float() - g.x[j + 1].float()).to(g.r[j].dtype)
        assert torch.equal(g.r[j], ref)
        ss = float((g.r[j].double() ** 2).sum())
        assert abs(float(g.rnorm2[j]) - ss) <= 1e-5 * max(ss, 1e-30)


@pytest.mark.parametrize("idx, batch", [(0, 4), (3, 3)])
def test_head_repeatable_and_label_range(idx, batch):
    """pnn_head_fwd_bwd: a second call on the same inputs gives the same bits (every sum of the head
    runs in a fixed order), and a label outside [0, classes) makes the loss NaN while the other
    samples' logits are unchanged."""
    import torch
    from paper_2103_08802_amd import binding as B
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    g.load_input(x, labels)
    g.forward()
    torch.cuda.synchronize()
    N = net.n_sub
    first = [t.clone() for t in (g.loss, g.logits, g.D[N - 1], g.deps)]
    B.pnn_head_fwd_bwd(g.plan, g.ytilde, g.eps, g.labels, g.logits, g.loss, g.D[N - 1], g.deps,
                       g.scratch, None)
    torch.cuda.synchronize()
    for a, b in zip(first, (g.loss, g.logits, g.D[N - 1], g.deps)):
        assert torch.equal(a, b)
    assert torch.isfinite(g.loss).all()
    bad = g.labels.clone()
    bad[0] = net.classes
    B.pnn_head_fwd_bwd(g.plan, g.ytilde, g.eps, bad, g.logits, g.loss, g.D[N - 1], g.deps,
                       g.scratch, None)
    torch.cuda.synchronize()
    assert torch.isnan(g.loss).all()
    assert torch.equal(g.logits, first[1])


@pytest.mark.gpu
@pytest.mark.parametrize("idx,batch", [(0, 4), (3, 2)])
def test_nonfinite_flags(idx, batch):
    """The non-finite flags: clear after a clean step; the combine raises flag 0 when an r_j element
    is not finite (only when given a scratch), the head raises flag 1 when the loss is not finite;
    pnn_flags_clear resets both."""
    import torch
    from paper_2103_08802_amd import binding as B
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    g = ParaRealGPU(net, params)
    g.load_input(x, labels)
    off = g.plan.inspect(0, 0, 5, 0)

    def flags():
        torch.cuda.synchronize()
        return g.scratch[off:off + 8].view(torch.int32).cpu().tolist()

    B.pnn_flags_clear(g.plan, g.scratch, None)
    g.forward()
    assert flags() == [0, 0]
    N = net.n_sub
    y = g.y[N - 2].clone()
    g.y[N - 2].view(-1)[7] = float("nan")
    B.parareal_combine_fwd(g.plan, g.y, g.x, g.r, None, None, None)            # no scratch: no flag
    assert flags() == [0, 0]
    B.parareal_combine_fwd(g.plan, g.y, g.x, g.r, None, g.scratch, None)
    assert flags() == [1, 0]
    B.pnn_flags_clear(g.plan, g.scratch, None)
    assert flags() == [0, 0]
    g.y[N - 2].copy_(y)
    g.ytilde.view(-1)[3] = float("inf")
    B.pnn_head_fwd_bwd(g.plan, g.ytilde, g.eps, g.labels, g.logits, g.loss, g.D[N - 1], g.deps,
                       g.scratch, None)
    assert flags() == [0, 1]
    assert not torch.isfinite(g.loss).all()


def pooled_16ch_net(dtype, batch):
    """Two sub-networks on a 16-channel 32x32 input, g^1 ending at 16x16: C^2 max-pools the
    16-channel input (whole 16-byte channel chunks per thread) before its 1x1 convolution."""
    from pnn_synth.nets import Net, _SegBuilder, _pre_pool_conv
    ch = 16
    img, half = (32, 32, ch), (16, 16, ch)
    pre0 = _SegBuilder(img).done(0)
    pre1 = _pre_pool_conv(img, half)
    b = _SegBuilder(img)
    z = b.conv(0, ch, 3, 2, 1, preact=True)
    fine0 = b.done(b.conv(z, ch, 3, 1, 1, preact=True))
    b = _SegBuilder(half)
    z = b.conv(0, ch, 3, 1, 1, preact=True)
    fine1 = b.done(b.conv(z, ch, 3, 1, 1, preact=True, res=0))
    b = _SegBuilder(half)
    coarse = [b.done(b.conv(0, ch, 3, 1, 1))]
    return Net(f"pool16-{dtype}-b{batch}", dtype, batch, img, 10, [pre0, pre1], [fine0, fine1],
               coarse, ch, (21, 22, 23))


@pytest.mark.parametrize("dtype,batch,tol", [("f32", 3, 1e-4), ("bf16", 4, 2e-2)])
def test_pooled_multichannel_input(dtype, batch, tol):
    """C^j max-pooling a multi-channel input (the vectorised pool path; the workloads pool only the
    3-channel image): every tensor within the fp32 / bf16 tolerance of the oracle."""
    _assert_tol(run_net(pooled_16ch_net(dtype, batch)), tol)


@pytest.mark.parametrize("n_sub,ups,batch", [(3, 2, 2), (4, 4, 3)])
def test_coarse_fwd_all_equals_per_block_calls(n_sub, ups, batch):
    """coarse_fwd_all (each block's input BN sums formed by the previous block's last convolution)
    against the N - 1 coarse_fwd calls, fp32: rt_j and ytilde agree to 1e-5 (the BN sums are the
    same numbers summed in another order)."""
    import torch
    from paper_2103_08802_amd.step import ParaRealGPU
    net = mini_resnet(n_sub, ups, batch)
    x, labels, params = S.make_all(net)
    out = []
    for chain in (False, True):
        g = ParaRealGPU(net, params)
        g.coarse_fwd_chain = chain
        g.load_input(x, labels)
        g.forward()
        torch.cuda.synchronize()
        out.append([g.to_np(t) for t in g.rt[1:] + [g.ytilde]])
    for a, b in zip(*out):
        assert rel_inf(b, a) <= 1e-5


def test_coarse_fwd_all_bf16_full_size():
    """The full-size bf16 workload: ytilde from coarse_fwd_all against the per-block calls.  The BN
    sums differ only in summation order, but the values they move across a bf16 rounding boundary
    change by one ulp (2^-8 relative) and feed the next block, 15 times: the two agree to about one
    bf16 ulp in L2 (measured 4.0e-3), bounded here by 1e-2, half the oracle tolerance that each of
    them meets block by block (test_gpu_nodes)."""
    import torch
    from paper_2103_08802_amd.step import ParaRealGPU
    net = S.config(3)
    x, labels, params = S.make_all(net)
    out = []
    for chain in (False, True):
        g = ParaRealGPU(net, params)
        g.coarse_fwd_chain = chain
        g.load_input(x, labels)
        g.forward()
        torch.cuda.synchronize()
        out.append(g.to_np(g.ytilde))
        del g
    err = rel_2(out[1], out[0])
    _say(f"[coarse_fwd_all] bf16 full size: ytilde L2 relative difference {err:.3e}")
    assert err <= 1e-2
