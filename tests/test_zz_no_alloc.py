"""The allocation-free head entry point (pnn_head_fwd_bwd_noalloc, its temporaries in the library's
fixed device array) against pnn_head_fwd_bwd with a scratch workspace: bit-identical logits, loss,
D_N and head gradients, on two calls in a row, the second on a smaller problem (the array keeps the
first call's values); and a problem beyond the array's size is rejected before anything runs."""
import ctypes

import numpy as np
import pytest

import pnn_synth as S

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def _head_case(idx, batch, seed):
    """Plan, ytilde-shaped input and head parameters / labels of a workload at ``batch``."""
    import torch
    from paper_2103_08802_amd import binding as B
    net = S.config(idx, batch)
    p = B.Plan(net)
    h, w, c = p.tensor_shape(1, net.n_sub - 1)
    K = net.classes
    rng = np.random.default_rng(seed)
    dt = torch.bfloat16 if net.dtype == "bf16" else torch.float32
    dev = torch.device("cuda")
    yt = torch.from_numpy(rng.standard_normal((batch, h, w, c)).astype(np.float32)).to(dev).to(dt)
    eps = torch.from_numpy((0.1 * rng.standard_normal(K * c + K)).astype(np.float32)).to(dev)
    labels = torch.from_numpy(rng.integers(0, K, batch).astype(np.int32)).to(dev)
    return net, p, yt, eps, labels


def _run(p, net, yt, eps, labels, noalloc):
    import torch
    from paper_2103_08802_amd import binding as B
    K = net.classes
    dev = yt.device
    logits = torch.zeros((net.batch, K), dtype=torch.float32, device=dev)
    loss = torch.zeros(1, dtype=torch.float32, device=dev)
    D_N = torch.zeros_like(yt)
    deps = torch.zeros_like(eps)
    s = torch.cuda.current_stream().cuda_stream
    if noalloc:
        B.pnn_head_fwd_bwd_noalloc(p, yt, eps, labels, logits, loss, D_N, deps, s)
    else:
        scratch = torch.zeros(p.workspace_size(B.PNN_WS_SCRATCH), dtype=torch.uint8, device=dev)
        B.pnn_head_fwd_bwd(p, yt, eps, labels, logits, loss, D_N, deps, scratch, s)
    torch.cuda.synchronize()
    return [logits, loss, D_N, deps]


def test_noalloc_head_matches_workspace_head():
    import torch
    cases = [(3, 32, 1), (3, 5, 2)]            # ResNet-1001 N=16 head at batch 32, then batch 5
    prepared = [_head_case(*c) for c in cases]
    for (idx, batch, _), (net, p, yt, eps, labels) in zip(cases, prepared):
        _say(f"[noalloc] workload {idx} batch {batch}: allocation-free head vs workspace head")
        ref = _run(p, net, yt, eps, labels, noalloc=False)
        got = _run(p, net, yt, eps, labels, noalloc=True)
        assert torch.isfinite(got[1]).all()
        for a, b in zip(got, ref):
            assert torch.equal(a, b)
        p.close()


def test_noalloc_head_rejects_oversized_problem():
    """B (C + K + 1) floats above the fixed 4 MiB array: PNN_ERR_TOO_LARGE, nothing enqueued (the
    pointers below are never dereferenced)."""
    from paper_2103_08802_amd import binding as B
    net = S.config(5, 1024)                    # VGG-16-4 at 224 px: 512 channels, 1000 classes
    p = B.Plan(net)
    L = B.lib()
    a = 1 << 30
    st = L.pnn_head_fwd_bwd_noalloc(p.handle, a, a + 256, a + 512, None, a + 768, a + 1024, a + 1280, None)
    assert st == -9
    assert B.pnn_status_string(-9).startswith("the problem exceeds")
    p.close()
