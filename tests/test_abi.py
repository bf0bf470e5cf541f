"""Host-side checks of the C ABI (no GPU needed): the library loads, exports every entry point that
include/pnn.h declares, builds plans for the five workloads, lays out parameters consistently with
the network descriptions, and rejects bad input with the documented status codes."""
import ctypes
import os
import re

import pytest

import pnn_synth as S
from oracle.net import param_count

B = pytest.importorskip("paper_2103_08802_amd.binding")
HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "pnn.h")


def _lib_or_skip():
    if not os.path.exists(B.LIB_PATH):
        pytest.skip("libpnn.so not built")
    return B.lib()


def test_header_declarations_are_exported():
    L = _lib_or_skip()
    text = open(HEADER).read()
    declared = set(re.findall(r"^\s*(?:pnn_status|void|const char\*)\s+(\w+)\s*\(", text, re.M))
    assert declared == set(B.EXPORTS)
    for name in declared:
        assert hasattr(L, name), name


@pytest.mark.parametrize("idx,coarse", [(i, "config") for i in range(6)] +
                         [(i, "paper") for i in range(1, 5)])
def test_plans_and_layouts(idx, coarse):
    _lib_or_skip()
    net = S.config(idx, 2, coarse=coarse)
    p = B.Plan(net)
    assert p.workspace_size(B.PNN_WS_SAVED) >= 0
    assert p.workspace_size(B.PNN_WS_SCRATCH) > 0
    pc = param_count(net)
    es = 2 if net.dtype == "bf16" else 4
    for part, segs, counts in ((0, net.pre, pc["pre"]), (1, net.fine, pc["fine"]), (2, net.coarse, pc["coarse"])):
        for j, seg in enumerate(segs):
            offs, tot = p.param_layout(part, j, 0)
            goffs, gtot = p.param_layout(part, j, 1)
            n_conv = sum(1 for n in seg.nodes if n.op == "conv")
            bn_params = sum(2 * S.segment_shapes(seg)[s][2] for s in seg.bns)
            conv_params = counts[j] - bn_params
            assert tot >= conv_params * es + bn_params * 4
            assert gtot >= (conv_params + bn_params) * 4
            assert all(o % 256 == 0 for o, n in zip(offs, seg.nodes) if n.op == "conv")
            assert len([o for o, n in zip(offs, seg.nodes) if n.op == "conv"]) == n_conv
    for j in range(net.n_sub):
        sh = S.segment_shapes(net.fine[j])
        assert p.tensor_shape(0, j) == sh[0]
        assert p.tensor_shape(1, j) == sh[net.fine[j].out]
    p.close()


@pytest.mark.parametrize("idx,coarse,dtype", [(i, "config", None) for i in range(6)] +
                         [(2, "paper", None), (3, "config", "f32"), (1, "config", "f32")])
def test_inspect_walk(idx, coarse, dtype):
    """Every tensor pnn_inspect can name lies inside its workspace: slot values (saved) and slot
    gradients (scratch) with their whole NHWC extent, BN output gradients and statistics by their
    offset; indices past the last answer PNN_ERR_INDEX."""
    _lib_or_skip()
    net = S.config(idx, 2, coarse=coarse)
    if dtype is not None:
        net.dtype = dtype
    p = B.Plan(net)
    saved, scratch = p.workspace_size(B.PNN_WS_SAVED), p.workspace_size(B.PNN_WS_SCRATCH)
    es = 2 if net.dtype == "bf16" else 4
    for part, segs in ((0, net.pre), (1, net.fine), (2, net.coarse)):
        for j, seg in enumerate(segs):
            sh = S.segment_shapes(seg)
            for what, ws in ((0, saved), (1, scratch)):
                for k in range(len(sh) + 2):
                    off = p.inspect(part, j, what, k)
                    if k == 0 or k == seg.out or k >= len(sh):
                        assert off is None, (part, j, what, k)
                        continue
                    if off is None:
                        continue
                    h, w, c = sh[k]
                    assert off + net.batch * h * w * c * es <= ws, (part, j, what, k)
            for what, ws in ((2, scratch), (3, saved)):
                n_ok = 0
                for k in range(len(seg.bns) + 2):
                    off = p.inspect(part, j, what, k)
                    if off is not None:
                        assert 0 <= off < ws
                        n_ok += 1
                assert n_ok <= len(seg.bns)
    p.close()


def test_error_codes():
    L = _lib_or_skip()
    h = ctypes.c_void_p()
    assert L.pnn_plan_create(None, ctypes.byref(h)) == -1                      # PNN_ERR_NULL
    net = S.config(0)
    d = B._DescHolder(net)
    d.desc.dtype = 7
    assert L.pnn_plan_create(ctypes.byref(d.desc), ctypes.byref(h)) == -3      # PNN_ERR_DTYPE
    d = B._DescHolder(net)
    d.desc.fine[1].in_c = 8                                                    # X_1 mismatch
    assert L.pnn_plan_create(ctypes.byref(d.desc), ctypes.byref(h)) == -2      # PNN_ERR_SHAPE
    net2 = S.config(0)
    net2.fine[0].nodes[0].cout = 24                                            # not a multiple of 16
    d = B._DescHolder(net2)
    assert L.pnn_plan_create(ctypes.byref(d.desc), ctypes.byref(h)) in (-2, -5)
    net3 = S.config(0)
    net3.fine[0].nodes[1].src = 5                                              # slot not produced yet
    d = B._DescHolder(net3)
    assert L.pnn_plan_create(ctypes.byref(d.desc), ctypes.byref(h)) == -2
    p = B.Plan(S.config(0))
    v = ctypes.c_size_t()
    assert L.pnn_workspace_size(p.handle, 9, ctypes.byref(v)) == -4            # PNN_ERR_WORKSPACE
    assert L.pnn_param_layout(p.handle, 1, 5, 0, None, ctypes.byref(v)) == -7  # PNN_ERR_INDEX
    assert L.coarse_fwd(p.handle, 3, 1, 1, 1, 2, 1, 1, None) == -7
    assert L.parareal_fine_fwd(p.handle, None, None, None, 1, 1, None) == -1
    assert L.pnn_set_streams(p.handle, 0) == -7                                # 1 .. 4 streams
    assert L.pnn_set_streams(p.handle, 5) == -7
    assert L.pnn_set_streams(p.handle, 1) == 0
    assert L.pnn_set_streams(None, 2) == -1
    # parareal_bwd: NULL arrays and aliased D_j / D_{j+1} are rejected before anything is enqueued
    assert L.parareal_bwd(p.handle, None, None, None, None, None, None, None, None, 1, 1, None) == -1
    N = S.config(0).n_sub
    arr = lambda vals: (ctypes.c_void_p * len(vals))(*vals)
    D = arr([16] * N)                                                          # D_0 aliases D_1
    ok = arr([16 * (i + 1) for i in range(N)])
    assert L.parareal_bwd(p.handle, D, ok, ok, ok, ok, ok, ok, ok, 1, 1, None) == -2
    # coarse_fwd_all: NULL arrays and aliased rt_j / rt_{j+1} are rejected the same way
    assert L.coarse_fwd_all(p.handle, None, None, None, 1, 1, None) == -1
    assert L.coarse_fwd_all(p.handle, D, ok, ok, 1, 1, None) == -2
    assert L.coarse_fwd_all(p.handle, ok, ok, ok, None, 1, None) == -1
    assert B.pnn_status_string(-5) == "network form not supported by this library"
    p.close()


def test_alignment_rules():
    """Tensor pointers must be 16-byte aligned and workspaces 256-byte aligned: a violation is
    rejected with PNN_ERR_ALIGN before anything is enqueued (checked here without a GPU: the
    pointers are never dereferenced)."""
    L = _lib_or_skip()
    net = S.config(3, 2)
    p = B.Plan(net)
    N = net.n_sub
    arr = lambda vals: (ctypes.c_void_p * len(vals))(*vals)
    base = 1 << 30
    ok = [base + (1 << 20) * (i + 1) for i in range(N)]
    ws, ws2 = base, base + (1 << 28)
    bad = list(ok)
    bad[3] += 8                                                                # one x_j off by 8 bytes
    A_ok, A_bad = arr(ok), arr(bad)
    assert L.parareal_fine_fwd(p.handle, A_bad, A_ok, A_ok, ws, ws2, None) == -8
    assert L.parareal_fine_fwd(p.handle, A_ok, A_ok, A_ok, ws + 128, ws2, None) == -8   # workspace
    assert L.parareal_fine_bwd(p.handle, A_ok, A_ok, A_ok, ws, A_bad, A_ok, ws2, None) == -8
    assert L.parareal_bwd(p.handle, A_bad, A_ok, A_ok, A_ok, A_ok, A_ok, A_ok, A_ok, ws, ws2, None) == -8
    assert L.parareal_combine_fwd(p.handle, A_ok, A_bad, A_ok, None, None, None) == -8
    assert L.parareal_combine_bwd(p.handle, A_bad, A_ok, None) == -8
    assert L.coarse_fwd(p.handle, 0, ok[0] + 4, ok[1], ok[2], ok[3], ws, ws2, None) == -8
    assert L.coarse_fwd_all(p.handle, A_ok, A_bad, A_ok, ws, ws2, None) == -8
    assert L.coarse_bwd(p.handle, 0, ok[0], ok[1], ok[2], ws, ok[3] + 2, ok[4], ws2, None) == -8
    assert L.coarse_bwd_all(p.handle, A_bad, A_ok, A_ok, ws, A_ok, ws2, None) == -8
    assert L.pnn_pre_fwd(p.handle, base + 1 + (1 << 29), A_ok, A_ok, ws, ws2, None) == -8
    assert L.pnn_pre_bwd(p.handle, base + (1 << 29), A_ok, A_ok, ws, A_bad, ws2, None) == -8
    assert L.pnn_head_fwd_bwd(p.handle, ok[0], ok[1], ok[2], None, ok[3] + 2, ok[4], ok[5], ws2, None) == -8
    assert L.pnn_head_fwd_bwd(p.handle, ok[0] + 8, ok[1], ok[2], None, ok[3], ok[4], ok[5], ws2, None) == -8
    assert L.pnn_sgd_step(p.handle, 1, A_bad, A_ok, A_ok, None, 0, ctypes.c_float(0.1), ctypes.c_float(0.9),
                          ctypes.c_float(5e-4), 1, None) == -8
    assert L.pnn_sgd_step(p.handle, 1, A_ok, A_ok, A_ok, A_bad, 1, ctypes.c_float(0.1), ctypes.c_float(0.9),
                          ctypes.c_float(5e-4), 1, None) == -8                  # master copies too
    assert L.pnn_flags_clear(p.handle, ws + 64, None) == -8
    assert B.pnn_status_string(-8) == "a pointer is not aligned as the interface requires"
    p.close()


def test_nonfinite_flag_words():
    """The non-finite flags: PNN_NFLAGS uint32 words inside scratch, on a 256-byte boundary, apart
    from the resident kernel's barrier words; pnn_flags_clear rejects NULL before enqueuing."""
    L = _lib_or_skip()
    p = B.Plan(S.config(3, 2))
    scr = p.workspace_size(B.PNN_WS_SCRATCH)
    off = p.inspect(0, 0, 5, 0)
    assert off % 256 == 0 and off + 8 <= scr
    assert off != p.inspect(0, 0, 4, 0)
    assert L.pnn_flags_clear(p.handle, None, None) == -1
    assert L.pnn_flags_clear(None, 1 << 30, None) == -1
    p.close()
