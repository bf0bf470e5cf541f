"""Thin ctypes binding of libpnn (``include/pnn.h``): argument marshalling only.

Every function here has the name of the C entry point it calls and takes device pointers as
Python ints (or objects with ``data_ptr()``, e.g. torch tensors).  All computation happens in the
library's HIP kernels; this module never falls back to anything else: if the library is missing it
raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpnn.so")

PNN_F32, PNN_BF16 = 0, 1
PNN_WS_SAVED, PNN_WS_SCRATCH = 0, 1
OPS = {"conv": 0, "bnact": 1, "maxpool3": 2}
STATUS = {0: "PNN_OK", -1: "PNN_ERR_NULL", -2: "PNN_ERR_SHAPE", -3: "PNN_ERR_DTYPE",
          -4: "PNN_ERR_WORKSPACE", -5: "PNN_ERR_UNSUPPORTED", -6: "PNN_ERR_HIP", -7: "PNN_ERR_INDEX",
          -8: "PNN_ERR_ALIGN", -9: "PNN_ERR_TOO_LARGE"}

# every symbol include/pnn.h declares
EXPORTS = ["pnn_plan_create", "pnn_plan_destroy", "pnn_workspace_size", "pnn_param_layout",
           "pnn_tensor_shape", "pnn_pre_fwd", "parareal_fine_fwd", "parareal_combine_fwd",
           "coarse_fwd", "pnn_head_fwd_bwd", "coarse_bwd", "parareal_fine_bwd",
           "parareal_combine_bwd", "pnn_pre_bwd", "pnn_status_string", "pnn_inspect",
           "pnn_timing_enable", "pnn_timing_read", "pnn_sgd_step", "coarse_bwd_all", "coarse_fwd_all",
           "pnn_set_streams",
           "parareal_bwd", "pnn_head_fwd_bwd_noalloc", "pnn_set_resident", "pnn_flags_clear"]


class PnnError(RuntimeError):
    def __init__(self, status, where):
        super().__init__(f"{where}: {STATUS.get(status, status)} ({status})")
        self.status = status


class NodeDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in
                ("op", "src", "dst", "bn", "pool", "k", "stride", "pad", "cout", "res")]


class SegmentDesc(ctypes.Structure):
    _fields_ = [("in_h", ctypes.c_int), ("in_w", ctypes.c_int), ("in_c", ctypes.c_int),
                ("n_nodes", ctypes.c_int), ("nodes", ctypes.POINTER(NodeDesc)),
                ("n_bn", ctypes.c_int), ("bn_slot", ctypes.POINTER(ctypes.c_int)),
                ("out_slot", ctypes.c_int)]


class NetDesc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("batch", ctypes.c_int), ("img_h", ctypes.c_int),
                ("img_w", ctypes.c_int), ("img_c", ctypes.c_int), ("n_sub", ctypes.c_int),
                ("n_classes", ctypes.c_int), ("pre", ctypes.POINTER(SegmentDesc)),
                ("fine", ctypes.POINTER(SegmentDesc)), ("coarse", ctypes.POINTER(SegmentDesc))]


_lib = None
_vp = ctypes.c_void_p
_PP = ctypes.POINTER(ctypes.c_void_p)


def lib():
    """Load libpnn.so (built in-tree by ``__graft_entry__.build()``); raise if it is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"libpnn.so not built ({LIB_PATH}); run __graft_entry__.build()")
    L = ctypes.CDLL(LIB_PATH)
    i, sz = ctypes.c_int, ctypes.c_size_t
    L.pnn_plan_create.argtypes = [ctypes.POINTER(NetDesc), ctypes.POINTER(_vp)]
    L.pnn_plan_destroy.argtypes = [_vp]
    L.pnn_plan_destroy.restype = None
    L.pnn_workspace_size.argtypes = [_vp, i, ctypes.POINTER(sz)]
    L.pnn_param_layout.argtypes = [_vp, i, i, i, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    L.pnn_tensor_shape.argtypes = [_vp, i, i, ctypes.POINTER(i), ctypes.POINTER(i), ctypes.POINTER(i)]
    L.pnn_pre_fwd.argtypes = [_vp, _vp, _PP, _PP, _vp, _vp, _vp]
    L.parareal_fine_fwd.argtypes = [_vp, _PP, _PP, _PP, _vp, _vp, _vp]
    L.parareal_combine_fwd.argtypes = [_vp, _PP, _PP, _PP, _vp, _vp, _vp]
    L.coarse_fwd.argtypes = [_vp, i, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    L.pnn_head_fwd_bwd.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    L.pnn_head_fwd_bwd_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    L.coarse_bwd.argtypes = [_vp, i, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    L.parareal_fine_bwd.argtypes = [_vp, _PP, _PP, _PP, _vp, _PP, _PP, _vp, _vp]
    L.parareal_combine_bwd.argtypes = [_vp, _PP, _PP, _vp]
    L.pnn_pre_bwd.argtypes = [_vp, _vp, _PP, _PP, _vp, _PP, _vp, _vp]
    L.pnn_status_string.argtypes = [i]
    L.pnn_status_string.restype = ctypes.c_char_p
    L.pnn_inspect.argtypes = [_vp, i, i, i, i, ctypes.POINTER(sz)]
    L.pnn_timing_enable.argtypes = [_vp, i]
    L.pnn_set_streams.argtypes = [_vp, i]
    L.pnn_set_resident.argtypes = [_vp, i]
    L.pnn_flags_clear.argtypes = [_vp, _vp, _vp]
    L.pnn_timing_read.argtypes = [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_longlong),
                                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]
    L.coarse_bwd_all.argtypes = [_vp, _PP, _PP, _PP, _vp, _PP, _vp, _vp]
    L.coarse_fwd_all.argtypes = [_vp, _PP, _PP, _PP, _vp, _vp, _vp]
    L.parareal_bwd.argtypes = [_vp, _PP, _PP, _PP, _PP, _PP, _PP, _PP, _PP, _vp, _vp, _vp]
    f = ctypes.c_float
    L.pnn_sgd_step.argtypes = [_vp, i, _PP, _PP, _PP, _PP, i, f, f, f, i, _vp]
    for name in EXPORTS:
        getattr(L, name)          # every declared entry point must be exported
    _lib = L
    return L


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _arr(xs):
    a = (ctypes.c_void_p * len(xs))(*[_ptr(x) for x in xs])
    return ctypes.cast(a, _PP), a


def _check(st, where):
    if st != 0:
        raise PnnError(st, where)


# ------------------------------------------------------------------------------------------------
# network description marshalling
# ------------------------------------------------------------------------------------------------

class _DescHolder:
    """ctypes mirror of a ``pnn_synth.Net`` (keeps every array alive while in use)."""

    def __init__(self, net):
        self.keep = []

        def seg(s):
            nodes = (NodeDesc * max(1, len(s.nodes)))()
            for i, n in enumerate(s.nodes):
                nodes[i] = NodeDesc(OPS[n.op], n.src, n.dst, n.bn, n.pool, n.k, n.stride, n.pad,
                                    n.cout, n.res)
            bns = (ctypes.c_int * max(1, len(s.bns)))(*s.bns)
            self.keep += [nodes, bns]
            return SegmentDesc(s.in_shape[0], s.in_shape[1], s.in_shape[2], len(s.nodes), nodes,
                               len(s.bns), bns, s.out)

        def segs(lst):
            a = (SegmentDesc * max(1, len(lst)))(*[seg(s) for s in lst])
            self.keep.append(a)
            return a

        H, W, C = net.in_shape
        self.desc = NetDesc(PNN_BF16 if net.dtype == "bf16" else PNN_F32, net.batch, H, W, C,
                            net.n_sub, net.classes, segs(net.pre), segs(net.fine), segs(net.coarse))


class Plan:
    """Owns a pnn_plan* built from a ``pnn_synth.Net``."""

    def __init__(self, net):
        L = lib()
        self.net = net
        holder = _DescHolder(net)
        h = ctypes.c_void_p()
        _check(L.pnn_plan_create(ctypes.byref(holder.desc), ctypes.byref(h)), "pnn_plan_create")
        self.handle = h

    def close(self):
        if self.handle:
            lib().pnn_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_size(self, kind):
        v = ctypes.c_size_t()
        _check(lib().pnn_workspace_size(self.handle, kind, ctypes.byref(v)), "pnn_workspace_size")
        return v.value

    def param_layout(self, part, j, grad):
        seg = [self.net.pre, self.net.fine, self.net.coarse][part][j]
        n = len(seg.nodes) + 2 * len(seg.bns)
        offs = (ctypes.c_size_t * max(1, n))()
        tot = ctypes.c_size_t()
        _check(lib().pnn_param_layout(self.handle, part, j, grad, offs, ctypes.byref(tot)),
               "pnn_param_layout")
        return [offs[i] for i in range(n)], tot.value

    def inspect(self, part, j, what, idx):
        """Byte offset of an internal tensor (see pnn_inspect), or None if the library does not
        hold it."""
        v = ctypes.c_size_t()
        st = lib().pnn_inspect(self.handle, part, j, what, idx, ctypes.byref(v))
        if st == -7:
            return None
        _check(st, "pnn_inspect")
        return v.value

    def tensor_shape(self, which, j):
        h, w, c = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        _check(lib().pnn_tensor_shape(self.handle, which, j, ctypes.byref(h), ctypes.byref(w),
                                      ctypes.byref(c)), "pnn_tensor_shape")
        return h.value, w.value, c.value


# ------------------------------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ------------------------------------------------------------------------------------------------

def pnn_pre_fwd(plan, image, x, delta, saved, scratch, stream):
    xa, k1 = _arr(x)
    da, k2 = _arr(delta)
    _check(lib().pnn_pre_fwd(plan.handle, _ptr(image), xa, da, _ptr(saved), _ptr(scratch), stream),
           "pnn_pre_fwd")


def parareal_fine_fwd(plan, x, phi, y, saved, scratch, stream):
    xa, k1 = _arr(x)
    pa, k2 = _arr(phi)
    ya, k3 = _arr(y)
    _check(lib().parareal_fine_fwd(plan.handle, xa, pa, ya, _ptr(saved), _ptr(scratch), stream),
           "parareal_fine_fwd")


def parareal_combine_fwd(plan, y, x, r, rnorm2, scratch, stream):
    ya, k1 = _arr(y)
    xa, k2 = _arr(x)
    ra, k3 = _arr(r if r else [0])
    _check(lib().parareal_combine_fwd(plan.handle, ya, xa, ra, _ptr(rnorm2), _ptr(scratch), stream),
           "parareal_combine_fwd")


def coarse_fwd(plan, j, rt_j, eta_j, add, rt_next, saved, scratch, stream):
    _check(lib().coarse_fwd(plan.handle, j, _ptr(rt_j), _ptr(eta_j), _ptr(add), _ptr(rt_next),
                            _ptr(saved), _ptr(scratch), stream), "coarse_fwd")


def pnn_head_fwd_bwd(plan, ytilde, eps, labels, logits, loss, D_N, deps, scratch, stream):
    _check(lib().pnn_head_fwd_bwd(plan.handle, _ptr(ytilde), _ptr(eps), _ptr(labels), _ptr(logits),
                                  _ptr(loss), _ptr(D_N), _ptr(deps), _ptr(scratch), stream),
           "pnn_head_fwd_bwd")


def pnn_head_fwd_bwd_noalloc(plan, ytilde, eps, labels, logits, loss, D_N, deps, stream):
    _check(lib().pnn_head_fwd_bwd_noalloc(plan.handle, _ptr(ytilde), _ptr(eps), _ptr(labels), _ptr(logits),
                                          _ptr(loss), _ptr(D_N), _ptr(deps), stream),
           "pnn_head_fwd_bwd_noalloc")


def coarse_bwd(plan, j, D_next, rt_j, eta_j, saved, D_j, deta_j, scratch, stream):
    _check(lib().coarse_bwd(plan.handle, j, _ptr(D_next), _ptr(rt_j), _ptr(eta_j), _ptr(saved),
                            _ptr(D_j), _ptr(deta_j), _ptr(scratch), stream), "coarse_bwd")


def parareal_fine_bwd(plan, dy, x, phi, saved, dx, dphi, scratch, stream):
    a1, k1 = _arr(dy)
    a2, k2 = _arr(x)
    a3, k3 = _arr(phi)
    a4, k4 = _arr(dx)
    a5, k5 = _arr(dphi)
    _check(lib().parareal_fine_bwd(plan.handle, a1, a2, a3, _ptr(saved), a4, a5, _ptr(scratch), stream),
           "parareal_fine_bwd")


def parareal_combine_bwd(plan, dx, D, stream):
    a1, k1 = _arr(dx)
    a2, k2 = _arr(D)
    _check(lib().parareal_combine_bwd(plan.handle, a1, a2, stream), "parareal_combine_bwd")


def coarse_fwd_all(plan, rt, eta, add, saved, scratch, stream):
    a1, k1 = _arr(rt)
    a2, k2 = _arr(eta)
    a3, k3 = _arr(add)
    _check(lib().coarse_fwd_all(plan.handle, a1, a2, a3, _ptr(saved), _ptr(scratch), stream),
           "coarse_fwd_all")


def coarse_bwd_all(plan, D, rt, eta, saved, deta, scratch, stream):
    a1, k1 = _arr(D)
    a2, k2 = _arr(rt)
    a3, k3 = _arr(eta)
    a4, k4 = _arr(deta)
    _check(lib().coarse_bwd_all(plan.handle, a1, a2, a3, _ptr(saved), a4, _ptr(scratch), stream),
           "coarse_bwd_all")


def parareal_bwd(plan, D, rt, eta, deta, x, phi, dx, dphi, saved, scratch, stream):
    a1, k1 = _arr(D)
    a2, k2 = _arr(rt)
    a3, k3 = _arr(eta)
    a4, k4 = _arr(deta)
    a5, k5 = _arr(x)
    a6, k6 = _arr(phi)
    a7, k7 = _arr(dx)
    a8, k8 = _arr(dphi)
    _check(lib().parareal_bwd(plan.handle, a1, a2, a3, a4, a5, a6, a7, a8, _ptr(saved), _ptr(scratch), stream),
           "parareal_bwd")


def pnn_sgd_step(plan, part, params, grads, momentum, lr, mu, weight_decay, nesterov, stream,
                 master=None, master_init=False):
    a1, k1 = _arr(params)
    a2, k2 = _arr(grads)
    a3, k3 = _arr(momentum)
    a4, k4 = _arr(master) if master is not None else (None, None)
    _check(lib().pnn_sgd_step(plan.handle, part, a1, a2, a3, a4, int(bool(master_init)), lr, mu,
                              weight_decay, int(bool(nesterov)), stream), "pnn_sgd_step")


def pnn_pre_bwd(plan, image, g, delta, saved, ddelta, scratch, stream):
    a1, k1 = _arr(g)
    a2, k2 = _arr(delta)
    a3, k3 = _arr(ddelta)
    _check(lib().pnn_pre_bwd(plan.handle, _ptr(image), a1, a2, _ptr(saved), a3, _ptr(scratch), stream),
           "pnn_pre_bwd")


def pnn_set_streams(plan, streams):
    _check(lib().pnn_set_streams(plan.handle, streams), "pnn_set_streams")


def pnn_set_resident(plan, on):
    _check(lib().pnn_set_resident(plan.handle, int(bool(on))), "pnn_set_resident")


def pnn_flags_clear(plan, scratch, stream):
    _check(lib().pnn_flags_clear(plan.handle, _ptr(scratch), stream), "pnn_flags_clear")


def pnn_timing_enable(plan, family):
    _check(lib().pnn_timing_enable(plan.handle, family), "pnn_timing_enable")


def pnn_timing_read(plan):
    ms, n, fl, by = ctypes.c_double(), ctypes.c_longlong(), ctypes.c_double(), ctypes.c_double()
    _check(lib().pnn_timing_read(plan.handle, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl),
                                 ctypes.byref(by)), "pnn_timing_read")
    return ms.value, n.value, fl.value, by.value


def pnn_status_string(st):
    return lib().pnn_status_string(st).decode()
