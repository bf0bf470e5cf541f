"""Writes tests/golden/conditioning.json: how far the bf16-storage oracle moves from itself when a
handful of its inputs are moved by one bfloat16 ulp, tensor family by tensor family, for the whole
training steps and the teacher-forced sub-networks that tests/test_gpu_e2e_bf16.py compares with
the GPU.

This is the smallest perturbation a bf16 implementation can differ by: any two implementations
that accumulate in a different order round some stored values differently by one ulp.  Deep
BN/ReLU networks at initialisation amplify such differences (ReLU masks and max-pool choices flip
across the whole depth), so this self-difference is a lower bound on what any bf16 implementation,
the GPU path included, can be held to end to end.

Calls only the oracle (oracle/) and the seeded input generators (pnn_synth/).

    python tests/golden/conditioning.py            # every case (about 20 minutes on 8 cores)
    python tests/golden/conditioning.py vgg16-b128 # one case
"""
from __future__ import annotations

import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import pnn_synth as S                                    # noqa: E402
from oracle import prim as P                             # noqa: E402
from oracle.net import ParaRealOracle, seg_backward, seg_forward   # noqa: E402
from tests.e2e_tensors import (family, grad_named, oracle_tensors, perturb_ulp,   # noqa: E402
                               rel_2)

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "conditioning.json")
PERTURBED = 4          # elements moved by one ulp
SEED = 77

# case name -> (workload index, batch, kind, sub-networks)
CASES = {
    "vgg16-b128": (1, 128, "step", None),
    "resnet1001-n4-b64": (2, 64, "step", None),
    "resnet1001-n16-b32": (3, 32, "step", None),
    "resnet1001-64px-n8-b8": (4, 8, "step", None),
    "resnet1001-64px-n8-b128-g1": (4, 128, "sub", 0),
    "resnet1001-64px-n8-b128-g3": (4, 128, "sub", 2),
    "resnet1001-64px-n8-b128-g6": (4, 128, "sub", 5),
    "resnet1001-64px-n8-b128-g8": (4, 128, "sub", 7),
}


def summarize(diff):
    """{family: {max, median, count, argmax}} of {tensor: e_2}, plus the non-parameter tensors."""
    fam = {}
    for k, v in diff.items():
        fam.setdefault(family(k), []).append((v, k))
    out = {"families": {}, "tensors": {}}
    for f, vals in sorted(fam.items()):
        e = np.array([v for v, _ in vals])
        out["families"][f] = {"max": float(e.max()), "median": float(np.median(e)), "count": len(vals),
                              "argmax": max(vals)[1]}
    for k, v in diff.items():
        if family(k) in ("forward", "D", "dx", "head"):
            out["tensors"][k] = v
    return out


def step_case(idx, batch):
    """Whole step: the seeded image against the same image with PERTURBED elements one ulp up."""
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    o = ParaRealOracle(net, params, bf16=True)
    ref = oracle_tensors(net, *o.step(x, labels))
    got = oracle_tensors(net, *o.step(perturb_ulp(x, PERTURBED, SEED), labels))
    return {k: rel_2(got[k], ref[k]) for k in ref}


def sub_case(idx, batch, j):
    """Sub-network g^j alone at the full batch: x_j = C^j(image) against x_j with PERTURBED
    elements one ulp up, the same output gradient (a seeded N(0, 1) tensor standing in for D_j:
    the relative differences do not depend on its scale)."""
    net = S.config(idx, batch)
    x, labels, params = S.make_all(net)
    st = P.round_bf16
    xj, _ = seg_forward(net.pre[j], params["pre"][j], x, st)
    rng = np.random.default_rng(SEED + j)
    res = []
    for xin in (xj, perturb_ulp(xj, PERTURBED, SEED)):
        y, run = seg_forward(net.fine[j], params["fine"][j], xin, st)
        D = st(rng.standard_normal(y.shape)) if not res else res[0]["_D"]
        dx, dphi = seg_backward(run, D, st)
        del run
        t = {f"y{j}": y, f"dx{j}": dx, "_D": D}
        t.update(grad_named("fine", j, dphi))
        res.append(t)
    ref, got = res
    return {k: rel_2(got[k], ref[k]) for k in ref if k != "_D"}


def main(names):
    data = json.load(open(OUT)) if os.path.exists(OUT) else {}
    data["_about"] = ("e_2 of every tensor of the bf16-storage oracle against itself with "
                      f"{PERTURBED} input elements moved up by one bf16 ulp (seed {SEED}); written by "
                      "tests/golden/conditioning.py")
    for name in names:
        idx, batch, kind, j = CASES[name]
        t = time.time()
        diff = step_case(idx, batch) if kind == "step" else sub_case(idx, batch, j)
        data[name] = summarize(diff)
        print(f"{name}: {time.time() - t:.0f} s", flush=True)
        for f, v in data[name]["families"].items():
            print(f"  {f:12s} max {v['max']:.3e} median {v['median']:.3e} ({v['argmax']})", flush=True)
        with open(OUT, "w") as fh:
            json.dump(data, fh, indent=1, sort_keys=True)


if __name__ == "__main__":
    main(sys.argv[1:] or list(CASES))
