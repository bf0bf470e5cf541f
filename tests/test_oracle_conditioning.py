"""The conditioning of the workloads' training steps, measured on the oracle alone (CPU): how far the
bf16-storage oracle moves from itself when four image elements (or, for a teacher-forced
sub-network, four of its input elements) are moved by one bfloat16 ulp.

tests/golden/conditioning.json holds these self-differences per tensor family for every case that
tests/test_gpu_e2e_bf16.py compares with the GPU (written by tests/golden/conditioning.py, which
calls only the oracle and the seeded input generators; the full table takes about 20 minutes on 8
cores).  Here: the table covers those cases, the VGG-16 row is recomputed live and must reproduce
the stored numbers (the oracle is deterministic), and the ResNet-1001 rows show the property the
GPU bar rests on: at the workloads' batches a one-ulp input change moves the deep gradients by
O(1), far beyond 2e-2, so no bf16 implementation can be held to 2e-2 on them end to end."""
import json
import os

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
TABLE = os.path.join(HERE, "golden", "conditioning.json")

GPU_ROWS = ["vgg16-b128", "resnet1001-n4-b64", "resnet1001-n16-b32", "resnet1001-64px-n8-b8",
            "resnet1001-64px-n8-b128-g1", "resnet1001-64px-n8-b128-g3", "resnet1001-64px-n8-b128-g6",
            "resnet1001-64px-n8-b128-g8"]


def _table():
    with open(TABLE) as f:
        return json.load(f)


def test_table_covers_every_gpu_case():
    t = _table()
    for row in GPU_ROWS:
        assert row in t, row
        fam = t[row]["families"]
        assert "fine.conv" in fam and fam["fine.conv"]["count"] > 0


def test_resnet_gradients_are_ill_conditioned():
    """Every ResNet-1001 row: the largest self-difference of the fine filter gradients is above 0.5,
    and that of the whole-step forward tensors above 2e-2 (the deep y_j)."""
    t = _table()
    for row in GPU_ROWS[1:]:
        fam = t[row]["families"]
        assert fam["fine.conv"]["max"] > 0.5, row
        assert fam["fine.bn"]["max"] > 0.5, row
        if "forward" in fam and not row.split("-")[-1].startswith("g"):
            assert fam["forward"]["max"] > 2e-2, row


def test_vgg_row_reproduces():
    """Recompute the VGG-16 workload's row (two oracle steps at batch 128) and compare with the
    stored table: the same numbers to rounding."""
    from tests.golden import conditioning as C
    stored = _table()["vgg16-b128"]["families"]
    idx, batch, kind, _ = C.CASES["vgg16-b128"]
    live = C.summarize(C.step_case(idx, batch))["families"]
    assert set(live) == set(stored)
    for f, v in live.items():
        assert v["max"] == pytest.approx(stored[f]["max"], rel=1e-9, abs=1e-15), f
        assert v["median"] == pytest.approx(stored[f]["median"], rel=1e-9, abs=1e-15), f
