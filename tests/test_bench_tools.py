"""The profile summarisers of bench.py (no GPU work): HBM bytes per launch from the two PMC runs
scaled by the calibration copy, and the per-family and SQ-counter tables, on small synthetic
counter / trace files."""
import csv
import importlib.util
import json
import os

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def _write(path, header, rows):
    with open(path, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(header)
        w.writerows(rows)


def _pmc(path, counter, copy_kib, kern_kib):
    hdr = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"]
    rows = [[1, "__amd_rocclr_copyBuffer", counter, copy_kib]]
    rows += [[2 + i, "void pnn::conv_kernel<unsigned short, 0, 0, 2, 4>(pnn::ConvLaunch)", counter, v]
             for i, v in enumerate(kern_kib)]
    _write(path, hdr, rows)


def test_families_scale_by_the_calibration_copy(tmp_path):
    b = _bench()
    mib = b.COPY_BYTES >> 20
    # FETCH_SIZE reads half of the copy's bytes, WRITE_SIZE all of them (KiB per dispatch)
    _pmc(tmp_path / "f.csv", "FETCH_SIZE", mib * 512, [100.0, 300.0])
    _pmc(tmp_path / "w.csv", "WRITE_SIZE", mib * 1024, [50.0, 50.0])
    _write(tmp_path / "t.csv", ["Kernel_Name", "Start_Timestamp", "End_Timestamp"],
           [["void pnn::conv_kernel<unsigned short, 0, 0, 2, 4>(pnn::ConvLaunch)", 0, 2000],
            ["void pnn::conv_kernel<unsigned short, 0, 0, 2, 4>(pnn::ConvLaunch)", 5000, 7000]])
    out = tmp_path / "fam.md"
    b.summarize_families(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), str(tmp_path / "t.csv"),
                         str(out), "cmd")
    row = [l for l in out.read_text().splitlines() if l.startswith("| `conv_kernel`")][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    fetched_mb = 2 * 200.0 * 1024 / 1e6          # mean 200 KiB, scale 2
    written_mb = 50.0 * 1024 / 1e6
    assert abs(float(cells[2]) - fetched_mb) < 0.05 and abs(float(cells[3]) - written_mb) < 0.05
    assert cells[4] == "2.00"                      # microseconds
    assert abs(float(cells[5]) - (fetched_mb + written_mb) * 1e6 / 2000) < 1.0


def test_sq_ratios(tmp_path):
    b = _bench()
    names = ["SQ_WAVES", "SQ_WAVE_CYCLES", "SQ_BUSY_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_LDS",
             "SQ_ACTIVE_INST_LDS", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_LDS_BANK_CONFLICT"]
    vals = [10, 1000, 400, 500, 30, 40, 200, 80]
    k = "void pnn::conv_kernel<unsigned short, 1, 3, 2, 4>(pnn::ConvLaunch)"
    _write(tmp_path / "sq.csv", ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"],
           [[7, k, n, v] for n, v in zip(names, vals)])
    out = tmp_path / "sq.md"
    b.summarize_sq(str(tmp_path / "sq.csv"), str(out), "cmd")
    row = [l for l in out.read_text().splitlines() if "conv_kernel<unsigned short, 1, 3, 2, 4>" in l][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[1:] == ["1", "10", "100", "0.50", "0.03", "0.04", "2.00"]


def test_mfma_summary_and_record(tmp_path, monkeypatch):
    """MfmaUtil weighted by dispatch duration, MFMA FLOPs per dispatch and their ratio to the
    algorithmic FLOPs; the conv_kernel record carries the sources' hash and is read back by
    stored_mfma (None once a source changes)."""
    b = _bench()
    k = "void pnn::conv_kernel<unsigned short, 0, 0, 2, 4>(pnn::ConvLaunch)"
    rows = []
    for d, (u, fl, t0, t1) in enumerate([(10.0, 3e9, 0, 1000), (40.0, 1e9, 2000, 5000)]):
        rows.append([d, k, "MfmaUtil", u, t0, t1])
        rows.append([d, k, "MfmaFlopsBF16", fl, t0, t1])
    _write(tmp_path / "m.csv", ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                                "Start_Timestamp", "End_Timestamp"], rows)
    monkeypatch.setattr(b, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "profiles")
    os.makedirs(tmp_path / "paper_2103_08802_amd" / "csrc")
    for n in b.KERNEL_SOURCES["conv_kernel"]:
        (tmp_path / "paper_2103_08802_amd" / "csrc" / n).write_text(n)
    out = tmp_path / "m.md"
    b.summarize_mfma(str(tmp_path / "m.csv"), str(out), 1e9, "cmd")
    row = [l for l in out.read_text().splitlines() if l.startswith("| `conv_kernel`")][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[1] == "2" and cells[2] == "32.50" and cells[3] == "2.000"   # (10*1 + 40*3) / 4 us
    rec = json.loads((tmp_path / "profiles" / "mfma_conv_kernel.json").read_text())
    assert rec["mfma_over_algorithmic"] == 2.0
    assert b.stored_mfma("conv_kernel") == {"mfma_util_pct": 32.5, "mfma_flops_per_launch": 2000000000}
    (tmp_path / "paper_2103_08802_amd" / "csrc" / "k_conv.hip").write_text("changed")
    assert b.stored_mfma("conv_kernel") is None


def test_pmc_record_and_source_hash(tmp_path, monkeypatch):
    b = _bench()
    mib = b.COPY_BYTES >> 20
    _pmc(tmp_path / "f.csv", "FETCH_SIZE", mib * 512, [1000.0])
    _pmc(tmp_path / "w.csv", "WRITE_SIZE", mib * 1024, [250.0])
    monkeypatch.setattr(b, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "profiles")
    os.makedirs(tmp_path / "paper_2103_08802_amd" / "csrc")
    for n in b.KERNEL_SOURCES["conv_kernel"]:
        (tmp_path / "paper_2103_08802_amd" / "csrc" / n).write_text(n)
    b.summarize_pmc(str(tmp_path / "f.csv"), str(tmp_path / "w.csv"), "conv_kernel", "cmd")
    rec = json.loads((tmp_path / "profiles" / "traffic_conv_kernel.json").read_text())
    assert rec["fetch_bytes_per_launch"] == 2 * 1000 * 1024
    assert rec["write_bytes_per_launch"] == 250 * 1024
    assert rec["sources_sha256"] == b._sources_sha("conv_kernel")
