"""Host logic of bench.py that needs no GPU: the HBM-traffic summary of two
rocprofv3 counter runs (calibration against a plain streaming kernel) and
the generic per-kernel counter table, on synthetic counter files."""
import csv
import importlib.util
import os

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


FIELDS = ["Correlation_Id", "Dispatch_Id", "Agent_Id", "Queue_Id", "Process_Id", "Thread_Id", "Grid_Size",
          "Kernel_Id", "Kernel_Name", "Workgroup_Size", "LDS_Block_Size", "Scratch_Size", "VGPR_Count",
          "Accum_VGPR_Count", "SGPR_Count", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _csv(path, rows):
    """rows: (dispatch, kernel name, counter, value); two agents' halves per value
    (the per-dispatch figure is the sum over records)."""
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, FIELDS)
        w.writeheader()
        for d, name, ctr, val in rows:
            for half in (0.25, 0.75):
                w.writerow({**{k: 0 for k in FIELDS}, "Dispatch_Id": d, "Kernel_Name": name, "Counter_Name": ctr,
                            "Counter_Value": val * half})
    return path


NEG = "void at::native::vectorized_elementwise_kernel<8, at::native::neg_kernel_cuda(at::TensorIteratorBase&)>(int)"
COMPACT = "kara::(anonymous namespace)::compact_kernel(kara::Geom, int const*)"
SELECT = "void kara::(anonymous namespace)::select_kernel<8>(kara::Geom, int)"
SCORE = "void kara::(anonymous namespace)::score_kernel<0, 128, 4>(kara::(anonymous namespace)::ScoreArgs)"
SPLIT = "kara::(anonymous namespace)::split_sum_kernel(float const*, float*, int, int)"


def test_calibration_totals_every_dispatch_of_the_streaming_kernel(bench, tmp_path):
    gib = 4.0
    true_bytes = gib * 2**30
    # the negation runs as two dispatches; FETCH_SIZE reads half the bytes
    # moved, WRITE_SIZE all of them (KiB per dispatch)
    half_kib = true_bytes / 2 / 1024
    fetch = [(1, NEG, "FETCH_SIZE", half_kib / 2), (2, NEG, "FETCH_SIZE", half_kib / 2),
             (3, COMPACT, "FETCH_SIZE", 1000.0), (4, SELECT, "FETCH_SIZE", 10.0), (5, SELECT, "FETCH_SIZE", 30.0),
             (6, SCORE, "FETCH_SIZE", 5000.0), (7, SPLIT, "FETCH_SIZE", 100.0)]
    write = [(1, NEG, "WRITE_SIZE", half_kib), (2, NEG, "WRITE_SIZE", half_kib),
             (3, COMPACT, "WRITE_SIZE", 2000.0), (4, SELECT, "WRITE_SIZE", 4.0), (5, SELECT, "WRITE_SIZE", 6.0),
             (6, SCORE, "WRITE_SIZE", 300.0), (7, SPLIT, "WRITE_SIZE", 7.0)]
    f = _csv(tmp_path / "fetch.csv", fetch)
    w = _csv(tmp_path / "write.csv", write)
    text = bench.summarize_pmc(str(f), str(w), "qwen14b", gib)
    assert "(2 dispatches)" in text
    blob = bench.json.loads(text.split("```json", 1)[1].split("```", 1)[0])
    assert blob["fetch_scale"] == pytest.approx(2.0)
    assert blob["write_scale"] == pytest.approx(1.0)
    kib = 1024.0
    # one pass of a stage per dispatch of its first kernel
    want_sc = (1000.0 * 2 + 2000.0) * kib + (10.0 * 2 + 4.0 + 30.0 * 2 + 6.0) * kib
    assert blob["select_compact"]["hbm_bytes_per_launch"] == pytest.approx(want_sc)
    want_score = (5000.0 * 2 + 300.0 + 100.0 * 2 + 7.0) * kib
    assert blob["score"]["hbm_bytes_per_launch"] == pytest.approx(want_score)
    assert blob["select_compact"]["sources_sha256"] == bench.sources_sha256(bench.TRAFFIC_SOURCES["select_compact"])


def test_calibration_missing_is_an_error(bench, tmp_path):
    f = _csv(tmp_path / "fetch.csv", [(3, COMPACT, "FETCH_SIZE", 1000.0)])
    w = _csv(tmp_path / "write.csv", [(3, COMPACT, "WRITE_SIZE", 1000.0)])
    with pytest.raises(SystemExit, match="calibration kernel is missing"):
        bench.summarize_pmc(str(f), str(w), "qwen14b", 4.0)


def test_counter_table_means_per_dispatch(bench, tmp_path):
    a = _csv(tmp_path / "a.csv", [(1, COMPACT, "TCC_EA0_RDREQ_128B_sum", 10.0), (2, COMPACT, "TCC_EA0_RDREQ_128B_sum", 30.0),
                                  (3, SELECT, "TCC_EA0_RDREQ_128B_sum", 4.0)])
    b = _csv(tmp_path / "b.csv", [(1, COMPACT, "TCC_EA0_WRREQ_64B_sum", 8.0), (2, COMPACT, "TCC_EA0_WRREQ_64B_sum", 8.0)])
    table = bench.summarize_counters([str(a), str(b)])
    lines = {ln.split("|")[1].strip(): ln for ln in table.splitlines()[2:]}
    cells = [c.strip() for c in lines["kara::compact_kernel"].split("|")[1:-1]]
    assert cells[1] == "2"                       # dispatches
    assert float(cells[2]) == pytest.approx(20.0)  # mean of 10 and 30 (columns sorted by name)
    assert float(cells[3]) == pytest.approx(8.0)
    cells = [c.strip() for c in lines["kara::select_kernel<8>"].split("|")[1:-1]]
    assert cells[1] == "1" and float(cells[2]) == pytest.approx(4.0) and cells[3] == ""


def test_staged_traffic_goes_stale_when_sources_change(bench, tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    blob = {"score": {"hbm_bytes_per_launch": 1.0, "sources_sha256": bench.sources_sha256(bench.TRAFFIC_SOURCES["score"])},
            "select_compact": {"hbm_bytes_per_launch": 2.0, "sources_sha256": "0" * 64}}
    (prof / "hbm_traffic_x.md").write_text("text\n```json\n" + bench.json.dumps(blob) + "\n```\n")
    monkeypatch.setattr(bench, "traffic_path", lambda wl: str(prof / f"hbm_traffic_{wl}.md"))
    got = bench.load_traffic("x")
    assert got == {"score": 1.0, "select_compact": None}
