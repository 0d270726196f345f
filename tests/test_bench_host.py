"""Host-side logic of bench.py that needs no GPU: turning rocprofv3 counter CSVs into
HBM bytes per GEMM launch, and the stored-reading lookup keyed by the GEMM sources."""
import csv
import json
import os
import sys

import pytest

from conftest import ROOT

sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _write_csv(path, rows):
    with open(path, "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for k, c, v in rows:
            w.writerow({"Kernel_Name": k, "Counter_Name": c, "Counter_Value": v})


@pytest.mark.parametrize("tall", [False, True])
def test_ingest_pmc_scales_by_copy_calibration(tmp_path, monkeypatch, tall):
    kind = "swiglu_gemm_tall_kernel" if tall else "swiglu_gemm_kernel"
    up = f"void rfx::(anonymous namespace)::{kind}<true>(unsigned short const*, int)"
    dn = f"void rfx::(anonymous namespace)::{kind}<false>(unsigned short const*, int)"
    other = "void rfx::(anonymous namespace)::topk_kernel(float const*)"
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    cfetch, cwrite = tmp_path / "cf.csv", tmp_path / "cw.csv"
    # two dispatches per GEMM: per-dispatch means 300 / 150 KiB read, 20 / 40 KiB written
    _write_csv(fetch, [(up, "FETCH_SIZE", 200), (up, "FETCH_SIZE", 400), (dn, "FETCH_SIZE", 150),
                       (dn, "FETCH_SIZE", 150), (other, "FETCH_SIZE", 9)])
    _write_csv(write, [(up, "WRITE_SIZE", 20), (up, "WRITE_SIZE", 20), (dn, "WRITE_SIZE", 40),
                       (dn, "WRITE_SIZE", 40)])
    # the copy reads half of what it moves on FETCH_SIZE (factor 2), all of it on WRITE_SIZE;
    # small readings of other kernels are not the copy
    ck = bench.COPY_CAL_BYTES / 1024.0
    _write_csv(cfetch, [("copyBuffer", "FETCH_SIZE", ck / 2), ("copyBuffer", "FETCH_SIZE", ck / 2),
                        ("fill", "FETCH_SIZE", 3)])
    _write_csv(cwrite, [("copyBuffer", "WRITE_SIZE", ck), ("fill", "WRITE_SIZE", 1)])
    tf = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tf))
    bench.ingest_pmc("wl", "row-major", str(fetch), str(write), str(cfetch), str(cwrite))
    data = json.loads(tf.read_text())
    assert data["calibration"]["fetch_factor"] == pytest.approx(2.0)
    assert data["calibration"]["write_factor"] == pytest.approx(1.0)
    ent = {e["kernel"]: e for e in data["entries"]}
    assert ent["gemm_up"]["kernel_name"] == f"{kind}<true>"
    assert ent["gemm_up"]["dispatches"] == [2, 2]
    assert ent["gemm_up"]["read_bytes"] == 300 * 1024 * 2
    assert ent["gemm_up"]["write_bytes"] == 20 * 1024
    assert ent["gemm_down"]["traffic_bytes"] == 150 * 1024 * 2 + 40 * 1024
    # the lookup returns the stored bytes while the GEMM source is unchanged ...
    assert bench.measured_traffic("wl", "row-major", "gemm_up") == 300 * 2048 + 20 * 1024
    assert bench.measured_traffic("other", "row-major", "gemm_up") is None
    # ... and nothing once the digest no longer matches
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 64)
    assert bench.measured_traffic("wl", "row-major", "gemm_up") is None


def test_ingest_pmc_counts_routed_launches_only_with_a_shared_expert(tmp_path, monkeypatch):
    # per forward: the routed up and down GEMMs and the shared expert's dense up and down
    # on the same kernels, the shared ones on a second stream, so either pair member may
    # come first; only the routed launch (the larger reading of each pair) counts
    up = "void rfx::(anonymous namespace)::swiglu_gemm_kernel<true>(int)"
    dn = "void rfx::(anonymous namespace)::swiglu_gemm_kernel<false>(int)"
    fetch, write = tmp_path / "f.csv", tmp_path / "w.csv"
    frows, wrows = [], []
    routed = [(up, 1000, 10), (dn, 500, 50)]
    shared = [(up, 7, 1), (dn, 3, 2)]
    for fwd in range(3):
        order = routed + shared if fwd != 1 else [shared[0], routed[0], shared[1], routed[1]]
        for name, f, w in order:
            frows.append((name, "FETCH_SIZE", f))
            wrows.append((name, "WRITE_SIZE", w))
    def dump(path, rows):
        with open(path, "w", newline="") as fh:
            w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name",
                                               "Counter_Value"])
            w.writeheader()
            # rows out of dispatch order in the file: the ingest sorts by Dispatch_Id
            for i, (k, c, v) in reversed(list(enumerate(rows))):
                w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": k, "Counter_Name": c,
                            "Counter_Value": v})
    dump(fetch, frows)
    dump(write, wrows)
    ck = bench.COPY_CAL_BYTES / 1024.0
    cf, cw = tmp_path / "cf.csv", tmp_path / "cw.csv"
    _write_csv(cf, [("copyBuffer", "FETCH_SIZE", ck)])
    _write_csv(cw, [("copyBuffer", "WRITE_SIZE", ck)])
    tf = tmp_path / "traffic.json"
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tf))
    bench.ingest_pmc("wl", "row-major", str(fetch), str(write), str(cf), str(cw), shared=True)
    ent = {e["kernel"]: e for e in json.loads(tf.read_text())["entries"]}
    assert ent["gemm_up"]["dispatches"] == [3, 3]
    assert ent["gemm_up"]["read_bytes"] == 1000 * 1024
    assert ent["gemm_up"]["write_bytes"] == 10 * 1024
    assert ent["gemm_down"]["read_bytes"] == 500 * 1024
    assert ent["gemm_down"]["write_bytes"] == 50 * 1024
    # a launch count that is not two per forward is an error, not a silent mean
    dump(fetch, frows[:-1])
    dump(write, wrows[:-1])
    with pytest.raises(SystemExit):
        bench.ingest_pmc("wl", "row-major", str(fetch), str(write), str(cf), str(cw), shared=True)


def test_ingest_pmc_missing_kernel_is_an_error(tmp_path, monkeypatch):
    fetch = tmp_path / "f.csv"
    _write_csv(fetch, [("void rfx::(anonymous namespace)::topk_kernel(float const*)", "FETCH_SIZE", 1)])
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    ck = bench.COPY_CAL_BYTES / 1024.0
    cf = tmp_path / "cf.csv"
    _write_csv(cf, [("copyBuffer", "FETCH_SIZE", ck / 2)])
    cw = tmp_path / "cw.csv"
    _write_csv(cw, [("copyBuffer", "WRITE_SIZE", ck)])
    with pytest.raises(SystemExit):
        bench.ingest_pmc("wl", "row-major", str(fetch), str(fetch), str(cf), str(cw))
    assert not os.path.exists(tmp_path / "traffic.json")


def test_stage_roofline_credits_only_algorithmic_bytes():
    import bench
    d, f, T, E = 2048, 1024, 8192, 64
    # MFMA-bound stack layer: FLOPs decide, weights + h once are the algorithmic bytes
    up = bench.stage_roofline("gemm_up", 0.4, d, f, 42826, 64, T, E)
    assert up["bound"] == "mfma" and up["algorithmic_flops"] == 4 * d * f * 42826
    assert up["algorithmic_bytes"] == 64 * 2 * f * d * 2 + T * d * 2
    assert up["overhead_bytes"] == (42826 - T) * d * 2 + 42826 * f * 2
    assert abs(up["achieved"] - 4 * d * f * 42826 / 0.4e-3 / 1e12) < 0.01
    # weight-bound single layer: bytes decide, pipeline traffic is not credited
    dn = bench.stage_roofline("gemm_down", 0.06, d, f, 5106, 64, 1024, E)
    assert dn["bound"] == "hbm" and dn["algorithmic_bytes"] == 64 * d * f * 2 + 1024 * d * 2
    assert dn["overhead_bytes"] == 5106 * f * 2 + (5106 - 1024) * d * 2
    assert dn["frac"] == round(dn["algorithmic_bytes"] / 0.06e-3 / 1e9 / bench.PEAK_HBM_GBS, 4)
