"""Host logic of bench.py: turning rocprofv3 counter passes into the per-launch
traffic figure (scaled by a copy of known size) and looking it up again only
while the kernel's sources are unchanged."""

import csv
import importlib.util
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def write_pass(d, counter, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "x_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for name, v in rows:
            w.writerow({"Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def test_summarize_scales_by_the_copy_and_keeps_one_entry_per_routine(tmp_path, monkeypatch):
    b = load_bench()
    out = tmp_path / "traffic.json"
    monkeypatch.setattr(b, "TRAFFIC_FILE", str(out))
    k1 = "igemm_dma_kernel<bool _Accum, int, E, 128, 128, 64, 4, 2, 0, 8>"
    k2 = "conv1x1_stream_kernel<bool _Accum, 256, 32, 128, 2"
    # a 4 MiB copy that FETCH_SIZE reports as 2 MiB (factor 2) and WRITE_SIZE as 4 MiB
    write_pass(tmp_path / "f", "FETCH_SIZE", [("__amd_rocclr_copyBuffer", 2048.0), ("__amd_rocclr_copyBuffer", 8.0),
                                              ("void " + k1 + "(x)", 100.0), ("void " + k1 + "(x)", 300.0),
                                              ("void " + k2 + ", true>(y)", 50.0)])
    write_pass(tmp_path / "w", "WRITE_SIZE", [("__amd_rocclr_copyBuffer", 4096.0),
                                              ("void " + k1 + "(x)", 10.0), ("void " + k1 + "(x)", 30.0),
                                              ("void " + k2 + ", false>(y)", 20.0)])
    b.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), "r1", k1, str(out), calib_mib=4)
    # mean fetch 200 KiB x 2 + mean write 20 KiB x 1
    assert b.traffic_for("r1") == (200 * 2 + 20) * 1024
    b.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), "r2", k2, str(out), calib_mib=4)
    assert b.traffic_for("r2") == (50 * 2 + 20) * 1024
    assert b.traffic_for("r1") == (200 * 2 + 20) * 1024   # the first entry is kept
    assert b.traffic_for("r3") is None
    # a changed source hash makes the figure stale
    monkeypatch.setattr(b, "kernel_source_hash", lambda ksub=None: "different")
    assert b.traffic_for("r1") is None


def test_kernel_sources_cover_every_kernel_file():
    b = load_bench()
    kfiles = {f for f in os.listdir(b.KDIR) if f.endswith((".hip", ".hpp"))}
    assert kfiles == set(b.ALL_KERNEL_SOURCES)
    for files in b.KERNEL_SOURCES.values():
        assert set(files) <= kfiles


def test_more_than_one_gpu_exits_with_a_message(capsys, monkeypatch):
    b = load_bench()
    monkeypatch.setattr("sys.argv", ["bench.py", "--gpus", "2"])
    with pytest.raises(SystemExit) as e:
        b.main()
    assert e.value.code == 2
    assert "one GPU" in capsys.readouterr().err
