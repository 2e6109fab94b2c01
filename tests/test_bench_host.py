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
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for k, (name, v) in enumerate(rows):
            w.writerow({"Dispatch_Id": k + 1, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": v})


def test_summarize_attributes_dispatches_to_layers_and_scales_by_the_copy(tmp_path, monkeypatch):
    import json
    b = load_bench()
    out = tmp_path / "traffic.json"
    # a path of 3 layers: layer 1 one launch (a converter + its routine = 2
    # launches for layer 2), layer 3 one launch; one warm-up and two timed steps
    ka = "_ZN2sn1k16conv1x1_stream_kernelIDF16bLi256EEEvNS0_10StreamArgsE"
    kc = "_ZN2sn1k14convert_kernelItLi0ELi1EEEvPKT_PS2_iiiiii"
    kb = "_ZN2sn1k16igemm_dma_kernelIDF16bLi1ELi128EEEvNS0_6IgArgsE"
    launches = [1, 2, 2, 3]
    info = {"workload": "w", "warmup": 1, "steps": 2, "routines": ["input/nchw", "r1", "r2", "r1"],
            "launch_layers": launches}
    (tmp_path / "pass.json").write_text(json.dumps(info))
    step = [ka, kc, kb, ka]
    fetch = [("__amd_rocclr_fillBuffer", 1.0)]          # a torch kernel before the steps
    write = [("__amd_rocclr_fillBuffer", 1.0)]
    for s_i, scale in enumerate([9.0, 1.0, 3.0]):       # the warm-up step is ignored
        fetch += [(k, scale * (10 + q)) for q, k in enumerate(step)]
        write += [(k, scale * 2.0) for k in step]
    # a 4 MiB copy that FETCH_SIZE reports as 2 MiB (factor 2) and WRITE_SIZE as 4 MiB
    fetch.append(("__amd_rocclr_copyBuffer", 2048.0))
    write.append(("__amd_rocclr_copyBuffer", 4096.0))
    write_pass(tmp_path / "f", "FETCH_SIZE", fetch)
    write_pass(tmp_path / "w", "WRITE_SIZE", write)
    b.summarize_pmc(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "pass.json"), str(out), calib_mib=4)
    summ = json.loads(out.read_text())
    by = {e["layer"]: e for e in summ["layers"]}
    assert set(by) == {1, 2, 3} and by[2]["launches"] == 2
    # timed-step means: fetch KiB (10, 11 + 12, 13) x 2 (scales 1 and 3), write 2 x 2 per launch
    assert by[1]["bytes"] == (10 * 2 * 2 + 2 * 2) * 1024
    assert by[2]["bytes"] == ((11 + 12) * 2 * 2 + 2 * 2 * 2) * 1024
    assert by[3]["bytes"] == (13 * 2 * 2 + 2 * 2) * 1024
    # lookup: every layer of the routine must be covered, by the same routine
    t, why = b.traffic_for_layers([1, 3], "r1", summ)
    assert t == (by[1]["bytes"] + by[3]["bytes"]) // 2 and why is None
    t, why = b.traffic_for_layers([1, 2], "r1", summ)
    assert t is None and "another routine" in why
    t, why = b.traffic_for_layers([1, 4], "r1", summ)
    assert t is None
    # changed kernel sources make the figure stale
    monkeypatch.setattr(b, "kernel_source_hash", lambda ksub=None: "different")
    t, why = b.traffic_for_layers([1, 3], "r1", summ)
    assert t is None and "changed" in why


def test_summarize_trace_averages_timed_steps_per_layer(tmp_path):
    import json
    b = load_bench()
    ka, kb = "_ZN2sn1k12dw3x3_kernelIDF16bLi2ELi1ELi4EEEvNS0_7Dw3ArgsE", "void sn::k::gap_kernel<x>(y)"
    info = {"workload": "w", "warmup": 1, "steps": 2, "routines": ["input/nchw", "r1", "r2"],
            "launch_layers": [1, 2, 2], "bytes_needed": {"1": 3000, "2": 8000}}
    (tmp_path / "pass.json").write_text(json.dumps(info))
    d = tmp_path / "t"
    d.mkdir()
    fields = ["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"]
    with open(d / "x_kernel_trace.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=fields)
        w.writeheader()
        rows = [("__amd_rocclr_fillBuffer", 5)]
        for dur in ([100, 100, 100], [10, 20, 30], [30, 40, 50]):   # warm-up step, two timed steps
            rows += [(ka, dur[0]), (kb, dur[1]), (kb, dur[2])]
        t = 1000
        for k, (name, dur) in enumerate(rows):
            w.writerow({"Dispatch_Id": k + 1, "Kernel_Name": name, "Start_Timestamp": t, "End_Timestamp": t + dur})
            t += dur + 7
    out = tmp_path / "o.json"
    b.summarize_trace(str(d), str(tmp_path / "pass.json"), str(out))
    res = json.loads(out.read_text())
    by = {e["layer"]: e for e in res["layers"]}
    assert by[1]["us"] == 0.02 and by[1]["gbs"] == 150.0          # (10 + 30) / 2 ns, 3000 B
    assert by[2]["kernel_ns"] == [30.0, 40.0] and by[2]["gbs"] == round(8000 / 70, 1)
    assert res["step_kernel_us"] == 0.09


def test_strided_pointwise_layers_count_the_pixels_they_read():
    b = load_bench()
    from paper_2110_06037_amd import build_from_spec
    from workloads import fuse_residual, resnet50
    spec = fuse_residual(resnet50(2, "bf16"))
    g = build_from_spec(spec, device=-1)
    rt = {"algo": 1}
    seen = 0
    for i, L in enumerate(spec["layers"], start=1):
        _, _, full = b.layer_work(spec, g, i, rt)
        need = b.bytes_needed(spec, g, i, rt)
        if L["type"] == "conv" and L["r"] == 1 and L["stride"] == 2:
            n, c, h, w = g.layer_shape(L["in"][0])
            _, _, p, q = g.layer_shape(i)
            assert full - need == 2 * n * c * (h * w - p * q) and need < full
            seen += 1
        else:
            assert need == full
    assert seen == 3   # the stride-2 projections of stages 2-4
    g.close()


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
