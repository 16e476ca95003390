"""Host-side pieces of bench.py: the algorithmic byte model and the selection
of the timed dispatches from a kernel trace (no GPU)."""
import csv
import os

import pytest

import bench


def test_byte_model_per_parameter():
    """Each kernel's bytes per launch are its arrays' reads and writes, plus
    packed words (d/8 bytes) and one binary32 scale per chunk."""
    d, nch, nw, W = 1 << 20, 256, (1 << 20) // 64, 128
    pk, sc = 8 * nw, 4 * nch
    deferred = bench.algorithmic_bytes(d, nch, nw, W, deferred=True, gbytes=4)
    assert deferred["local+var"] == 28 * d + pk + sc       # g, gbar, anchor, v; m, x, v
    assert deferred["sync1"] == 16 * d + pk + sc           # g, m, err; err
    assert deferred["srv"] == W * (pk + sc) + 8 * d + pk + sc
    assert deferred["recon+var"] == 2 * (pk + sc) + 20 * d  # anchor, v, gbar; anchor, v
    eager = bench.algorithmic_bytes(d, nch, nw, W, deferred=False, gbytes=4)
    assert eager["local+var"] == 40 * d
    assert eager["sync1"] == 20 * d + pk + sc
    assert eager["recon+var"] == pk + sc + 32 * d
    half = bench.algorithmic_bytes(d, nch, nw, W, deferred=True, gbytes=2)
    assert deferred["local+var"] - half["local+var"] == 4 * d  # g and gbar in 16 bits
    fv = bench.algorithmic_bytes_fv(d, nch, nw, W, 4)
    assert fv["fv_full"] == 28 * d and fv["fv_apply"] == 20 * d + pk + sc


def test_gpt2_bytes_per_launch():
    """The GPT-2-1.5B shard's per-launch figures quoted with the benchmark."""
    import paper_2202_06009_amd as zo
    from synth import configs as C
    wl = C.get("gpt2-1.5b")
    _, ln, _, nw = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    b = bench.algorithmic_bytes(wl.n, len(ln), nw, wl.world, deferred=True)
    assert round(b["local+var"] / 1e9, 3) == 43.808
    assert round(b["sync1"] / 1e9, 3) == 25.117
    assert round(b["srv"] / 1e9, 3) == 37.627
    assert round(b["recon+var"] / 1e9, 3) == 31.542


def _write_trace(path, launches):
    cols = ["Kind", "Kernel_Name", "Start_Timestamp", "End_Timestamp"]
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=cols)
        w.writeheader()
        for name, start, dur in launches:
            w.writerow({"Kind": "KERNEL_DISPATCH", "Kernel_Name": f"void {name}(int)",
                        "Start_Timestamp": start, "End_Timestamp": start + dur})


def test_trace_summary_keeps_the_timed_dispatches(tmp_path, capsys):
    """Two warmup and three timed bench steps, then later launches of the same
    kernels at other sizes: only dispatches 2..4 of each slot count, whatever
    the template variant."""
    launches, t = [], 0
    for step in range(5):
        for name, dur in ((("zo::k_local<true, 0, true, 0>" if step == 0 else
                            "zo::k_local<true, 1, false, 0>"), 7000),
                          ("zo::k_sync1<1024, 4, true, 2, 0>", 4000),
                          ("zo::k_srv_lut<512, 16>", 7500 + 10 * step),
                          ("zo::k_recon<true, true, 0>", 5000)):
            launches.append((name, t, 1000 * dur))
            t += 10 ** 7
    for _ in range(4):  # the server share: the same kernels, much shorter
        for name in ("zo::k_sync1<1024, 4, true, 2, 0>", "zo::k_srv_lut<512, 16>",
                     "zo::k_recon<true, true, 0>"):
            launches.append((name, t, 1000 * 80))
            t += 10 ** 6
    _write_trace(os.path.join(tmp_path, "run_kernel_trace.csv"), launches)
    bench.summarize_trace(str(tmp_path), "deferred", "tiny", warmup=2, steps=3)
    out = capsys.readouterr().out
    rows = {line.split("(")[1].split(")")[0]: line for line in out.splitlines()
            if line.startswith("| `")}
    assert set(rows) == {"local+var", "sync1", "srv", "recon+var"}
    for key, avg in (("local+var", 7000.0), ("sync1", 4000.0), ("srv", 7530.0),
                     ("recon+var", 5000.0)):
        cells = [c.strip() for c in rows[key].split("|")]
        assert cells[2] == "3", key           # calls
        assert float(cells[3]) == pytest.approx(avg), key
    assert "k_local<true, 0, true, 0>" not in out  # the first, pre-sync variant is warmup


def test_traffic_summary_only_for_its_workload_and_source(tmp_path, monkeypatch):
    """The measured traffic is reported only for the workload, mode and kernel
    source the counters were taken on."""
    import json
    f = tmp_path / "traffic.json"
    f.write_text(json.dumps({"source_sha256": bench.source_hash(), "mode": "deferred",
                             "workload": "gpt2-1.5b",
                             "kernels": {"local+var": {"traffic_bytes": 1.0}}}))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(f))
    assert bench.measured_traffic("local+var", "deferred", "gpt2-1.5b") == 1.0
    assert bench.measured_traffic("local+var", "deferred", "bert-base") is None
    assert bench.measured_traffic("local+var", "eager", "gpt2-1.5b") is None
    assert bench.measured_traffic("srv", "deferred", "gpt2-1.5b") is None
    f.write_text(json.dumps({"source_sha256": "0" * 64, "mode": "deferred",
                             "workload": "gpt2-1.5b",
                             "kernels": {"local+var": {"traffic_bytes": 1.0}}}))
    assert bench.measured_traffic("local+var", "deferred", "gpt2-1.5b") is None


def test_variant_byte_model():
    """Bytes of the kernel variants of the schedule: the general forms are the
    whole-state figures (local 32, local+var 40, compress 20 + words, eager
    reconstruction 24 + words, 32 with the variance line)."""
    d, nch, nw, W = 1 << 20, 256, (1 << 20) // 64, 64
    cp = 8 * nw + 4 * nch
    vb = lambda name, gb=4: bench.variant_bytes(name, d, nch, nw, W, gb)
    assert vb("local") == 32 * d and vb("local+var") == 40 * d
    assert vb("sync1") == 20 * d + cp and vb("recon") == 24 * d + cp
    assert vb("recon+var") == 32 * d + cp
    assert vb("local (u=0)") == 20 * d + cp and vb("local (u=gm)") == 28 * d
    assert vb("sync1 (u=0)") == 12 * d + 2 * cp and vb("sync1 (u=gm)") == 16 * d + cp
    assert vb("recon (deferred)+var") == 20 * d + 2 * cp
    assert vb("local", 2) == 30 * d and vb("local+var", 2) == 36 * d
    for name in bench.VARIANT_KERNELS:
        assert vb(name) > 0


def test_kernel_names_map_to_variants():
    """Template names from a kernel trace map back to the byte model's variants."""
    for name, tmpl in bench.VARIANT_KERNELS.items():
        for var in ((False, True) if name != "srv" and not name.startswith("sync1") else (False,)):
            for gt, gb in ((0, 4), (2, 2)):
                k = "zo::" + tmpl.format(var="true" if var else "false", gt=gt)
                k = k.replace("L, V", "1024, 4").replace("LD, G", "512, 16")
                assert bench.variant_of_kernel(k) == (name + ("+var" if var else ""),
                                                      4 if name == "srv" else gb), k
    assert bench.variant_of_kernel("zo::k_copy<true>") is None


def test_counter_summary_ratios(tmp_path, capsys):
    """The counter summary averages each counter per dispatch for the step's
    kernels and the reference kernels, and forms the unit-free ratios: reads
    in flight per channel and read latency from the request-level sums."""
    cols = ["Kernel_Name", "Counter_Name", "Counter_Value"]
    rows = []
    for rep in range(2):  # two dispatches of each kernel: the mean is taken
        for name, level, req, cyc in (("zo::k_local<true, 1, false, 0>", 600.0, 2.0, 3.0),
                                      ("zo::k_copy<true>", 100.0 + 20 * rep, 0.5, 1.0),
                                      ("zo::k_stream<4, 3>", 300.0, 1.0, 1.5)):
            rows += [(f"void {name}(int)", "TCC_EA0_RDREQ_LEVEL", level),
                     (f"void {name}(int)", "TCC_EA0_RDREQ", req),
                     (f"void {name}(int)", "TCC_CYCLE", cyc)]
    d = tmp_path / "pmc"
    d.mkdir()
    with open(d / "run_counter_collection.csv", "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(cols)
        w.writerows(rows)
    bench.summarize_counters([str(d)], "deferred")
    out = capsys.readouterr().out.splitlines()
    assert out[0] == "| counter | local+var | copy | 4r+3w |"
    table = {line.split("|")[1].strip(): [c.strip() for c in line.split("|")[2:-1]]
             for line in out[2:]}
    assert table["TCC_EA0_RDREQ_LEVEL"] == ["600", "110", "300"]
    assert table["memory read latency (L2 cycles)"] == ["300", "220", "300"]
    assert table["memory reads in flight per L2 channel"] == ["200", "110", "200"]
    # rows whose counters were not taken are left out
    assert "L2 cycles with a request pending" not in table
    assert "LDS instructions per wave" not in table
