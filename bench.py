"""Benchmark of the 0/1 Adam hot path on one MI355X.

Workload: the GPT-2-1.5B-shaped shard (d = 1,557,611,200 binary32 params in
580 segments, chunk 16384, W = 128 workers whose packed sign buffers sit in
HBM, the single server over the whole shard).  One bench step is two
optimizer steps that together run every kernel of the path once:
  step 2k   (local, variance update):  K_local+var         (zo_local_step)
  step 2k+1 (sync, variance update):   K_sync1             (zo_compress_pack_ef)
                                       K_srv, W = 128      (zo_unpack_average)
                                       K_recon+var         (zo_sync_update)
The reconstruction defers its x and u writes (the new model stays in the
anchor buffer, u is an implicit zero and m is rebuilt from a 1-bit copy of
the server output; the next local step writes x and m but leaves u = +0 +
gamma m implicit, which the compress forms from the m it reads; same values,
28 bytes per parameter less per bench step); --eager-sync-writes times the
eager variant.
Inputs (gradient, averaged gradient, peers' packed signs and scales) are
generated once on the device before timing and stay resident in HBM.
`value` is optimizer-step parameter updates per second (2 d per bench step).

Per-kernel durations come from HIP events recorded on the stream the kernels
run on; the dominant kernel's algorithmic bytes per launch over its average
duration gives the roofline line.  The CPU baseline times the oracle on a
bounded contiguous slice of the same shard (rank 0, N = 1 only).
"""
import argparse
import csv
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# the device code of the library: the traffic summary is valid for these sources only
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2202_06009_amd", "csrc", f)
                  for f in ("zo_device.h", "zo_kernels.hip", "zo_server.hip", "zo_kernels_ua.hip")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gpt2-1.5b_hbm_traffic.json")
COPY_BYTES = 4 << 30          # size of the calibration copies
# kernel-name prefixes in rocprofv3 output -> bench names; every hot kernel
# uses one kind of access (nontemporal or plain), calibrated by the matching copy.
# The second template argument of k_local / k_recon is the deferred variant
# (the very first local step of a run has no sync before it and is skipped).
def kernel_keys(mode):
    """Regular expressions for the names of the timed kernels in a mode
    ("deferred", "eager" or "frozen-variance", with "/f16" or "/bf16" for
    16-bit gradients) -> (bench name, access kind).  The last template
    argument of the gradient-reading kernels is the gradient type (0 binary32,
    1 binary16, 2 bfloat16); the steady-state variants only (the first local
    step and compress of a run, before any sync, are other instantiations)."""
    copies = {r"zo::k_copy<true>": ("copy_nt", None), r"zo::k_copy<false>": ("copy_plain", None)}
    base, _, dt = mode.partition("/")
    gt = {"": 0, "f16": 1, "bf16": 2}[dt]
    if base == "frozen-variance":
        return {rf"zo::k_fv_full<{gt}>": ("fv_full", "nt"),
                rf"zo::k_sync1<\d+, \d+, false, 0, {gt}>": ("sync1", "nt"),
                r"zo::k_srv_lut<": ("srv", "plain"), r"zo::k_fv_apply": ("fv_apply", "nt")} | copies
    dv = "true" if base == "deferred" else "false"
    # k_local<VAR, UIN, WU, GT>: deferred, the local step after a sync has
    # UIN = 1 (u = +0) and WU = false, and the compress after it UIN = 2
    # (u = +0 + gamma m); eager UIN = 0 throughout
    lv = f"true, 1, false, {gt}" if base == "deferred" else f"true, 0, true, {gt}"
    su = 2 if base == "deferred" else 0
    return {rf"zo::k_local<{lv}>": ("local+var", "nt"),
            rf"zo::k_sync1<\d+, \d+, true, {su}, {gt}>": ("sync1", "nt"),
            r"zo::k_srv_lut<": ("srv", "plain"),
            rf"zo::k_recon<true, {dv}, {gt}>": ("recon+var", "nt")} | copies


def device_clocks(dev=0):
    """Peak shader and memory clocks in MHz as the HIP runtime reports them
    (hipDeviceGetAttribute: hipDeviceAttributeClockRate = 5 and
    hipDeviceAttributeMemoryClockRate = 60, in kHz), or {} when unavailable."""
    import ctypes
    try:
        hip = ctypes.CDLL("libamdhip64.so")
    except OSError:
        return {}
    out = {}
    for key, attr in (("sclk_mhz", 5), ("mclk_mhz", 60)):
        v = ctypes.c_int(0)
        if hip.hipDeviceGetAttribute(ctypes.byref(v), ctypes.c_int(attr), ctypes.c_int(dev)) == 0:
            out[key] = v.value / 1000.0
    return out


def source_hash():
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


# Reference kernels of a counter run (--copy-calibration): the calibration
# copy and the stream mixes, plain streams of R read and S write arrays.
REFERENCE_KERNELS = {r"zo::k_copy<true>": "copy", r"zo::k_stream<1, 1>": "1r+1w",
                     r"zo::k_stream<3, 1>": "3r+1w", r"zo::k_stream<3, 2>": "3r+2w",
                     r"zo::k_stream<4, 3>": "4r+3w"}


def summarize_counters(dirs, mode):
    """Mean per dispatch of every counter in the rocprofv3 --pmc runs under
    `dirs`, for each timed kernel of `mode` and each reference kernel present,
    as a markdown table, with the ratios that need no unit: instructions per
    wave, the share of the LDS's active cycles lost to bank conflicts, the
    average latency of the L2's memory requests (requests in flight summed
    over cycles, over requests) and the share of L2 cycles stalled for
    memory credits."""
    keys = {p: k for p, (k, kind) in kernel_keys(mode).items() if kind is not None}
    keys.update(REFERENCE_KERNELS)
    vals = {}
    for d in dirs:
        for root, _, files in os.walk(d):
            for fn in files:
                if not fn.endswith("counter_collection.csv"):
                    continue
                for r in csv.DictReader(open(os.path.join(root, fn))):
                    name = r["Kernel_Name"].replace("void ", "")
                    for pattern, key in keys.items():
                        if re.match(pattern, name):
                            vals.setdefault(key, {}).setdefault(r["Counter_Name"], []).append(
                                float(r["Counter_Value"]))
    names = [k for k in keys.values() if k in vals]
    mean = {k: {c: sum(v) / len(v) for c, v in vals[k].items()} for k in names}
    counters = sorted({c for k in names for c in mean[k]})
    print("| counter | " + " | ".join(names) + " |")
    print("|---|" + "---|" * len(names))
    for c in counters:
        print(f"| {c} | " + " | ".join(f"{mean[k].get(c, float('nan')):.4g}" for k in names) + " |")
    def ratio(k, a, b):
        m = mean[k]
        return f"{m[a] / m[b]:.3g}" if a in m and b in m and m[b] else "-"
    for label, a, b in (("VALU instructions per wave", "SQ_INSTS_VALU", "SQ_WAVES"),
                        ("LDS instructions per wave", "SQ_INSTS_LDS", "SQ_WAVES"),
                        ("SALU instructions per wave", "SQ_INSTS_SALU", "SQ_WAVES"),
                        ("vector memory reads per wave", "SQ_INSTS_VMEM_RD", "SQ_WAVES"),
                        ("LDS bank-conflict cycles / LDS active cycles", "SQ_LDS_BANK_CONFLICT",
                         "SQ_LDS_IDX_ACTIVE"),
                        ("memory reads in flight per L2 channel", "TCC_EA0_RDREQ_LEVEL",
                         "TCC_CYCLE"),
                        ("memory writes in flight per L2 channel", "TCC_EA0_WRREQ_LEVEL",
                         "TCC_CYCLE"),
                        ("memory read latency (L2 cycles)", "TCC_EA0_RDREQ_LEVEL", "TCC_EA0_RDREQ"),
                        ("memory write latency (L2 cycles)", "TCC_EA0_WRREQ_LEVEL",
                         "TCC_EA0_WRREQ"),
                        ("L2 cycles with a read stalled for DRAM credits",
                         "TCC_EA0_RDREQ_DRAM_CREDIT_STALL", "TCC_CYCLE"),
                        ("L2 cycles with a write stalled for DRAM credits",
                         "TCC_EA0_WRREQ_DRAM_CREDIT_STALL", "TCC_CYCLE"),
                        ("L2 cycles with a write request stalled", "TCC_EA0_WRREQ_STALL",
                         "TCC_CYCLE"),
                        ("L2 cycles with a request pending", "TCC_BUSY", "TCC_CYCLE")):
        row = [ratio(k, a, b) for k in names]
        if any(r != "-" for r in row):
            print(f"| {label} | " + " | ".join(row) + " |")


def trace_rows(trace_dir):
    """Kernel dispatches of a rocprofv3 --kernel-trace run under `trace_dir`,
    from its CSV files or its SQLite results database (the `kernels` view), as
    dicts with Kernel_Name, Start_Timestamp, End_Timestamp (ns) and
    Grid_Size_X."""
    rows = []
    for root, _, files in os.walk(trace_dir):
        for fn in sorted(files):
            path = os.path.join(root, fn)
            if fn.endswith("kernel_trace.csv"):
                rows += list(csv.DictReader(open(path)))
            elif fn.endswith("_results.db"):
                import sqlite3
                con = sqlite3.connect(path)
                try:
                    for name, start, end, grid in con.execute(
                            "select name, start, end, grid_x from kernels"):
                        rows.append({"Kernel_Name": name, "Start_Timestamp": start,
                                     "End_Timestamp": end, "Grid_Size_X": grid})
                finally:
                    con.close()
    return rows


def summarize_trace(trace_dir, mode, workload, warmup, steps):
    """Per-kernel durations of a `rocprofv3 --kernel-trace` run of this bench
    (the default command: `warmup` + `steps` bench steps) over the timed
    dispatches only: for each of the step's four kernel slots (all template
    variants of the slot's kernel, in launch order), dispatches warmup ..
    warmup + steps - 1.  Later launches of the same kernels (the server share
    and the schedule run after the timed region) are left out.  Prints a
    markdown table with the algorithmic bytes of the workload."""
    import statistics
    import paper_2202_06009_amd as zo
    from synth import configs as C
    base, _, dt = mode.partition("/")
    fv = base == "frozen-variance"
    slots = ([("fv_full", r"zo::k_fv_full<"), ("sync1", r"zo::k_sync1<"),
              ("srv", r"zo::k_srv_(lut|plain)<"), ("fv_apply", r"zo::k_fv_apply")] if fv else
             [("local+var", r"zo::k_local<"), ("sync1", r"zo::k_sync1<"),
              ("srv", r"zo::k_srv_(lut|plain)<"), ("recon+var", r"zo::k_recon<")])
    rows = trace_rows(trace_dir)
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    wl = C.get(workload)
    _, ln, _, nwords = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    gbytes = {"": 4, "f16": 2, "bf16": 2}[dt]
    model = algorithmic_bytes_fv(wl.n, len(ln), nwords, wl.world, gbytes) if fv else \
        algorithmic_bytes(wl.n, len(ln), nwords, wl.world, deferred=base == "deferred",
                          gbytes=gbytes)
    print("| kernel | calls | avg µs | median µs | min µs | max µs | algorithmic GB/launch "
          "| GB/s | % of 8 TB/s |")
    print("|---|---|---|---|---|---|---|---|---|")
    for key, pat in slots:
        ds = [r for r in rows if re.match(pat, r["Kernel_Name"].replace("void ", ""))]
        ds = ds[warmup:warmup + steps]
        us = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0 for r in ds]
        names = sorted({r["Kernel_Name"].replace("void ", "").split("(")[0] for r in ds})
        avg = sum(us) / len(us)
        gbs = model[key] / 1e9 / (avg / 1e6)
        print(f"| `{', '.join(names)}` ({key}) | {len(us)} | {avg:.1f} | "
              f"{statistics.median(us):.1f} | {min(us):.1f} | {max(us):.1f} | "
              f"{model[key] / 1e9:.3f} | {gbs:.0f} | {100 * gbs / HBM_PEAK_GBS:.1f} |")


def variant_of_kernel(name):
    """(variant, bytes per gradient element) of an Algorithm 1 kernel's
    template name, or None: the inverse of VARIANT_KERNELS."""
    m = re.match(r"zo::k_local<(true|false), (\d), (true|false), (\d)>", name)
    if m:
        base = {"0": "local", "1": "local (u=0)", "2": "local (u=gm)"}[m.group(2)]
        return base + ("+var" if m.group(1) == "true" else ""), (4, 2, 2)[int(m.group(4))]
    m = re.match(r"zo::k_sync1<\d+, \d+, true, (\d), (\d)>", name)
    if m:
        base = {"0": "sync1", "1": "sync1 (u=0)", "2": "sync1 (u=gm)"}[m.group(1)]
        return base, (4, 2, 2)[int(m.group(2))]
    if re.match(r"zo::k_srv_(lut|plain)<", name):
        return "srv", 4
    m = re.match(r"zo::k_recon<(true|false), (true|false), (\d)>", name)
    if m:
        base = "recon (deferred)" if m.group(2) == "true" else "recon"
        return base + ("+var" if m.group(1) == "true" else ""), (4, 2, 2)[int(m.group(3))]
    return None


def summarize_kernels(trace_dir, workload):
    """Every kernel of a `rocprofv3 --kernel-trace` run grouped by template
    name and grid size, with the algorithmic bytes of the Algorithm 1 variants
    at their largest grid for the name (the whole shard of `workload`; smaller
    grids are other sizes, e.g. the server share).  Prints a markdown table."""
    import statistics
    import paper_2202_06009_amd as zo
    from synth import configs as C
    rows = trace_rows(trace_dir)
    wl = C.get(workload)
    _, ln, _, nwords = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    groups = {}
    for r in rows:
        name = r["Kernel_Name"].replace("void ", "").split("(")[0]
        grid = int(r.get("Grid_Size_X") or r.get("Grid_Size") or 0)
        us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0
        groups.setdefault((name, grid), []).append(us)
    biggest = {}
    for name, grid in groups:
        biggest[name] = max(grid, biggest.get(name, 0))
    print("| kernel | grid | calls | avg µs | median µs | variant | algorithmic GB/launch "
          "| GB/s | % of 8 TB/s |")
    print("|---|---|---|---|---|---|---|---|---|")
    for (name, grid), us in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        avg = sum(us) / len(us)
        v = variant_of_kernel(name)
        cols = ["", "", "", ""]
        if v is not None and grid == biggest[name]:
            nb = variant_bytes(v[0], wl.n, len(ln), nwords, wl.world, v[1])
            gbs = nb / 1e9 / (avg / 1e6)
            cols = [v[0], f"{nb / 1e9:.3f}", f"{gbs:.0f}", f"{100 * gbs / HBM_PEAK_GBS:.1f}"]
        print(f"| `{name}` | {grid} | {len(us)} | {avg:.1f} | {statistics.median(us):.1f} | "
              + " | ".join(cols) + " |")


def summarize_pmc(fetch_dir, write_dir, out_path, mode, workload):
    """Turn two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE) over
    `bench.py --copy-calibration` into per-launch HBM traffic, each counter
    scaled by what it reads for the calibration copy of COPY_BYTES.
    `mode` names what the runs timed: "deferred" or "eager" sync writes of
    Algorithm 1, or "frozen-variance" (Algorithm 4)."""
    keys = kernel_keys(mode)
    def load(d, counter):
        vals = {}
        for root, _, files in os.walk(d):
            for fn in files:
                if not fn.endswith("counter_collection.csv"):
                    continue
                for r in csv.DictReader(open(os.path.join(root, fn))):
                    if r["Counter_Name"] != counter:
                        continue
                    name = r["Kernel_Name"].replace("void ", "")
                    for pattern, (key, _) in keys.items():
                        if re.match(pattern, name):
                            vals.setdefault(key, []).append(float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in vals.items()}
    fetch, write = load(fetch_dir, "FETCH_SIZE"), load(write_dir, "WRITE_SIZE")
    factors = {kind: {"fetch": COPY_BYTES / (1024.0 * fetch[f"copy_{kind}"]),
                      "write": COPY_BYTES / (1024.0 * write[f"copy_{kind}"])}
               for kind in ("nt", "plain")}
    kernels = {}
    for prefix, (key, kind) in keys.items():
        if kind is None or key not in fetch or key not in write:
            continue
        f, w = factors[kind]["fetch"], factors[kind]["write"]
        kernels[key] = {"fetch_kib": fetch[key], "write_kib": write[key], "access": kind,
                        "traffic_bytes": 1024.0 * (fetch[key] * f + write[key] * w)}
    out = {"source_sha256": source_hash(), "mode": mode, "workload": workload,
           "copy_bytes": COPY_BYTES,
           "copy_kib": {k: {"fetch": fetch[f"copy_{k}"], "write": write[f"copy_{k}"]}
                        for k in ("nt", "plain")},
           "factors": factors, "kernels": kernels}
    with open(out_path, "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps(out, indent=1))


def measured_traffic(kernel, mode, workload):
    """HBM bytes per launch from the committed counter summary, or None when
    it is missing or was taken on different kernel source, in another mode or
    on another workload."""
    try:
        with open(TRAFFIC_FILE) as fh:
            t = json.load(fh)
    except (OSError, ValueError):
        return None
    if (t.get("source_sha256") != source_hash() or t.get("mode") != mode
            or t.get("workload") != workload):
        return None
    if kernel not in t.get("kernels", {}):
        return None
    return t["kernels"][kernel]["traffic_bytes"]


def algorithmic_bytes_fv(d, nchunks, nwords, W, gbytes=4):
    """Algorithm 4: bytes each kernel must move per launch (gbytes: bytes per
    gradient element)."""
    pk = 8 * nwords
    sc = 4 * nchunks
    return {
        # reads gbar, x, m, v; writes x, m, v
        "fv_full": (24 + gbytes) * d,
        # reads g, err; writes err, own packed words, own scales
        "sync1": (8 + gbytes) * d + pk + sc,
        "srv": W * (pk + sc) + 8 * d + pk + sc,
        # reads server words + scales, x, m, v; writes x, m
        "fv_apply": pk + sc + 20 * d,
    }


# Kernel variants of Algorithm 1 (zo_local_step, zo_compress_pack_ef,
# zo_unpack_average, zo_sync_update) by where u is before the call, and the
# kernel template each launches (GT = gradient type).  "(u=0)": the first call
# after a deferred sync (u = +0, m from the 1-bit copy of the server output);
# "(u=gm)": u = +0 + gamma m left implicit by that first local step.
VARIANT_KERNELS = {
    "local": "k_local<{var}, 0, true, {gt}>",
    "local (u=0)": "k_local<{var}, 1, false, {gt}>",
    "local (u=gm)": "k_local<{var}, 2, true, {gt}>",
    "sync1": "k_sync1<L, V, true, 0, {gt}>",
    "sync1 (u=0)": "k_sync1<L, V, true, 1, {gt}>",
    "sync1 (u=gm)": "k_sync1<L, V, true, 2, {gt}>",
    "srv": "k_srv_lut<LD, G>",
    "recon": "k_recon<{var}, false, {gt}>",
    "recon (deferred)": "k_recon<{var}, true, {gt}>",
}


def variant_bytes(name, d, nchunks, nwords, W, gbytes=4):
    """Algorithmic bytes per launch of a kernel variant of Algorithm 1: every
    array it must read and write once, packed words (8 per word) and one
    binary32 scale per chunk included; a name ending in "+var" has the
    variance line fused (gbar read, v written).  gbytes: bytes per element of
    g and gbar."""
    cp = 8 * nwords + 4 * nchunks          # one packed buffer: words and scales
    var = name.endswith("+var")
    base = name[:-4] if var else name
    table = {
        # reads g, m, x, v, u; writes m, x, u
        "local": (28 + gbytes) * d,
        # reads g, the server copy, the anchor, v; writes m, x
        "local (u=0)": (16 + gbytes) * d + cp,
        # reads g, m, x, v; writes m, x, u
        "local (u=gm)": (24 + gbytes) * d,
        # reads g, m, u, err; writes err, own words and scales
        "sync1": (16 + gbytes) * d + cp,
        # reads g, m, err; writes err, own words and scales
        "sync1 (u=gm)": (12 + gbytes) * d + cp,
        # reads g, the server copy, err; writes err, own words and scales
        "sync1 (u=0)": (8 + gbytes) * d + 2 * cp,
        # reads W packed buffers and the server error; writes the server error
        # and the server words and scales
        "srv": W * cp + 8 * d + cp,
        # reads server words and scales, v, anchor; writes m, x, anchor, u
        "recon": 24 * d + cp,
        # reads server words and scales, v, anchor; writes anchor and the copy
        "recon (deferred)": 12 * d + 2 * cp,
    }
    return table[base] + ((gbytes + 4) * d if var else 0)


def algorithmic_bytes(d, nchunks, nwords, W, deferred=True, gbytes=4):
    """Bytes each kernel must move per launch: every state read once and
    written once, packed words and per-chunk scales included (gbytes: bytes
    per gradient element of g and gbar).  With deferred sync writes the
    reconstruction writes neither x, m nor u but copies the server's packed
    words and scales; the local step after it reads x from the anchor and m
    from that copy, and neither reads nor writes u (u = +0 + gamma m there);
    the compress that follows forms u from the m it reads."""
    v = {"local+var": "local (u=0)+var" if deferred else "local+var",
         "sync1": "sync1 (u=gm)" if deferred else "sync1",
         "srv": "srv",
         "recon+var": "recon (deferred)+var" if deferred else "recon+var"}
    return {k: variant_bytes(name, d, nchunks, nwords, W, gbytes) for k, name in v.items()}


def placement_study(zo, torch, d, reps=5):
    """The plain stream kernel (zo_diag_stream) over the general local step's
    arrays (reads g, m, x, v, u; rewrites m, x, u in place: 32 B/param) of
    length d, timed (best of `reps` launches after one untimed) with the five
    arrays placed in different ways: five separate allocations; one
    allocation holding them back to back or 4 KiB or 2 MiB + 4 KiB apart; five
    separate allocations after 48 GB of other allocations, or followed by
    them.  Every layout's memory is returned to the driver before the next."""
    gbytes = 32.0 * d / 1e9
    f32 = dict(dtype=torch.float32, device="cuda")
    dummy_n = 12 * 10 ** 9  # 48 GB of binary32

    def timed(arrs):
        g, m, x, v, u = arrs
        best = None
        for r in range(reps + 1):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            zo.zo_diag_stream([g, m, x, v, u], [m, x, u])
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            if r and (best is None or ms < best):
                best = ms
        return {"ms": round(best, 4), "gbs": round(gbytes / (best / 1000.0), 1),
                "frac": round(gbytes / (best / 1000.0) / HBM_PEAK_GBS, 4)}

    def separate():
        return [torch.zeros(d, **f32) for _ in range(5)]

    def slab(pad):
        buf = torch.zeros(5 * (d + pad), **f32)
        return [buf[i * (d + pad):i * (d + pad) + d] for i in range(5)]

    out = {}
    layouts = (("separate", lambda: (separate(), None)),
               ("one allocation, back to back", lambda: (slab(0), None)),
               ("one allocation, 4 KiB apart", lambda: (slab(1024), None)),
               ("one allocation, 2 MiB + 4 KiB apart", lambda: (slab((2 << 20) // 4 + 1024), None)),
               ("separate, after 48 GB of other allocations",
                lambda: (lambda dm: (separate(), dm))(torch.empty(dummy_n, **f32))),
               ("separate, followed by 48 GB of other allocations",
                lambda: (lambda a: (a, torch.empty(dummy_n, **f32)))(separate())),
               ("separate, again", lambda: (separate(), None)))
    for name, make in layouts:
        arrs, dummy = make()
        out[name] = timed(arrs)
        print(f"[bench] placement: {name}: {out[name]}", file=sys.stderr, flush=True)
        del arrs, dummy
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    return out


def stream_mix_ceilings(zo, torch, state, g, gb, d, mode):
    """HBM rate of a plain streaming kernel (zo_diag_stream) with each hot
    kernel's mix of full-length arrays, on the bench's own buffers (used as
    scratch after the timed region): the rate such a mix can reach on this
    GPU.  An array the kernel reads and rewrites (v, the error buffers, the
    anchor) is a source and a destination of the mix, so it is updated in
    place as in the kernel; the other arrays are read-only or write-only.  The
    server's row-strided packed reads have no such plain mix."""
    S = state
    deferred = mode == "deferred"
    x, m, v, u, err, anchor = (S[k] for k in ("x", "m", "v", "u", "err", "anchor"))
    mixes = {
        # reads gbar, x, m, v; rewrites x, m, v
        "fv_full": ([gb, x, m, v], [x, m, v]),
        # reads g, err; rewrites err
        "sync1": ([g, err], [err]),
        # reads x, m, v; rewrites x, m
        "fv_apply": ([x, m, v], [x, m]),
    } if mode == "frozen-variance" else {
        # deferred: reads g, gbar, the anchor, v; writes m and x, rewrites v.
        # eager: reads g, gbar, x, v, m, u; rewrites all four states
        "local+var": ([g, gb, anchor, v], [m, x, v]) if deferred else
                     ([g, gb, x, v, m, u], [x, v, m, u]),
        # reads g, m, err (and u, eager); rewrites err
        "sync1": ([g, m, err] + ([] if deferred else [u]), [err]),
        # reads v, the anchor, gbar; rewrites the anchor and v (and writes m,
        # x, u, eager)
        "recon+var": ([v, anchor, gb], [anchor, v] + ([] if deferred else [m, x, u])),
    }
    out = {}
    for name, (src, dst) in mixes.items():
        best = None
        for rep in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            zo.zo_diag_stream(src, dst)
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1)
            if rep and (best is None or ms < best):
                best = ms
        gbs = (len(src) + len(dst)) * 4.0 * d / 1e9 / (best / 1000.0)
        in_place = sum(1 for t in dst if any(t is s for s in src))
        out[name] = {"reads": len(src), "writes": len(dst), "in_place": in_place,
                     "gbs": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}
    return out


def graph_replay(zo, torch, wl, state, g_in, gb_in, packed, scales, srv_packed, srv_scales,
                 deferred, grad_dtype, replays):
    """The bench step (local+variance, then sync+variance) recorded once in a
    HIP graph after one eager step pair, then replayed `replays` times: the
    step's time without host launch overhead.  Each replay repeats the
    recorded step (constant learning rate, the same inputs), as the timed
    region does."""
    d = wl.n
    T = 4
    opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=wl.world, chunk=wl.chunk,
                    seg_off=wl.seg_off, tv=list(range(T)), tu=list(range(1, T, 2)),
                    state=state, defer_sync_writes=deferred, grad_dtype=grad_dtype)
    gamma = 1e-4

    def pair(t):
        opt.local_step(t, gamma, g_in, gb_in)
        opt.compress_pack_ef(t + 1, gamma, g_in, packed[0], scales[0])
        opt.unpack_average(t + 1, packed, scales, srv_packed, srv_scales)
        opt.sync_update(t + 1, srv_packed, srv_scales, gb_in)

    pair(0)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        opt.set_stream(None)  # the capture stream
        pair(2)
    opt.set_stream(None)
    graph.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(replays):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / replays
    opt.close()
    del graph
    return {"replays": replays, "ms_per_step": round(ms, 4),
            "params_per_s": round(2.0 * d / (ms / 1000.0), 1)}


def server_pattern(zo, torch, wl, state, packed, W, nwords, reps=4):
    """The server's access pattern without its arithmetic (zo_diag_server_pattern
    on a handle over the whole shard, best of the last reps-1 launches): the
    rate the single server's reads of W packed rows and read-modify-write of
    its error can reach.  None for chunks of at most 1024 elements."""
    if wl.chunk <= 1024:
        return None
    d = wl.n
    opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=W, chunk=wl.chunk,
                    seg_off=wl.seg_off, tv=[], tu=[0], state=state)
    best = None
    for rep in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        opt.diag_server_pattern(packed)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        if rep and (best is None or ms < best):
            best = ms
    opt.close()
    gb = (W * nwords * 8 + 8.0 * d) / 1e9
    return {"ms": round(best, 4), "gb_per_launch": round(gb, 3),
            "gbs": round(gb / (best / 1000.0), 1),
            "frac": round(gb / (best / 1000.0) / HBM_PEAK_GBS, 4)}


def server_share(zo, torch, wl, state, g_in, packed, scales, srv_packed, srv_scales, W, reps=10):
    """The server at its per-GPU shape under the sharded design: GPU k = W/2
    serves a chunk-aligned range of about d/W elements, whose W-slot input
    holds every worker's words and scales for that range only (what the
    all-to-all delivers).  Each rep is a full sync step on a handle whose
    server range is that share (compress and reconstruct over all d, as every
    GPU runs them); the server launch is timed with HIP events.  Inputs are
    the bench's buffers (the slot of the range's own words is synthetic)."""
    start, ln, word, nwords = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    nch, d = len(ln), wl.n
    k = W // 2
    c0 = next(c for c in range(nch) if start[c] >= k * d // W)
    c1 = next((c for c in range(c0, nch) if start[c] >= (k + 1) * d // W), nch)
    w0, w1 = int(word[c0]), int(word[c1] if c1 < nch else nwords)
    ne = int(start[c1 - 1] + ln[c1 - 1] - start[c0])
    rp = packed[:, w0:w1].contiguous()
    rs = scales[:, c0:c1].contiguous()
    opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=W, chunk=wl.chunk,
                    seg_off=wl.seg_off, tv=[], tu=list(range(reps)), state=state,
                    srv_chunk_begin=c0, srv_chunk_end=c1, defer_sync_writes=True,
                    grad_dtype="f32" if g_in.dtype == torch.float32 else
                    ("bf16" if g_in.dtype == torch.bfloat16 else "f16"))
    ms = []
    try:
        for t in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            opt.compress_pack_ef(t, 1e-4, g_in, packed[0], scales[0])
            e0.record()
            opt.unpack_average(t, rp, rs, srv_packed, srv_scales)
            e1.record()
            opt.sync_update(t, srv_packed, srv_scales, None)
            torch.cuda.synchronize()
            if t >= 2:
                ms.append(e0.elapsed_time(e1))
    finally:
        opt.close()
    avg = sum(ms) / len(ms)
    pk, sc = 8 * (w1 - w0), 4 * (c1 - c0)
    nbytes = W * (pk + sc) + 8 * ne + pk + sc
    return {"gpu": k, "chunks": [c0, c1], "params": ne, "ms": round(avg, 4),
            "gb_per_launch": round(nbytes / 1e9, 4),
            "gbs": round(nbytes / 1e9 / (avg / 1000.0), 1),
            "frac": round(nbytes / 1e9 / (avg / 1000.0) / HBM_PEAK_GBS, 4)}


def schedule_run(zo, torch, wl, state, g_in, gb_in, packed, scales, srv_packed, srv_scales,
                 deferred, grad_dtype):
    """The workload's own schedule once (its T_v and T_u over its steps, its
    learning rates): sync steps while the variance is updated, then local
    steps between ever rarer syncs.  Timed with HIP events around the whole
    run (after one untimed run of the same schedule on another handle);
    run-level params/s = d * steps / time.  A third run brackets every launch
    with events of its own and sorts it into the kernel variant it ran (by
    where u was before the call), so `kernels` holds, per variant, the
    launches, their average time and the algorithmic rate against 8 TB/s (the
    events cost a few microseconds per launch, which matters only for tiny
    shards, so the run-level figures come from the run without them).  Inputs
    are the bench's buffers, reused at every step."""
    tu, tv = set(wl.tu), set(wl.tv)
    _, ln, _, nwords = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    gbytes = g_in.element_size()
    gt = {4: 0, 2: 1 if g_in.dtype == torch.float16 else 2}[gbytes]

    def run(timed):
        opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=wl.world,
                        chunk=wl.chunk, seg_off=wl.seg_off, tv=wl.tv, tu=wl.tu, state=state,
                        defer_sync_writes=deferred, grad_dtype=grad_dtype)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        marks = []

        def call(name, f):
            if timed:
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                f()
                b.record()
                marks.append((name, a, b))
            else:
                f()
        try:
            torch.cuda.synchronize()
            e0.record()
            for t in range(wl.steps):
                gam, gb = wl.gamma(t), (gb_in if t in tv else None)
                vs = "+var" if gb is not None else ""
                umode = zo.zo_state_location(opt.h)[1]
                u = {zo.U_IN_BUFFER: "", zo.U_ZERO: " (u=0)", zo.U_GAMMA_M: " (u=gm)"}[umode]
                if t in tu:
                    call("sync1" + u, lambda: opt.compress_pack_ef(t, gam, g_in, packed[0],
                                                                   scales[0]))
                    call("srv", lambda: opt.unpack_average(t, packed, scales, srv_packed,
                                                           srv_scales))
                    call(("recon (deferred)" if deferred else "recon") + vs,
                         lambda: opt.sync_update(t, srv_packed, srv_scales, gb))
                else:
                    call("local" + u + vs, lambda: opt.local_step(t, gam, g_in, gb))
            e1.record()
            torch.cuda.synchronize()
        finally:
            opt.close()
        return e0.elapsed_time(e1), marks

    run(False)
    ms, _ = run(False)
    ms_marked, marks = run(True)
    per = {}
    for name, a, b in marks:
        per.setdefault(name, []).append(a.elapsed_time(b))
    kernels = {}
    total_bytes = 0.0
    for name, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        avg = sum(v) / len(v)
        nb = variant_bytes(name, wl.n, len(ln), nwords, wl.world, gbytes)
        total_bytes += nb * len(v)
        base = name[:-4] if name.endswith("+var") else name
        kernels[name] = {
            "kernel": VARIANT_KERNELS[base].format(var="true" if name.endswith("+var")
                                                   else "false", gt=gt),
            "launches": len(v), "ms": round(avg, 4), "ms_total": round(sum(v), 3),
            "gb_per_launch": round(nb / 1e9, 3),
            "gbs": round(nb / 1e9 / (avg / 1000.0), 1),
            "frac": round(nb / 1e9 / (avg / 1000.0) / HBM_PEAK_GBS, 4)}
    return {"steps": wl.steps, "syncs": len(tu), "variance_updates": len(tv),
            "local_steps": wl.steps - len(tu), "ms": round(ms, 3),
            "ms_per_step": round(ms / wl.steps, 4),
            "ms_with_kernel_events": round(ms_marked, 3),
            "params_per_s": round(wl.n * wl.steps / (ms / 1000.0), 1),
            # every launch's algorithmic bytes over the run's time
            "hbm_frac": round(total_bytes / 1e9 / (ms / 1000.0) / HBM_PEAK_GBS, 4),
            "kernels": kernels}


def general_kernels(zo, torch, wl, state, g_in, gb_in, packed, scales, srv_packed, srv_scales,
                    grad_dtype, reps):
    """Each step of the path in its general form, every state read and written
    once (eager sync writes, u in its buffer): the local step with and
    without the variance line, the fused compress, and the reconstruction
    with and without the variance line, each launched `reps` times after two
    untimed launches and timed with HIP events; algorithmic bytes by
    variant_bytes.  Run A: local steps only, the variance line every other
    step; run B: a sync at every step, the variance line every other step."""
    _, ln, _, nwords = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    gbytes = g_in.element_size()
    T = 2 * (reps + 2)
    times = {}

    def timed(name, t, f):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        f()
        b.record()
        if t >= 4:
            times.setdefault(name, []).append((a, b))

    gam = 1e-4
    opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=wl.world, chunk=wl.chunk,
                    seg_off=wl.seg_off, tv=list(range(0, T, 2)), tu=[], state=state,
                    grad_dtype=grad_dtype)
    try:
        for t in range(T):
            gb = gb_in if t % 2 == 0 else None
            timed("local+var" if gb is not None else "local", t,
                  lambda: opt.local_step(t, gam, g_in, gb))
        torch.cuda.synchronize()
    finally:
        opt.close()
    opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=wl.world, chunk=wl.chunk,
                    seg_off=wl.seg_off, tv=list(range(0, T, 2)), tu=list(range(T)), state=state,
                    grad_dtype=grad_dtype)
    try:
        for t in range(T):
            gb = gb_in if t % 2 == 0 else None
            timed("sync1", t, lambda: opt.compress_pack_ef(t, gam, g_in, packed[0], scales[0]))
            opt.unpack_average(t, packed, scales, srv_packed, srv_scales)
            timed("recon+var" if gb is not None else "recon", t,
                  lambda: opt.sync_update(t, srv_packed, srv_scales, gb))
        torch.cuda.synchronize()
    finally:
        opt.close()
    out = {}
    for name in ("local", "local+var", "sync1", "recon", "recon+var"):
        v = [a.elapsed_time(b) for a, b in times[name]]
        avg = sum(v) / len(v)
        nb = variant_bytes(name, wl.n, len(ln), nwords, wl.world, gbytes)
        base = name[:-4] if name.endswith("+var") else name
        out[name] = {"kernel": VARIANT_KERNELS[base].format(
                         var="true" if name.endswith("+var") else "false",
                         gt={4: 0, 2: 1 if g_in.dtype == torch.float16 else 2}[gbytes]),
                     "launches": len(v), "ms": round(avg, 4),
                     "gb_per_launch": round(nb / 1e9, 3),
                     "gbs": round(nb / 1e9 / (avg / 1000.0), 1),
                     "frac": round(nb / 1e9 / (avg / 1000.0) / HBM_PEAK_GBS, 4)}
    return out


def _oracle_share(wl, c0, c1, fv, barrier, results):
    """One process of the chunk-parallel oracle run: chunks [c0, c1) of the
    shard, inputs generated at their global indices, then (after every
    process is ready) the same two steps as cpu_baseline, timed."""
    import numpy as np
    import oracle as orc
    import synth
    from synth import configs as C
    full = orc.Layout.from_segments(wl.seg_off, wl.chunk)
    lay = orc.Layout.from_lengths(full.clen[c0:c1])
    n, e0, w0 = lay.n, int(full.cstart[c0]), int(full.cword[c0])
    ks = C.ksigma(wl.sigma_g)
    x0 = synth.normal_host(n, e0, synth.key(0, C.STREAM_X, 0), C.ksigma(wl.sigma_x))
    g = synth.normal_host(n, e0, synth.key(0, C.STREAM_G, 0), ks, wl.outlier_per_mille,
                          wl.outlier_factor)
    gb = synth.normal_host(n, e0, synth.key(0, C.STREAM_GBAR, 0), ks, wl.outlier_per_mille,
                           wl.outlier_factor)
    W = wl.world
    base = np.float32(0.8 * wl.sigma_g if fv else 2 * 1e-4 * 0.18 * wl.sigma_g)
    pw = np.stack([synth.bits_host(lay.nwords, w0, synth.key(w, C.STREAM_BITS, 1))
                   for w in range(1, W)])
    ps = np.stack([synth.scales_host(c1 - c0, c0, synth.key(w, C.STREAM_SCALES, 1), base)
                   for w in range(1, W)])
    gam = np.float32(1e-4)
    if fv:
        worker = orc.FVWorker(lay, x0, wl.beta1, wl.beta2, wl.eps)
        barrier.wait()
        t0 = time.perf_counter()
        worker.step(gam, g, True, gbar=gb)
        worker.step(gam, g, False, peer_words=pw, peer_scales=ps)
    else:
        worker = orc.Worker(lay, x0, wl.beta1, wl.beta2, wl.eps)
        barrier.wait()
        t0 = time.perf_counter()
        worker.step(gam, g, False, True, gbar=gb)
        worker.step(gam, g, True, True, gbar=gb, peer_words=pw, peer_scales=ps)
    results.put((n, time.perf_counter() - t0))


def gpu_device_open():
    """Whether this process already holds the GPU device open (a profiler
    preloaded into it may initialise the GPU before the program starts)."""
    try:
        for fd in os.listdir("/proc/self/fd"):
            try:
                if os.readlink(f"/proc/self/fd/{fd}") == "/dev/kfd":
                    return True
            except OSError:
                pass
    except OSError:
        return True  # cannot tell: assume it is
    return False


def cpu_baseline_parallel(wl, sample_chunks, fv, cores):
    """The oracle as it stands, chunk-parallel on `cores` host cores: the
    sample's chunks split into contiguous ranges, one forked process each
    (every computation is chunk-local, so the ranges' results are the full
    run's).  Must run before this process initialises the GPU: the children
    are forks that never exec and never touch the GPU."""
    import multiprocessing as mp
    from oracle import Layout
    ctx = mp.get_context("fork")
    full = Layout.from_segments(wl.seg_off, wl.chunk)
    nch = min(sample_chunks, full.nchunks)
    cores = max(1, min(cores, nch))
    cuts = [nch * k // cores for k in range(cores + 1)]
    barrier, results = ctx.Barrier(cores), ctx.Queue()
    procs = [ctx.Process(target=_oracle_share,
                         args=(wl, cuts[k], cuts[k + 1], fv, barrier, results))
             for k in range(cores)]
    for p in procs:
        p.start()
    got = [results.get() for _ in procs]
    for p in procs:
        p.join()
    n = sum(r[0] for r in got)
    dt = max(r[1] for r in got)
    return {"value": 2 * n / dt, "unit": "params/s", "cores": cores, "kind": "oracle",
            "sample": f"first {nch} chunks ({n} params), split into {cores} contiguous chunk "
                      f"ranges, one process each: the same two steps; slowest process "
                      f"{dt:.2f} s"}


def cpu_baseline(wl, sample_chunks, fv=False):
    """Time the oracle on the first `sample_chunks` chunks of the shard: one
    local step with variance update and one sync step with variance update
    (Algorithm 4: one full-precision and one compressed step), W = 128
    (input generation excluded)."""
    import numpy as np
    import oracle as orc
    import synth
    from synth import configs as C
    full = orc.Layout.from_segments(wl.seg_off, wl.chunk)
    nch = min(sample_chunks, full.nchunks)
    lay = orc.Layout.from_lengths(full.clen[:nch])
    n = lay.n
    ks = C.ksigma(wl.sigma_g)
    x0 = synth.normal_host(n, 0, synth.key(0, C.STREAM_X, 0), C.ksigma(wl.sigma_x))
    g = synth.normal_host(n, 0, synth.key(0, C.STREAM_G, 0), ks, wl.outlier_per_mille,
                          wl.outlier_factor)
    gb = synth.normal_host(n, 0, synth.key(0, C.STREAM_GBAR, 0), ks, wl.outlier_per_mille,
                           wl.outlier_factor)
    W = wl.world
    base = np.float32(0.8 * wl.sigma_g if fv else 2 * 1e-4 * 0.18 * wl.sigma_g)
    pw = np.stack([synth.bits_host(lay.nwords, 0, synth.key(w, C.STREAM_BITS, 1))
                   for w in range(1, W)])
    ps = np.stack([synth.scales_host(nch, 0, synth.key(w, C.STREAM_SCALES, 1), base)
                   for w in range(1, W)])
    if fv:
        worker = orc.FVWorker(lay, x0, wl.beta1, wl.beta2, wl.eps)
        t0 = time.perf_counter()
        worker.step(np.float32(1e-4), g, True, gbar=gb)
        t1 = time.perf_counter()
        worker.step(np.float32(1e-4), g, False, peer_words=pw, peer_scales=ps)
        what = "one full-precision and one compressed step of Algorithm 4"
        kinds = ("full-precision", "compressed")
    else:
        worker = orc.Worker(lay, x0, wl.beta1, wl.beta2, wl.eps)
        t0 = time.perf_counter()
        worker.step(np.float32(1e-4), g, False, True, gbar=gb)
        t1 = time.perf_counter()
        worker.step(np.float32(1e-4), g, True, True, gbar=gb, peer_words=pw, peer_scales=ps)
        what = "one local+variance step and one sync+variance step"
        kinds = ("local+var", "sync+var")
    t2 = time.perf_counter()
    dt = t2 - t0
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            model = next(l.split(":", 1)[1].strip() for l in f if l.startswith("model name"))
    except (OSError, StopIteration):
        pass
    return {"value": 2 * n / dt, "unit": "params/s", "cores": 1, "kind": "oracle",
            "sample": f"first {nch} chunks ({n} params) of the same shard, W={W}: {what}, "
                      f"{dt:.2f} s",
            "ns_per_param": {kinds[0]: round((t1 - t0) * 1e9 / n, 2),
                             kinds[1]: round((t2 - t1) * 1e9 / n, 2)},
            "cpu": model}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="gpt2-1.5b")
    ap.add_argument("--cpu-sample-chunks", type=int, default=2048,
                    help="chunks of the shard the CPU oracle is timed on (GPT-2: 33.5M params)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-cores", type=int,
                    default=min(16, len(os.sched_getaffinity(0))),
                    help="processes of the chunk-parallel oracle run (1: skip it)")
    ap.add_argument("--eager-sync-writes", action="store_true",
                    help="the reconstruction writes x and u at every sync")
    ap.add_argument("--grad-dtype", choices=("f32", "f16", "bf16"), default="f32",
                    help="element type of the gradient inputs g and gbar")
    ap.add_argument("--algorithm", choices=("zero-one", "frozen-variance"), default="zero-one",
                    help="frozen-variance: Algorithm 4 (1-bit Adam's compression stage), one "
                         "full-precision and one compressed step per bench step")
    ap.add_argument("--placement-study", action="store_true",
                    help="time the general local step's stream mix with its arrays placed in "
                         "several ways (one JSON line), then exit")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="counter-collection run: first run plain and nontemporal copies of a "
                         "known size, and skip the measurements after the timed region")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the HBM traffic summary from two rocprofv3 --pmc runs and exit")
    ap.add_argument("--summarize-trace", metavar="TRACE_DIR",
                    help="print the timed kernels' durations from a rocprofv3 --kernel-trace "
                         "run of this command (same --workload/--warmup/--steps) and exit")
    ap.add_argument("--summarize-kernels", metavar="TRACE_DIR",
                    help="print every kernel of a rocprofv3 --kernel-trace run of this "
                         "command, grouped by template and grid, and exit")
    ap.add_argument("--summarize-counters", nargs="+", metavar="PMC_DIR",
                    help="print the timed kernels' counters from rocprofv3 --pmc runs and exit")
    args = ap.parse_args()
    fv = args.algorithm == "frozen-variance"
    mode = "frozen-variance" if fv else ("eager" if args.eager_sync_writes else "deferred")
    if args.grad_dtype != "f32":
        mode += f"/{args.grad_dtype}"
    if args.summarize_pmc:
        summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], TRAFFIC_FILE, mode,
                      args.workload)
        return
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, mode)
        return
    if args.summarize_kernels:
        summarize_kernels(args.summarize_kernels, args.workload)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, mode, args.workload, args.warmup, args.steps)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: the library is one worker's step on one GPU and "
              f"implements no multi-GPU exchange (asked for --gpus {args.gpus})", file=sys.stderr)
        sys.exit(2)

    from synth import configs as C
    wl = C.get(args.workload)
    # the chunk-parallel oracle run forks, so it runs before anything here
    # initialises the GPU
    cpu_parallel = None
    if (not args.no_cpu_baseline and not args.placement_study and args.cpu_cores > 1
            and not gpu_device_open()):
        print(f"[bench] timing the CPU oracle on {args.cpu_cores} cores", file=sys.stderr,
              flush=True)
        cpu_parallel = cpu_baseline_parallel(wl, args.cpu_sample_chunks, fv, args.cpu_cores)

    import torch
    import paper_2202_06009_amd as zo
    import synth

    zo.lib()
    if args.placement_study:
        res = placement_study(zo, torch, wl.n)
        print(json.dumps({"placement_study": res, "workload": wl.name, "params": wl.n,
                          "gb_per_launch": round(32.0 * wl.n / 1e9, 3),
                          "env": {"device": torch.cuda.get_device_properties(0).name,
                                  **device_clocks(0)}}))
        return
    if args.copy_calibration:
        src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for nt in (True, False):
            for _ in range(3):
                zo.zo_diag_copy(src, dst, nontemporal=nt)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()
    d, W = wl.n, wl.world
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    _, ln, word, nwords = zo.zo_plan_chunks(wl.seg_off, wl.chunk)
    nchunks = len(ln)
    print(f"[bench] {wl.name}: d={d} W={W} chunk={wl.chunk} chunks={nchunks} words={nwords}",
          file=sys.stderr, flush=True)

    f32 = dict(dtype=torch.float32, device=dev)
    state = {k: torch.empty(d, **f32) for k in ("x", "m", "v", "u", "err", "srv_err", "anchor")}
    g = torch.empty(d, **f32)
    gb = torch.empty(d, **f32)
    packed = torch.empty((W, nwords), dtype=torch.int64, device=dev)
    scales = torch.empty((W, nchunks), **f32)
    srv_packed = torch.empty(nwords, dtype=torch.int64, device=dev)
    srv_scales = torch.empty(nchunks, **f32)
    gdt = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[args.grad_dtype]
    gbytes = torch.empty(0, dtype=gdt).element_size()

    ks = C.ksigma(wl.sigma_g)
    synth.normal_dev(state["x"], 0, synth.key(0, C.STREAM_X, 0), C.ksigma(wl.sigma_x))
    synth.normal_dev(g, 0, synth.key(0, C.STREAM_G, 0), ks, wl.outlier_per_mille,
                     wl.outlier_factor)
    synth.normal_dev(gb, 0, synth.key(0, C.STREAM_GBAR, 0), ks, wl.outlier_per_mille,
                     wl.outlier_factor)
    g_in, gb_in = (g, gb) if gdt == torch.float32 else (g.to(gdt), gb.to(gdt))
    # peers compress u (two steps of gamma m) under Algorithm 1, g under Algorithm 4
    base = 0.8 * wl.sigma_g if fv else 2 * 1e-4 * 0.18 * wl.sigma_g
    for w in range(1, W):
        synth.bits_dev(packed[w], 0, synth.key(w, C.STREAM_BITS, 1))
        synth.scales_dev(scales[w], 0, synth.key(w, C.STREAM_SCALES, 1), base)

    total_steps = 2 * (args.warmup + args.steps)
    if fv:
        opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=W, chunk=wl.chunk,
                        seg_off=wl.seg_off, tv=list(range(0, total_steps, 2)), tu=[],
                        state=state, algorithm="frozen-variance", grad_dtype=args.grad_dtype)
        names = ("fv_full", "sync1", "srv", "fv_apply")
    else:
        opt = zo.ZoAdam(beta1=wl.beta1, beta2=wl.beta2, eps=wl.eps, world=W, chunk=wl.chunk,
                        seg_off=wl.seg_off, tv=list(range(total_steps)),
                        tu=list(range(1, total_steps, 2)), state=state,
                        defer_sync_writes=not args.eager_sync_writes,
                        grad_dtype=args.grad_dtype)
        names = ("local+var", "sync1", "srv", "recon+var")
    torch.cuda.synchronize()
    gamma = 1e-4

    def bench_step(k, ev=None):
        t = 2 * k
        first = (lambda: opt.fullprec_step(t, gamma, gb_in)) if fv else \
            (lambda: opt.local_step(t, gamma, g_in, gb_in))
        calls = (
            first,
            lambda: opt.compress_pack_ef(t + 1, gamma, g_in, packed[0], scales[0]),
            lambda: opt.unpack_average(t + 1, packed, scales, srv_packed, srv_scales),
            lambda: opt.sync_update(t + 1, srv_packed, srv_scales, None if fv else gb_in),
        )
        for i, call in enumerate(calls):
            if ev is not None:
                ev[i][0].record()
            call()
            if ev is not None:
                ev[i][1].record()

    for k in range(args.warmup):
        bench_step(k)
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in names]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        bench_step(args.warmup + k, evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    times = {n: sorted(evs[k][i][0].elapsed_time(evs[k][i][1]) for k in range(args.steps))
             for i, n in enumerate(names)}
    per_kernel = {n: sum(v) / len(v) for n, v in times.items()}
    median = {n: (v[(len(v) - 1) // 2] + v[len(v) // 2]) / 2 for n, v in times.items()}
    inexact = opt.inexact_chunks()
    opt.close()
    props = torch.cuda.get_device_properties(dev)
    # Measurements after the timed region.  A counter-collection run
    # (--copy-calibration) skips them: its counters must come from the timed
    # kernels, the calibration copies and the reference streams only (the
    # server share and the schedule run launch the same kernels at other
    # sizes, the ceiling the same copy kernel).
    extras = not args.copy_calibration
    if args.copy_calibration and args.grad_dtype == "f32":
        # reference streams for the counters: each kernel's mix, and one read
        # and one write array
        stream_mix_ceilings(zo, torch, state, g, gb, d, mode)
        zo.zo_diag_stream([g], [state["x"]])
        torch.cuda.synchronize()
    share = sched = mix = pattern = graphed = general = None
    copy_gbs = float("nan")
    if extras and not fv:
        share = server_share(zo, torch, wl, state, g_in, packed, scales, srv_packed, srv_scales,
                             W)
        sched = schedule_run(zo, torch, wl, state, g_in, gb_in, packed, scales, srv_packed,
                             srv_scales, not args.eager_sync_writes, args.grad_dtype)
        general = general_kernels(zo, torch, wl, state, g_in, gb_in, packed, scales, srv_packed,
                                  srv_scales, args.grad_dtype, args.steps)
    if extras:
        # the practical ceiling: a plain copy of one state vector (best of three)
        copy_ms = []
        for _ in range(3):
            c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            c0.record()
            zo.zo_diag_copy(state["x"], state["m"], nontemporal=True)
            c1.record()
            torch.cuda.synchronize()
            copy_ms.append(c0.elapsed_time(c1))
        copy_gbs = 8.0 * d / 1e9 / (min(copy_ms) / 1000.0)
        # (the diagnostic streams binary32 arrays: no like-for-like mix for 16-bit gradients)
        if args.grad_dtype == "f32":
            mix = stream_mix_ceilings(zo, torch, state, g, gb, d, mode)
        pattern = server_pattern(zo, torch, wl, state, packed, W, nwords)
        if not fv:
            # last: a capture that fails on some stack costs only this field
            try:
                graphed = graph_replay(zo, torch, wl, state, g_in, gb_in, packed, scales,
                                       srv_packed, srv_scales, not args.eager_sync_writes,
                                       args.grad_dtype, args.steps)
            except RuntimeError as e:
                graphed = {"error": str(e)[:200]}

    ms_per_step = wall * 1000.0 / args.steps
    value = 2.0 * d / (ms_per_step / 1000.0)
    bytes_ = algorithmic_bytes_fv(d, nchunks, nwords, W, gbytes) if fv else \
        algorithmic_bytes(d, nchunks, nwords, W, deferred=not args.eager_sync_writes,
                          gbytes=gbytes)
    kernels = {n: {"ms": round(per_kernel[n], 4),
                   "ms_median": round(median[n], 4),
                   "params_per_s": round(d / (per_kernel[n] / 1000.0), 1),
                   "gb_per_launch": round(bytes_[n] / 1e9, 3),
                   "gbs": round(bytes_[n] / 1e9 / (per_kernel[n] / 1000.0), 1),
                   "frac": round(bytes_[n] / 1e9 / (per_kernel[n] / 1000.0) / HBM_PEAK_GBS, 4),
                   "frac_of_copy": None if not extras else round(
                       bytes_[n] / 1e9 / (per_kernel[n] / 1000.0) / copy_gbs, 4)}
               for n in names}
    if pattern is not None and "srv" in kernels:
        # the server's algorithmic rate against its access pattern's
        kernels["srv"]["frac_of_pattern"] = round(kernels["srv"]["gbs"] / pattern["gbs"], 4)
    dom = max(names, key=lambda n: per_kernel[n])
    step_bytes = sum(bytes_.values())
    tb = measured_traffic(dom, mode, wl.name)
    traffic_gb = None if tb is None else round(tb / 1e9, 3)
    out = {
        "metric": "0/1 Adam step params/sec and achieved HBM GB/s (% of peak), 1 MI355X",
        "value": round(value, 1),
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{wl.name} flat shard, " + (
                       "Algorithm 4: one full-precision and one compressed step per bench step"
                       if fv else "one local+variance step and one sync+variance step per "
                                  "bench step"),
                   "algorithm": args.algorithm, "grad_dtype": args.grad_dtype,
                   "params": d, "segments": wl.nseg, "world": W, "chunk": wl.chunk,
                   "chunks": nchunks, "server": "single (all chunks)",
                   "sync_writes": None if fv else ("eager" if args.eager_sync_writes
                                                   else "deferred"),
                   "optimizer_steps_per_bench_step": 2},
        "hbm_gbs_step": round(step_bytes / 1e9 / (ms_per_step / 1000.0), 1),
        "hbm_frac_step": round(step_bytes / 1e9 / (ms_per_step / 1000.0) / HBM_PEAK_GBS, 4),
        "kernels": kernels,
        "inexact_chunks": inexact,
        "copy_gbs": round(copy_gbs, 1) if extras else None,
        "stream_mix_ceiling": mix,
        # the single server's memory accesses without its arithmetic
        "server_pattern": pattern,
        # the same bench step recorded once in a HIP graph and replayed
        "graph_replay": graphed,
        # the workload's own schedule once (mostly local steps after the warm-up phase)
        "schedule_run": sched,
        # the server at one GPU's share of a W-GPU sharded run, and that GPU's time for a
        # local+variance and a sync+variance step there, collectives excluded
        "server_share": share,
        "sharded_ms_per_step_no_collectives": None if share is None else round(
            per_kernel["local+var"] + per_kernel["sync1"] + share["ms"] + per_kernel["recon+var"],
            4),
        "env": {"device": props.name, "arch": getattr(props, "gcnArchName", None),
                "compute_units": props.multi_processor_count, "hip": torch.version.hip,
                "torch": torch.__version__, **device_clocks(dev.index or 0)},
        # each step of the path in its general form (every state read and written)
        "general_kernels": general,
        "roofline": {"bound": "hbm", "kernel": dom,
                     "achieved": kernels[dom]["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": kernels[dom]["frac"], "traffic": traffic_gb,
                     "gb_per_launch": kernels[dom]["gb_per_launch"]},
    }
    if general is not None and dom in general:
        # the same row with every state read and written (no deferred writes)
        out["roofline"]["general_form"] = {k: general[dom][k] for k in (
            "kernel", "gb_per_launch", "gbs", "frac")}
    if sched is not None and sched.get("kernels"):
        top = next(iter(sched["kernels"]))  # the variant with the most time in the schedule
        out["roofline"]["schedule_dominant"] = {"variant": top} | {
            k: sched["kernels"][top][k] for k in ("kernel", "launches", "ms_total",
                                                 "gb_per_launch", "gbs", "frac")}
        out["roofline"]["schedule_hbm_frac"] = sched["hbm_frac"]
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_chunks, fv)
        out["cpu_baseline_all_cores"] = cpu_parallel
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
