#!/usr/bin/env python3
"""Throughput of dense C = A * B on one MI355X: FP16->FP32, INT8->INT32 and
INT4->INT32 at square N in {512, 1024, 2048, 4096, 8192}.

One step is one pass over the whole precision x size sweep: 15 GEMMs, each on
its own seeded synthetic operands (seeds 10..24, FP16 U[-1,1], INT8 uniform
over [-128, 127], INT4 uniform over [-8, 7] packed two per byte), already
resident in HBM. Every GEMM goes through the library's C ABI on one stream.
Ops per GEMM are 2*N^3 (the paper's convention: its Table II TOPS column is
2*N^3 / duration).

Printed: one JSON line on stdout (progress goes to stderr) with
  value      whole-step throughput, total ops / wall time per step (TOP/s);
  points     per-GEMM median duration (HIP events on the launch stream, over
             the timed region; mean, min and max beside it), TOP/s and
             fraction of the precision's dense MFMA peak, and the oracle's
             check of sampled output rows (max FP16 normalised error, or
             bit-exactness);
  roofline   the dominant kernel (largest share of step time) against its
             precision's MFMA peak, with HBM traffic from the committed
             counter profile when it still matches the kernel sources;
  cpu_baseline  the CPU oracle timed on this host on a bounded row sample of
             the N = 8192 points, which also checks those GPU rows;
  clock_mhz  the shader clock sampled from the driver during the timed
             region (null where the driver does not expose it).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# Published dense (non-sparse) MFMA peaks of the MI355X, in T(FL)OP/s. gfx950
# has no 4-bit integer MFMA: INT4 runs either on the INT8 MFMA (peak 5000) or,
# converted to FP6, on the FP6 MFMA (peak 10100); a point is priced at the
# peak of the MFMA its kernel uses.
PEAK = {"f16": 2500.0, "s8": 5000.0, "s4": 5000.0}
PEAK_FP6 = 10100.0


def point_peak(dtype: str, variant_name: str) -> float:
    return PEAK_FP6 if variant_name.startswith(("fp6", "e2m3")) else PEAK[dtype]
PEAK_UNIT = {"f16": "TFLOP/s", "s8": "TOP/s", "s4": "TOP/s"}
IN_BYTES = {"f16": 2.0, "s8": 1.0, "s4": 0.5}
METRIC = "TFLOP/s | TOP/s at N=512–8192 for FP16, INT8, INT4; % of MFMA peak per dtype"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# precisions timed through mpgemm_gemm_ws with a workspace
WS_DTYPES = ("s4",)
# rows of each N = 8192 point the CPU oracle computes for the baseline sample
CPU_SAMPLE_ROWS = {"f16": 1024, "s8": 8192, "s4": 8192}


def gemm_ops(m: int, n: int, k: int) -> float:
    """Operations of one GEMM: a multiply and an add per (i, j, k) term, the
    convention of the paper's throughput figures (its Table II TOPS column is
    2 * N^3 / duration)."""
    return 2.0 * m * n * k


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# Sources that define each kernel family (by variant-name prefix), besides
# device_common.hpp and the build flags: stored counters stay valid while
# these are unchanged.
KERNEL_SOURCES = {"generic": ["generic_gemm.hpp"], "tile": ["tiled_gemm.hpp"], "pipe": ["tiled_gemm.hpp"],
                  "spread": ["tiled_gemm.hpp"], "staged": ["tiled_gemm.hpp"],
                  "pingpong": ["tiled_gemm.hpp"], "fp6pipe": ["tiled_gemm.hpp", "f6_gemm.hpp"],
                  "deep": ["tiled_gemm.hpp", "deep_gemm.hpp"], "skinny": ["skinny_gemm.hpp"],
                  "wide": ["tiled_gemm.hpp", "wide_gemm.hpp"],
                  "fp6wide": ["tiled_gemm.hpp", "f6_gemm.hpp", "wide_gemm.hpp", "wide_f6.hpp"],
                  "e2m3wide": ["tiled_gemm.hpp", "f6_gemm.hpp", "wide_gemm.hpp", "wide_i4.hpp"]}


def kernel_source_hash(variant_name: str) -> str:
    """Hash of the sources that define a variant's kernel (its family's
    headers, device_common.hpp and the build flags), to tell whether stored
    counters still apply to it."""
    fam = next((k for k in sorted(KERNEL_SOURCES, key=len, reverse=True) if variant_name.startswith(k)), None)
    if fam is None:
        raise ValueError(f"unknown kernel family of {variant_name}")
    csrc = os.path.join(ROOT, "paper_2608_10103_amd", "csrc")
    files = [os.path.join(csrc, f) for f in ["device_common.hpp"] + KERNEL_SOURCES[fam]]
    files.append(os.path.join(ROOT, "paper_2608_10103_amd", "build.py"))
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.basename(f).encode())
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def parse_points(spec: str):
    import seeded_inputs as si
    if spec == "sweep":
        return si.sweep_points()
    pts = []
    sweep = {(d, n): s for d, n, s in si.sweep_points()}
    for item in spec.split(","):
        d, n = item.split(":")[:2]
        n = int(n)
        pts.append((d, n, sweep.get((d, n), 10)))
    return pts


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--points", default="sweep",
                    help='"sweep" or a list like "f16:8192,s8:4096"')
    ap.add_argument("--variant", action="append", default=[],
                    help="force a kernel variant for a point: dtype:N:variant")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="instead of the sweep, run a plain device copy of this many MiB "
                         "--steps times (reference kernel for counter calibration)")
    ap.add_argument("--ingest-pmc", nargs=4, metavar=("GEMM_FETCH", "GEMM_WRITE", "COPY_FETCH", "COPY_WRITE"),
                    help="rocprofv3 --pmc output folders (FETCH_SIZE, WRITE_SIZE of the GEMM run; "
                         "the same of a --copy-mib run) -> profiles/traffic.json")
    ap.add_argument("--copy-mib-ref", type=int, default=256,
                    help="size of the copy the calibration folders were taken on")
    ap.add_argument("--counters-table", nargs="+", metavar="KIND=FOLDER",
                    help="print a per-point counter table from rocprofv3 --pmc folders of this "
                         "script's runs over --points: mfma= (SQ_VALU_MFMA_BUSY_CYCLES, SQ_WAVES, "
                         "SQ_WAVE_CYCLES, SQ_LDS_BANK_CONFLICT, GRBM_GUI_ACTIVE), fetch= (FETCH_SIZE), "
                         "write= (WRITE_SIZE), copyfetch= and copywrite= (the same of a --copy-mib run)")
    ap.add_argument("--write-traffic", action="store_true",
                    help="with --counters-table: store every point's HBM-side traffic per launch in "
                         "profiles/traffic.json")
    args = ap.parse_args()

    if args.ingest_pmc:
        ingest_pmc(args)
        return
    if args.counters_table:
        counters_table(args)
        return

    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_10103_amd as mp
    import seeded_inputs as si

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    mp.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    props = torch.cuda.get_device_properties(dev)
    forced = {}
    for f in args.variant:
        d, n, v = f.split(":")
        forced[(d, int(n))] = int(v)

    if args.copy_mib:
        x = torch.empty(args.copy_mib << 20, dtype=torch.uint8, device=dev)
        y = torch.empty_like(x)
        for _ in range(args.steps):
            y.copy_(x)
        torch.cuda.synchronize()
        log(f"copied {args.copy_mib} MiB x {args.steps}")
        return

    points = parse_points(args.points)
    bufs = []
    for dt, n, seed in points:
        log(f"generating {dt} N={n} seed={seed}")
        A, B = si.gen_operands(dt, n, n, n, seed=seed)
        Ad = torch.from_numpy(A).to(dev)
        Bd = torch.from_numpy(B).to(dev)
        C = torch.empty((n, n), dtype=torch.float32 if dt == "f16" else torch.int32, device=dev)
        v = forced.get((dt, n))
        # INT4 goes through mpgemm_gemm_ws with a workspace (allocated here,
        # before timing), which takes the FP6 kernel fed by the conversion
        # pre-pass where that is faster; FP16 and INT8 through their plain
        # entry points (no workspace); a forced variant gets the workspace it
        # needs
        use_ws = dt in WS_DTYPES or v is not None
        wsb = mp.workspace_size(dt, n, n, n, variant=v) if use_ws else 0
        ws = mp.new_workspace(wsb, dev) if wsb else None
        vsel = v if v is not None else mp.select_variant(dt, n, n, n, Ad.data_ptr(), Bd.data_ptr(),
                                                         C.data_ptr(), with_ws=ws is not None)
        bufs.append(dict(dt=dt, n=n, seed=seed, A=Ad, B=Bd, C=C, host=(A, B), variant=v,
                         vname=mp.variant_name(dt, vsel), ws=ws, ws_bytes=wsb))
    torch.cuda.synchronize()

    stream = torch.cuda.Stream(device=dev)  # default priority
    fns = mp.GEMM

    def step(events=None):
        for i, b in enumerate(bufs):
            if events is not None:
                events[i][0].record(stream)
            fns[b["dt"]](b["A"], b["B"], C=b["C"], stream=stream, variant=b["variant"], workspace=b["ws"])
            if events is not None:
                events[i][1].record(stream)

    log(f"warmup {args.warmup} steps")
    with torch.cuda.stream(stream):
        for _ in range(args.warmup):
            step()
    torch.cuda.synchronize()

    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            for _ in bufs] for _ in range(args.steps)]
    log(f"timing {args.steps} steps")
    clock = ClockSampler()
    torch.cuda.synchronize()
    clock.start()
    t0 = time.perf_counter()
    with torch.cuda.stream(stream):
        for s in range(args.steps):
            step(evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    clock_mhz = clock.stop()
    log(f"timed region {wall * 1e3:.1f} ms")

    ms_per_step = wall * 1e3 / args.steps
    total_ops = sum(gemm_ops(b["n"], b["n"], b["n"]) for b in bufs)
    value = total_ops / (ms_per_step * 1e-3) / 1e12

    pts = []
    for i, b in enumerate(bufs):
        ms = [evs[s][i][0].elapsed_time(evs[s][i][1]) for s in range(args.steps)]
        med_ms, mean_ms = float(np.median(ms)), float(np.mean(ms))
        ops = gemm_ops(b["n"], b["n"], b["n"])
        tops = ops / (med_ms * 1e-3) / 1e12
        pts.append(dict(dtype=b["dt"], n=b["n"], variant=b["vname"], ms=round(med_ms, 5),
                        ms_mean=round(mean_ms, 5), ms_min=round(float(np.min(ms)), 5),
                        ms_max=round(float(np.max(ms)), 5),
                        tops=round(tops, 2), frac_peak=round(tops / point_peak(b["dt"], b["vname"]), 4),
                        total_ms=mean_ms * args.steps))

    dom = max(pts, key=lambda p: p["total_ms"])
    n = dom["n"]
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        try:
            tr = json.load(open(TRAFFIC_FILE))
            key = f'{dom["dtype"]}:{n}:{dom["variant"]}'
            ent = tr.get("points", {}).get(key)
            if ent and ent.get("kernel_source_hash") == kernel_source_hash(dom["variant"]):
                traffic = ent["hbm_bytes_per_launch"]
        except (ValueError, KeyError, OSError):
            traffic = None
    roofline = dict(bound="mfma", kernel=f'{dom["dtype"]} N={n} {dom["variant"]}',
                    achieved=round(dom["tops"], 2), peak=point_peak(dom["dtype"], dom["variant"]),
                    unit=PEAK_UNIT[dom["dtype"]],
                    frac=round(dom["tops"] / point_peak(dom["dtype"], dom["variant"]), 4),
                    traffic=traffic,
                    algorithmic_bytes=int((2 * IN_BYTES[dom["dtype"]] + 4) * n * n),
                    algorithmic_ops=int(gemm_ops(n, n, n)))
    for p in pts:
        p.pop("total_ms")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(bufs, log)
        for p, chk in zip(pts, cpu.pop("point_checks")):
            p["check"] = chk

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16->f32, s8->s32, s4->s32",
        "data": "synthetic (seeded SplitMix64; FP16 U[-1,1], INT8 U{-128..127}, INT4 U{-8..7})",
        "config": {
            "workload": "precision x size sweep: square GEMM C=A*B (A row-major, B column-major), "
                        "FP16/INT8/INT4 at N in {512,1024,2048,4096,8192}, seeds 10..24"
                        if args.points == "sweep" else f"points {args.points}",
            "points": len(bufs),
            "ops_per_step": total_ops,
            "entry_points": "FP16 gemm_f16_f32, INT8 gemm_s8_s32 (no workspace); INT4 mpgemm_gemm_ws "
                            "with a caller workspace" if not forced else "forced variants via mpgemm_run_variant(_ws)",
            "workspace_bytes": int(sum(b["ws_bytes"] for b in bufs)),
        },
        "clock_mhz": clock_mhz,
        "device": {"name": props.name, "cus": props.multi_processor_count},
        "points": pts,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


class ClockSampler:
    """Samples the GPU shader clock the driver reports (the active level of
    pp_dpm_sclk in sysfs) every 5 ms on a host thread; stop() returns the
    median, min and max in MHz, or None where the file is not readable."""

    def __init__(self):
        import glob
        self.files = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
        self.samples = []
        self._run = False
        self._t = None

    def _read(self):
        for f in self.files:
            try:
                for line in open(f):
                    if line.rstrip().endswith("*"):
                        return float(line.split(":")[1].strip().rstrip("*").strip().lower().rstrip("mhz"))
            except (OSError, ValueError, IndexError):
                continue
        return None

    def _loop(self):
        while self._run:
            v = self._read()
            if v is not None:
                self.samples.append(v)
            time.sleep(0.005)

    def start(self):
        import threading
        if not self.files or self._read() is None:
            return
        self._run = True
        self._t = threading.Thread(target=self._loop, daemon=True)
        self._t.start()

    def stop(self):
        if self._t is None:
            return None
        self._run = False
        self._t.join()
        if not self.samples:
            return None
        return {"median": float(np.median(self.samples)), "min": float(np.min(self.samples)),
                "max": float(np.max(self.samples)), "samples": len(self.samples),
                "source": "pp_dpm_sclk active level"}


def _read_counter(folder, counter, name_filter):
    """Per-dispatch values of one counter from a rocprofv3 --pmc CSV folder."""
    import csv
    import glob
    vals = []
    for f in glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] == counter and name_filter(r["Kernel_Name"]):
                vals.append((r["Kernel_Name"], float(r["Counter_Value"])))
    if not vals:
        raise SystemExit(f"no {counter} values in {folder}")
    return vals


def ingest_pmc(args):
    """Scale the GEMM's FETCH_SIZE / WRITE_SIZE (KiB per dispatch) by what the
    same counters read for a plain copy of known size, and store the per-launch
    HBM-side traffic of the dominant kernel with the hash of its sources."""
    import paper_2608_10103_amd as mp
    gf, gw, cf, cw = args.ingest_pmc
    is_gemm = lambda n: "mpg::" in n
    is_copy = lambda n: "copy" in n.lower()
    copy_kib = float(args.copy_mib_ref) * 1024.0
    rf = float(np.median([v for _, v in _read_counter(cf, "FETCH_SIZE", is_copy)])) / copy_kib
    wf = float(np.median([v for _, v in _read_counter(cw, "WRITE_SIZE", is_copy)])) / copy_kib
    fetch = _read_counter(gf, "FETCH_SIZE", is_gemm)
    write = _read_counter(gw, "WRITE_SIZE", is_gemm)
    kname = fetch[0][0]
    f_kib = float(np.median([v for _, v in fetch]))
    w_kib = float(np.median([v for _, v in write]))
    pts = parse_points(args.points)
    dt, n, _ = pts[0]
    v = mp.select_variant(dt, n, n, n)
    key = f"{dt}:{n}:{mp.variant_name(dt, v)}"
    hbm = (f_kib / rf + w_kib / wf) * 1024.0
    out = {"copy_calibration": {"mib": args.copy_mib_ref, "fetch_scale": rf, "write_scale": wf},
           "points": {key: {"kernel_source_hash": kernel_source_hash(mp.variant_name(dt, v)),
                            "kernel_name": kname, "fetch_kib_per_launch": f_kib,
                            "write_kib_per_launch": w_kib,
                            "hbm_bytes_per_launch": int(hbm)}}}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    json.dump(out, open(TRAFFIC_FILE, "w"), indent=1)
    print(json.dumps(out))


def _dispatches(folder):
    """Library dispatches of a rocprofv3 --pmc CSV folder in dispatch order:
    [(kernel name, {counter: value}, duration in ns)]."""
    import csv
    import glob
    rows = {}
    for f in glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if "mpg::" not in r["Kernel_Name"]:
                continue
            d = rows.setdefault(int(r["Dispatch_Id"]), [r["Kernel_Name"], {},
                                                         int(r["End_Timestamp"]) - int(r["Start_Timestamp"])])
            d[1][r["Counter_Name"]] = float(r["Counter_Value"])
    if not rows:
        raise SystemExit(f"no library dispatches in {folder}")
    return [tuple(rows[k]) for k in sorted(rows)]


def counters_table(args):
    """Per-point counters of runs of this script over --points (every step
    launches the same library kernels in the same order: the INT4 FP6 pre-pass,
    where the chosen kernel needs one, then the GEMM). Medians over the runs'
    steps. Clock = GRBM_GUI_ACTIVE / 8 XCDs / duration; MFMA busy =
    SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x cycles); waves per SIMD =
    4 SQ_WAVE_CYCLES (counted in 4-cycle units) / (1024 x cycles); LDS bank
    conflicts per CU-cycle = SQ_LDS_BANK_CONFLICT / (256 x cycles); HBM-side
    bytes = FETCH_SIZE / read scale + WRITE_SIZE / write scale, the scales
    being what the same counters read per byte of a plain copy."""
    import paper_2608_10103_amd as mp
    folders = dict(kv.split("=", 1) for kv in args.counters_table)
    pts = parse_points(args.points)
    seq = []  # (point index, kernel role) per dispatch of one step
    for i, (dt, n, _) in enumerate(pts):
        name = mp.variant_name(dt, mp.select_variant(dt, n, n, n, with_ws=dt in WS_DTYPES))
        if name.startswith("fp6"):
            seq.append((i, "pre-pass"))
        seq.append((i, name))
    per = {}
    for kind, folder in folders.items():
        if kind.startswith("copy"):
            continue
        ds = _dispatches(folder)
        if len(ds) % len(seq):
            raise SystemExit(f"{folder}: {len(ds)} dispatches, not a multiple of {len(seq)} per step")
        for j, (kname, cnt, dur) in enumerate(ds):
            slot = per.setdefault(j % len(seq), {"kernel": kname, "dur": [], "c": {}})
            if kind == "mfma":
                slot["dur"].append(dur)
            for c, v in cnt.items():
                slot["c"].setdefault(c if c != "GRBM_GUI_ACTIVE" else f"GRBM_{kind}", []).append((v, dur))
    scale = {}
    for kind, cname in (("copyfetch", "FETCH_SIZE"), ("copywrite", "WRITE_SIZE")):
        if kind in folders:
            vals = [c[cname] for _, c, _ in _dispatches_any(folders[kind]) if cname in c]
            scale[cname] = float(np.median(vals)) / (args.copy_mib_ref * 1024.0)
    med = lambda xs: float(np.median(xs)) if xs else float("nan")
    traffic, prepass = {}, {}
    print("| point | kernel | median us | clock GHz | MFMA busy | waves/SIMD | LDS conflicts per CU-cycle | "
          "FETCH KiB | WRITE KiB | HBM-side MB | HBM GB/s | algorithmic MB | traffic / algorithmic |")
    print("|---|---|---|---|---|---|---|---|---|---|---|---|---|")
    for j, (i, role) in enumerate(seq):
        dt, n, _ = pts[i]
        slot = per.get(j)
        if slot is None:
            continue
        c = slot["c"]
        dur_ns = med(slot["dur"]) if slot["dur"] else med([d for _, d in c.get("GRBM_fetch", [])])
        cyc = med([v for v, _ in c.get("GRBM_mfma", [])]) / 8.0

        def per_cycle(name, denom):
            xs = [v for v, _ in c.get(name, [])]
            return med(xs) / (denom * cyc) if xs and cyc > 0 else float("nan")
        clock = cyc / dur_ns if dur_ns > 0 else float("nan")
        mfma = per_cycle("SQ_VALU_MFMA_BUSY_CYCLES", 1024.0)
        waves = 4.0 * per_cycle("SQ_WAVE_CYCLES", 1024.0)
        lds = per_cycle("SQ_LDS_BANK_CONFLICT", 256.0)
        fk = med([v for v, _ in c.get("FETCH_SIZE", [])])
        wk = med([v for v, _ in c.get("WRITE_SIZE", [])])
        hbm = (fk / scale["FETCH_SIZE"] + wk / scale["WRITE_SIZE"]) * 1024.0 if scale and fk == fk and wk == wk \
            else float("nan")
        # bytes per operand element the kernel reads: the FP6 GEMM reads the
        # pre-pass's 6-bit codes
        elem = 0.75 if role.startswith("fp6") else {"f16": 2.0, "s8": 1.0, "s4": 0.5}[dt]
        alg = 2 * n * n * elem + 4.0 * n * n if role != "pre-pass" else 2 * n * n * 0.5 + 2 * n * n * 0.75
        kname = slot["kernel"].split("(")[0].replace("void ", "")
        label = f"{dt} {n}" + (" (pre-pass)" if role == "pre-pass" else "")
        if role == "pre-pass":
            prepass[i] = hbm
        else:
            traffic[f"{dt}:{n}:{role}"] = {"kernel_source_hash": kernel_source_hash(role), "kernel_name": kname,
                                           "fetch_kib_per_launch": fk, "write_kib_per_launch": wk,
                                           "hbm_bytes_per_launch": int(hbm)}
            if i in prepass:
                traffic[f"{dt}:{n}:{role}"]["prepass_hbm_bytes_per_launch"] = int(prepass[i])
        print(f"| {label} | `{kname}` | {dur_ns / 1e3:.1f} | {clock:.2f} | {100 * mfma:.1f}% | {waves:.2f} | "
              f"{lds:.4f} | {fk:.0f} | {wk:.0f} | {hbm / 1e6:.1f} | {hbm / dur_ns:.0f} | {alg / 1e6:.1f} | "
              f"{hbm / alg:.2f} |")
    if args.write_traffic:
        out = {"copy_calibration": {"mib": args.copy_mib_ref, "fetch_scale": scale["FETCH_SIZE"],
                                    "write_scale": scale["WRITE_SIZE"]},
               "points": traffic}
        os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
        json.dump(out, open(TRAFFIC_FILE, "w"), indent=1)


def _dispatches_any(folder):
    """Every dispatch of a folder (the copy runs launch torch's kernels)."""
    import csv
    import glob
    rows = {}
    for f in glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if "copy" not in r["Kernel_Name"].lower():
                continue
            d = rows.setdefault(int(r["Dispatch_Id"]), [r["Kernel_Name"], {}, 0])
            d[1][r["Counter_Name"]] = float(r["Counter_Value"])
    return [tuple(rows[k]) for k in sorted(rows)]


def cpu_baseline(bufs, log):
    """The CPU oracle, timed on this host's cores on a bounded row sample of
    each N = 8192 point (or of the largest points present); its rows also
    check the GPU output of those points."""
    import oracle
    import seeded_inputs as si
    import torch

    nmax = max(b["n"] for b in bufs)
    big = [b for b in bufs if b["n"] == nmax]
    threads = oracle.default_threads()
    total_ops, total_s, checked, parts = 0.0, 0.0, True, []
    for b in big:
        dt, n = b["dt"], b["n"]
        nrows = min(CPU_SAMPLE_ROWS[dt], n)
        rows = si.sample_rows(b["seed"] + 2000, n, nrows, force=(0, n - 1))
        A, B = b["host"]
        log(f"cpu oracle {dt} N={n}: {len(rows)} rows on {threads} threads")
        t0 = time.perf_counter()
        if dt == "f16":
            ref, D = oracle.gemm_f16(A, B, rows=rows, threads=threads)
        elif dt == "s8":
            ref, D = oracle.gemm_s8(A, B, rows=rows, threads=threads), None
        else:
            ref, D = oracle.gemm_s4(A, B, rows=rows, threads=threads), None
        dt_s = time.perf_counter() - t0
        ops = gemm_ops(len(rows), n, n)
        total_ops += ops
        total_s += dt_s
        got = b["C"][torch.from_numpy(rows.astype(np.int64)).to(b["C"].device)].cpu().numpy()
        if dt == "f16":
            ok = oracle.normalized_error(got, ref, D) <= 1e-3
        else:
            ok = bool(np.array_equal(got.astype(np.int64), ref))
        checked = checked and ok
        parts.append(f"{dt} N={n}: {len(rows)} rows in {dt_s:.2f} s")
    # every point: the oracle on 8 sampled rows (plus the first and the last),
    # max FP16 normalised error or bit-exactness of those GPU rows
    checks = []
    for b in bufs:
        dt, n = b["dt"], b["n"]
        rows = si.sample_rows(b["seed"] + 3000, n, min(8, n), force=(0, n - 1))
        A, B = b["host"]
        got = b["C"][torch.from_numpy(rows.astype(np.int64)).to(b["C"].device)].cpu().numpy()
        if dt == "f16":
            ref, D = oracle.gemm_f16(A, B, rows=rows, threads=threads)
            checks.append({"rows": int(len(rows)), "max_norm_err": float(oracle.normalized_error(got, ref, D))})
        else:
            ref = oracle.gemm_s8(A, B, rows=rows, threads=threads) if dt == "s8" else \
                oracle.gemm_s4(A, B, rows=rows, threads=threads)
            checks.append({"rows": int(len(rows)), "bit_exact": bool(np.array_equal(got.astype(np.int64), ref))})
    try:
        model = next(l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo")
                     if l.startswith("model name"))
    except (OSError, StopIteration):
        model = "unknown"
    return {
        "value": round(total_ops / total_s / 1e12, 5),
        "unit": "TOP/s",
        "cores": threads,
        "kind": "oracle",
        "sample": "; ".join(parts) + " (2*rows*N*N ops each)",
        "cpu_model": model,
        "cpu_count": os.cpu_count(),
        "gpu_rows_match_oracle": checked and all(c.get("bit_exact", True) and c.get("max_norm_err", 0.0) <= 1e-3
                                                 for c in checks),
        "point_checks": checks,
    }


if __name__ == "__main__":
    main()
