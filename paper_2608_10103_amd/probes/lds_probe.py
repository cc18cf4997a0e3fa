"""LDS probes on one MI355X: swizzle ranking for 64-byte operand rows, and the
cost of LDS writes to concurrent operand reads.

    python -m paper_2608_10103_amd.probes.lds_probe [--out FILE.md]

Builds lds_probe.hip for gfx950 with hipcc into a temporary directory, runs
each kernel over 256 workgroups (one per CU) and prints a markdown table of
median run times (relative to the reference case of each table).
"""
from __future__ import annotations

import argparse
import ctypes
import os
import statistics
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))


def build(outdir: str) -> str:
    so = os.path.join(outdir, "liblds_probe.so")
    cmd = ["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O3", "-std=c++17", "-shared", "-fPIC",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           os.path.join(HERE, "lds_probe.hip"), "-o", so]
    subprocess.run(cmd, check=True, capture_output=True)
    return so


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--out", default="")
    ap.add_argument("--rounds", type=int, default=3)
    args = ap.parse_args(argv)
    import torch

    with tempfile.TemporaryDirectory() as tmp:
        lib = ctypes.CDLL(build(tmp))
        lib.probe_lds_read_swizzle.argtypes = [ctypes.c_int] * 5 + [ctypes.c_void_p, ctypes.c_void_p]
        lib.probe_lds_read_with_writes.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                                                   ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
        sink = torch.zeros(16, dtype=torch.int32, device="cuda")
        src = torch.zeros(1 << 20, dtype=torch.uint8, device="cuda")
        st = torch.cuda.current_stream()

        def timed(fn):
            out = []
            for _ in range(args.rounds):
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(st)
                rc = fn()
                e1.record(st)
                torch.cuda.synchronize()
                if rc != 0:
                    raise RuntimeError(f"probe launch failed: {rc}")
                out.append(e0.elapsed_time(e1))
            return statistics.median(out)

        lines = ["## Operand reads from 64-byte LDS rows: swizzle ranking",
                 "", "slot of chunk c of row q: c ^ (((q >> a) ^ (q >> b)) & 3); time relative to the "
                 "128-byte rows with (q ^ (q >> 3)) & 7 (no bank conflicts)", "",
                 "| rows | a | b | ms | relative |", "|---|---|---|---|---|"]
        cands = [(128, 0, 3)] + [(64, a, b) for a in range(7) for b in [-1] + list(range(a + 1, 8))]
        res = []
        for rb, a, b in cands:
            ms = timed(lambda: lib.probe_lds_read_swizzle(rb, a, b, 4096, 256, sink.data_ptr(),
                                                           st.cuda_stream))
            res.append((ms, rb, a, b))
        ref = res[0][0]
        for ms, rb, a, b in sorted(res):
            lines.append(f"| {rb} | {a} | {'-' if b < 0 else b} | {ms:.3f} | {ms / ref:.2f} |")
        lines += ["", "## Operand reads with one LDS write per eight 1 KiB reads (8 waves per CU)", "",
                  "| extra write per iteration | ms | relative |", "|---|---|---|"]
        kinds = ["none", "direct-to-LDS load, 16 B per lane (1 KiB)",
                 "direct-to-LDS load, 4 B per lane (256 B)", "ds_write_b128 (1 KiB)"]
        times = [timed(lambda k=k: lib.probe_lds_read_with_writes(k, src.data_ptr(), 4096, 256,
                                                                  sink.data_ptr(), st.cuda_stream))
                 for k in range(4)]
        for k, ms in enumerate(times):
            lines.append(f"| {kinds[k]} | {ms:.3f} | {ms / times[0]:.2f} |")
    text = "\n".join(lines) + "\n"
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
    return 0


if __name__ == "__main__":
    sys.exit(main())
