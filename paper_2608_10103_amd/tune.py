"""Interleaved timing of kernel variants (the library's tuning tool).

    python -m paper_2608_10103_amd.tune --dtypes f16,s8 --sizes 4096,8192 \
        --variants pipe256x256_w2x2_k128_s2,pipe256x256_w2x4_k128_s2 --rounds 7

For every (dtype, N) it runs each selected variant on the same seeded square
operands, round-robin for --rounds rounds (so clock drift under power limits
affects all variants alike), and prints the median time per launch, TOP/s,
the fraction of the variant's MFMA peak and whether its output equals the
first variant's (integers) or is within 1e-3 relative of it (FP16). Variant
names may be given as substrings; default: every tiled variant that supports
the shape. Correctness against the exact result is the tests' job; this tool
only times the library.
"""
from __future__ import annotations

import argparse
import json
import os
import sys

import numpy as np
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2608_10103_amd as mp  # noqa: E402
import seeded_inputs as si  # noqa: E402

PEAK = {"f16": 2500.0, "s8": 5000.0, "s4": 5000.0}
PEAK_FP6 = 10100.0


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--dtypes", default="f16,s8,s4")
    ap.add_argument("--sizes", default="8192")
    ap.add_argument("--variants", default="", help="comma-separated names or substrings")
    ap.add_argument("--rounds", type=int, default=5)
    ap.add_argument("--json", default="", help="write the results here")
    args = ap.parse_args(argv)
    want = [w for w in args.variants.split(",") if w]
    stream = torch.cuda.Stream()
    res = []
    for dt in args.dtypes.split(","):
        for n in (int(x) for x in args.sizes.split(",")):
            A, B = si.gen_operands(dt, n, n, n, seed=11)
            Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
            vs = []
            for v in range(mp.num_variants(dt)):
                name = mp.variant_name(dt, v)
                if v == 0 and n > 1024:
                    continue
                if want and not any(w in name for w in want):
                    continue
                if mp.variant_supports(dt, v, n, n, n, Ad.data_ptr(), Bd.data_ptr()):
                    vs.append((v, name))
            if not vs:
                continue
            out_dt = torch.float32 if dt == "f16" else torch.int32
            Cs = {v: torch.empty((n, n), dtype=out_dt, device="cuda") for v, _ in vs}
            reps = max(2, min(40, int(1e12 / (2 * n ** 3))))
            times = {v: [] for v, _ in vs}
            with torch.cuda.stream(stream):
                for v, _ in vs:
                    mp.GEMM[dt](Ad, Bd, C=Cs[v], stream=stream, variant=v)
                for _ in range(args.rounds):
                    for v, _ in vs:
                        e0 = torch.cuda.Event(enable_timing=True)
                        e1 = torch.cuda.Event(enable_timing=True)
                        e0.record(stream)
                        for _ in range(reps):
                            mp.GEMM[dt](Ad, Bd, C=Cs[v], stream=stream, variant=v)
                        e1.record(stream)
                        e1.synchronize()
                        times[v].append(e0.elapsed_time(e1) / reps)
            torch.cuda.synchronize()
            ref = Cs[vs[0][0]]
            base = float(np.median(times[vs[0][0]]))
            for v, name in vs:
                ms = float(np.median(times[v]))
                tops = 2 * n ** 3 / (ms * 1e-3) / 1e12
                peak = PEAK_FP6 if name.startswith("fp6") else PEAK[dt]
                if v == vs[0][0]:
                    same = "ref"
                elif dt == "f16":
                    same = "close" if bool((Cs[v] - ref).abs().max() <= 1e-3 * ref.abs().max()) else "DIFFERENT"
                else:
                    same = "identical" if torch.equal(Cs[v], ref) else "DIFFERENT"
                spread = 100 * (max(times[v]) - min(times[v])) / ms
                print(f"{dt} N={n:5d} v{v:2d} {name:32s} {ms * 1e3:9.1f} us {tops:8.1f} T/s "
                      f"{100 * tops / peak:5.1f}% of peak  rel {base / ms:5.3f}  spread {spread:4.1f}%  {same}",
                      flush=True)
                res.append(dict(dtype=dt, n=n, variant=v, name=name, us=ms * 1e3, tops=tops,
                                frac_peak=tops / peak, rel=base / ms, check=same))
            del Cs, Ad, Bd
            torch.cuda.empty_cache()
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
