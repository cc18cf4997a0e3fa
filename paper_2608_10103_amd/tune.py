"""Interleaved timing of kernel variants (the library's tuning tool).

    python -m paper_2608_10103_amd.tune --dtypes f16,s8 --sizes 4096,8192 \
        --variants pipe256x256_w2x2_k128_s2,pipe256x256_w2x4_k128_s2 --rounds 7
    python -m paper_2608_10103_amd.tune --dtypes s8 --shapes 16x8192x8192 \
        --variants spread128 --splits 1,2,4,8

For every (dtype, shape) it runs each selected variant (and, with --splits,
each split-K count a pipelined variant accepts) on the same seeded operands, round-robin for --rounds rounds (so clock drift under power limits
affects all variants alike), and prints the median time per launch, TOP/s,
the fraction of the variant's MFMA peak and whether its output equals the
first variant's (integers) or is within 1e-3 relative of it (FP16). Variant
names may be given as substrings; default: every tiled variant that supports
the shape. Correctness against the exact result is the tests' job; this tool
only times the library. --vendor adds the vendor library's GEMM on the same
operands (FP16: torch.matmul, half output; INT8: torch._int_mm) to the
rounds, as a yardstick for the same shapes; it is never part of the
library's own path.
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
    ap.add_argument("--sizes", default="8192", help="square sizes N")
    ap.add_argument("--shapes", default="", help="MxNxK,... (added to --sizes)")
    ap.add_argument("--splits", default="", help="split-K counts to try, e.g. 1,2,4 (default: automatic)")
    ap.add_argument("--variants", default="", help="comma-separated names or substrings")
    ap.add_argument("--rounds", type=int, default=5)
    ap.add_argument("--json", default="", help="write the results here")
    ap.add_argument("--vendor", action="store_true", help="also time the vendor library (FP16, INT8)")
    ap.add_argument("--transposed-b", action="store_true",
                    help="also time mpgemm_gemm_bt (B stored K x N row-major) on the same operands "
                         "(FP16, INT8, INT4)")
    args = ap.parse_args(argv)
    want = [w for w in args.variants.split(",") if w]
    stream = torch.cuda.Stream()
    res = []
    shapes = [(n, n, n) for n in (int(x) for x in args.sizes.split(",") if x)]
    shapes += [tuple(int(x) for x in sh.split("x")) for sh in args.shapes.split(",") if sh]
    split_list = [int(x) for x in args.splits.split(",") if x]
    for dt in args.dtypes.split(","):
        for (M, N, K) in shapes:
            A, B = si.gen_operands(dt, M, N, K, seed=11)
            Ad, Bd = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
            runs = []  # (variant, splits or None, label)
            for v in range(mp.num_variants(dt)):
                name = mp.variant_name(dt, v)
                if v == 0 and M * N * K > 1024 ** 3:
                    continue
                if want and not any((name == w[1:]) if w.startswith("=") else (w in name) for w in want):
                    continue
                if not mp.variant_supports(dt, v, M, N, K, Ad.data_ptr(), Bd.data_ptr()):
                    continue
                if not split_list:
                    # the automatic split of a call with a workspace (allocated here, once)
                    auto = mp.select_splits(dt, v, M, N, K)
                    runs.append((v, None, f"{name} (splits {auto})"))
                    continue
                for sp in split_list:
                    try:
                        mp.workspace_size(dt, M, N, K, variant=v, splits=sp)
                    except mp.HipError:
                        continue
                    runs.append((v, sp, f"{name} splits {sp}"))
            Bt = None
            if args.transposed_b:
                # the same B, K x N row-major (INT4: nibbles re-packed along N)
                if dt == "s4":
                    lo, hi = (B & 0xF).astype(np.int8), (B >> 4).astype(np.int8)
                    logical = np.empty((N, K), np.int8)
                    logical[:, 0::2] = np.where(lo >= 8, lo - 16, lo)
                    logical[:, 1::2] = np.where(hi >= 8, hi - 16, hi)
                    Bt = torch.from_numpy(si.pack_s4(np.ascontiguousarray(logical.T))).cuda()
                else:
                    Bt = Bd.t().contiguous()
                runs.append(("bt", None, "transposed B (mpgemm_gemm_bt)"))
            # (torch._int_mm takes more than 16 rows of A only)
            if args.vendor and (dt == "f16" or (dt == "s8" and M > 16)):
                runs.append(("vendor", None, "vendor library (A x B^T)"))
            if not runs:
                continue
            out_dt = torch.float32 if dt == "f16" else torch.int32
            Cs = [torch.empty((M, N), dtype=torch.float16 if (r[0] == "vendor" and dt == "f16") else out_dt,
                              device="cuda") for r in runs]
            reps = max(2, min(200, int(2e11 / (2 * M * N * K))))
            times = [[] for _ in runs]
            # each run's workspace (split K, FP6 pre-pass), zero-filled, allocated before timing
            wss = []
            for v, sp, _ in runs:
                n = mp.workspace_size(dt, M, N, K, variant=v, splits=sp) if isinstance(v, int) else 0
                wss.append(mp.new_workspace(n, "cuda") if n else None)

            def call(i):
                v, sp, _ = runs[i]
                if v == "bt":
                    mp.gemm_bt(dt, Ad, Bt, C=Cs[i], stream=stream)
                elif v == "vendor":
                    if dt == "f16":
                        torch.matmul(Ad, Bd.t(), out=Cs[i])
                    else:
                        torch._int_mm(Ad, Bd.t(), out=Cs[i])
                else:
                    mp.GEMM[dt](Ad, Bd, C=Cs[i], stream=stream, variant=v, splits=sp, workspace=wss[i])

            with torch.cuda.stream(stream):
                for i in range(len(runs)):
                    call(i)
                for _ in range(args.rounds):
                    for i in range(len(runs)):
                        e0 = torch.cuda.Event(enable_timing=True)
                        e1 = torch.cuda.Event(enable_timing=True)
                        e0.record(stream)
                        for _ in range(reps):
                            call(i)
                        e1.record(stream)
                        e1.synchronize()
                        times[i].append(e0.elapsed_time(e1) / reps)
            torch.cuda.synchronize()
            ref = Cs[0]
            base = float(np.median(times[0]))
            for i, (v, sp, label) in enumerate(runs):
                ms = float(np.median(times[i]))
                tops = 2 * M * N * K / (ms * 1e-3) / 1e12
                name = {"bt": "transposed_b", "vendor": "vendor"}.get(v) if isinstance(v, str) else mp.variant_name(dt, v)
                peak = PEAK_FP6 if name.startswith(("fp6", "e2m3")) else PEAK[dt]
                if i == 0:
                    same = "ref"
                elif dt == "f16":
                    same = "close" if bool((Cs[i].float() - ref).abs().max() <= 1e-3 * ref.abs().max()) else "DIFFERENT"
                else:
                    same = "identical" if torch.equal(Cs[i], ref) else "DIFFERENT"
                spread = 100 * (max(times[i]) - min(times[i])) / ms
                vtag = {"bt": "bt", "vendor": "vd"}.get(v) if isinstance(v, str) else f"{v:2d}"
                print(f"{dt} {M}x{N}x{K} v{vtag} {label:44s} {ms * 1e3:9.1f} us {tops:8.1f} T/s "
                      f"{100 * tops / peak:5.1f}% of peak  rel {base / ms:5.3f}  spread {spread:4.1f}%  {same}",
                      flush=True)
                res.append(dict(dtype=dt, M=M, N=N, K=K, variant=v, name=name, splits=sp, us=ms * 1e3,
                                tops=tops, frac_peak=tops / peak, rel=base / ms, check=same))
            del Cs, Ad, Bd, Bt
            torch.cuda.empty_cache()
    if args.json:
        with open(args.json, "w") as f:
            json.dump(res, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
