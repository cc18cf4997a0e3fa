"""Pins taken from values the paper prints (fixtures under tests/golden/)."""
import csv
import os

import pytest

import bench

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rows(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return list(csv.DictReader(line for line in f if not line.startswith("#")))


ROWS = _rows("paper_table2_headline_tops.csv")


def test_fixture_is_complete():
    assert [r["kernel"] for r in ROWS] == ["fp16_wmma", "int8_wmma", "int8_ptx_mma_k32", "int4_wmma",
                                          "int4_ptx_3stage", "int4_ptx_mma_k64"]


@pytest.mark.parametrize("row", ROWS, ids=[r["kernel"] for r in ROWS])
def test_operation_count_reproduces_paper_tops(row):
    # Table II prints each duration to its last digit and TOPS to three
    # decimals; the count must reproduce TOPS within those two roundings.
    n, ms, tops = int(row["n"]), float(row["duration_ms"]), float(row["tops"])
    digits = len(row["duration_ms"].split(".")[1]) if "." in row["duration_ms"] else 0
    half_ulp_ms = 0.5 * 10.0 ** (-digits)
    got = bench.gemm_ops(n, n, n) / (ms * 1e-3) / 1e12
    assert abs(got - tops) <= 0.0005 + got * half_ulp_ms / ms + 1e-12
    # counting one operation per (i, j, k) term, or four, is off by a factor
    # of two and fails
    for wrong in (bench.gemm_ops(n, n, n) / 2, bench.gemm_ops(n, n, n) * 2):
        assert abs(wrong / (ms * 1e-3) / 1e12 - tops) > 0.01


def test_operation_count_is_per_term():
    assert bench.gemm_ops(1, 1, 1) == 2.0
    assert bench.gemm_ops(3, 5, 7) == 2.0 * 3 * 5 * 7
    assert bench.gemm_ops(0, 5, 7) == 0.0
