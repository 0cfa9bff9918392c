"""The benchmark's byte and FLOP accounting reproduces the paper's Table 1 (roofline of the pi0.5 MLPs)."""
import os

import pytest

import bench

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "roofline_table1.txt")


def _rows():
    rows = []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        name, d, d_ff, tok, gflop, mb, ai, c4090, m4090, cthor, mthor = line.split()
        rows.append((name, int(d), int(d_ff), int(tok), gflop, mb, ai, c4090, m4090, cthor, mthor))
    return rows


def _matches(value, printed, slack=0.0):
    """value rounds to the printed figure (half a unit of its last digit, plus slack)."""
    decimals = len(printed.split(".")[1]) if "." in printed else 0
    return abs(value - float(printed)) <= 0.5 * 10.0 ** -decimals + slack + 1e-12


@pytest.mark.parametrize("row", _rows(), ids=lambda r: r[0])
def test_table1_row(row):
    name, d, d_ff, tok, gflop, mb, ai, c4090, m4090, cthor, mthor = row
    flops = bench.projection_flops(tok, d, d_ff)
    nbytes = bench.matrix_bytes(d, d_ff, 2)
    mb_count = nbytes / 2 ** 20           # the table's MB column counts 2^20-byte units ...
    assert _matches(flops / 1e9, gflop)
    assert _matches(mb_count, mb)
    mb_dec = float(mb) * 1e6              # ... and its AI and T_mem take each printed MB as 10^6 bytes
    assert _matches(flops / mb_dec, ai, slack=0.5)
    # T_comp = FLOP / peak FLOP/s, T_mem = bytes / peak B/s, in microseconds.  The VLM row's printed 4090
    # T_comp (345.3) sits 0.4 below 57.04 GFLOP / 165 TFLOP/s = 345.7; allowed as a rounding slip.
    assert _matches(float(gflop) * 1e9 / 165e12 * 1e6, c4090, slack=0.45)
    assert _matches(mb_dec / 1000e9 * 1e6, m4090)
    assert _matches(float(gflop) * 1e9 / 250e12 * 1e6, cthor)
    assert _matches(mb_dec / 270e9 * 1e6, mthor)


def test_action_layer_bytes():
    # One action-expert layer = three such projections; at 30% of 4096 neurons (K = 1229) in bf16:
    assert bench.active_weight_bytes(1229, 1024, 2) == 3 * 1229 * 1024 * 2 == 7_550_976
    assert bench.gateup_bytes(1229, 1024, 2) == 2 * bench.down_bytes(1229, 1024, 2)
    assert bench.active_weight_bytes(4096, 1024, 2) == 3 * bench.matrix_bytes(1024, 4096, 2)
