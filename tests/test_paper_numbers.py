"""The paper's printed arithmetic, reproduced from the oracle's counts
(CPU): the 32x amplification and the 128 / 16 requests per tile come from
oracle.read_amp, not from the fixture, so a change in the model that breaks
the paper's figures fails here."""
import pytest

import oracle
from oracle import KN_ROW, TILE
from tests._golden import load

G = 4096


def test_bandwidth_waste_section_2_5():
    g = load("paper_numbers.txt")
    # a 128-byte-wide compute tile (64 BF16) over a matrix with >= 4 KB rows
    # KN_ROW: N contiguous, 2048 BF16 = 4 KB per row; the tile is 64 wide along N
    amp = oracle.read_amp(1, 2048, 64, 1, 64, 64, KN_ROW, G)["amp"]
    assert amp == g["amplification"]
    mib = g["h200_sms"] * g["smem_kib_per_sm"] * amp / 1024
    assert mib == g["amplified_mib"]


def test_outstanding_requests_section_6_4():
    g = load("paper_numbers.txt")
    row = oracle.read_amp(1, 2048, 2048, 1, 256, 128, KN_ROW, G)["max_blocks_per_tile"]
    tm = oracle.read_amp(1, 2048, 2048, 1, 256, 128, TILE, G, layout_G=G, block_rows=32)["max_blocks_per_tile"]
    assert (row, tm) == (g["row_major_requests"], g["tile_major_requests"])
    extra = row - tm
    assert extra == g["extra_requests"] and extra * G // 1024 == g["extra_kib"]
    us = extra * G / (g["bus_tbps"] * 1e12) * 1e6
    assert us == pytest.approx(g["extra_us"], abs=0.005)


def test_memory_stacks_section_6_1():
    g = load("paper_numbers.txt")
    tbps = g["stacks"] * g["channels_per_stack"] * g["pins_per_channel"] * g["gbps_per_pin"] / 8 / 1000
    assert tbps == pytest.approx(g["total_tbps"], abs=5e-4)
