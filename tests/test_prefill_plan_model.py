"""CPU checks of the prefill kernel's K split, on a model that restates `prefill_plan()`,
`small_on_prefill()`, the kernel's range bounds and partial-output indices, and the split-K
reduce's 16-byte accesses in paper_2609_24875_amd/csrc/sph_kernels.hip (no GPU involved):

- every K range is non-empty and the ranges cover the chunks exactly once, in order;
- the split never needs more than one round of workgroups on the CUs (unless the grid alone is
  larger) and never more than 16 ranges;
- every partial output the kernel writes and every 16-byte group the reduce reads or clears lies
  inside the workspace the plan sizes, 16-byte aligned, and the reduce covers each written
  partial exactly once;
- batches 9..16 go to the prefill kernel exactly from 120 * 2^20 weights.
"""
from __future__ import annotations

import random

import pytest

PF_WAVES, PF_TPW, PF_KS_MAX = 8, 2, 16


def prefill_mc(m: int) -> int:
    return 16 if m <= 16 else 32 if m <= 32 else 64


def prefill_plan(n: int, k: int, m: int, cus: int = 256) -> dict:
    nt, ng = (n + 15) // 16, k // 128
    mc = prefill_mc(m)
    gx = (nt + PF_WAVES * PF_TPW - 1) // (PF_WAVES * PF_TPW)
    gy = (m + mc - 1) // mc
    g = gx * gy
    ks = max(1, min(cus // g, ng, PF_KS_MAX))
    ws = ks * m * nt * 16 * 4 if ks > 1 else 0
    return dict(nt=nt, ng=ng, mc=mc, gx=gx, gy=gy, ks=ks, ws=ws)


def small_on_prefill(n: int, k: int, m: int) -> bool:
    if m > 16:
        return True
    if m < 9:
        return False
    return n * k >= 120 << 20


def check(n: int, k: int, m: int, cus: int = 256):
    P = prefill_plan(n, k, m, cus)
    nt, ng, ks = P["nt"], P["ng"], P["ks"]
    assert 1 <= ks <= PF_KS_MAX and ks <= ng
    assert P["gx"] * P["gy"] * ks <= max(cus, P["gx"] * P["gy"])
    # K ranges of blockIdx.z: [nc z / ks, nc (z + 1) / ks)
    bounds = [(ng * z // ks, ng * (z + 1) // ks) for z in range(ks)]
    assert bounds[0][0] == 0 and bounds[-1][1] == ng
    for (a0, a1), (b0, _) in zip(bounds, bounds[1:]):
        assert a1 == b0
    assert all(c1 > c0 for c0, c1 in bounds)
    if ks == 1:
        return
    # partials written: z < ks, batch rows b < m, rows of tiles t < nt (all 16 rows of a tile)
    npad = nt * 16
    floats = P["ws"] // 4
    last = ((ks - 1) * m + (m - 1)) * npad + npad - 1
    assert last < floats
    # the reduce: thread t < m * npad / 4 reads f32x4 at float offset (z m + b) npad + 4 (t % nq)
    nq = npad // 4
    covered = 0
    for t in range(0, m * nq, max(1, (m * nq) // 257)):
        b, row = t // nq, (t % nq) * 4
        for z in range(ks):
            off = (z * m + b) * npad + row
            assert off % 4 == 0 and off + 3 < floats
        covered += 1
    assert covered > 0
    # each written partial belongs to exactly one (thread, component): rows are whole quads
    assert npad % 4 == 0


SHAPES = [(87, 640, 33), (300, 2048, 100), (16, 128, 64), (1, 256, 129), (12288, 4096, 32),
          (4096, 12288, 32), (4096, 12288, 24), (5120, 25600, 16), (51200, 5120, 16),
          (24576, 4096, 256), (1024, 2048, 17), (64, 4096, 40), (6144, 4096, 256), (17, 128, 17)]


@pytest.mark.parametrize("n,k,m", SHAPES)
def test_prefill_split_invariants(n, k, m):
    check(n, k, m)


def test_prefill_split_random_shapes():
    rng = random.Random(7)
    for _ in range(200):
        n = rng.randint(1, 60000)
        k = 128 * rng.randint(1, 200)
        m = rng.choice([9, 12, 16, 17, 24, 32, 33, 64, 65, 128, 256, 1000])
        check(n, k, m, cus=rng.choice([256, 304, 80]))


def test_split_ranges_never_exceed_the_reduce_limit():
    # the reduce keeps up to 16 ranges in registers; the smallest grids split the most
    for n, k in [(1, 128 * 64), (16, 128 * 200), (256, 128 * 100)]:
        P = prefill_plan(n, k, 17)
        assert P["ks"] == min(16, k // 128, 256 // (P["gx"] * P["gy"]))


def test_batch_9_to_16_routing_bound():
    bound = 120 << 20
    assert not small_on_prefill(24576, 4096, 16)          # 96 * 2^20: tile mode
    assert small_on_prefill(5120, 25600, 9)               # 125 * 2^20: prefill
    assert small_on_prefill(32768, 4096, 12)
    assert not small_on_prefill(51200, 5120, 8)           # batches up to 8 never
    assert small_on_prefill(16, 128, 17)                  # above 16 always
    for m in range(9, 17):
        assert small_on_prefill(1, bound, m) and not small_on_prefill(1, bound - 128, m)
