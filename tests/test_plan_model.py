"""CPU checks of the decode kernel's work plan, on a model that restates the formulas of
`plan()`, `wave_of_step()`, `udiv_by()`/`div_magic()` and `split_geo()` in
paper_2609_24875_amd/csrc/sph_kernels.hip (no GPU involved):

- the multiply-high division `floor(x / d) = (x * m) >> k`, `m = ceil(2^k / d)`,
  `k = 31 + ceil(log2 d)`, is exact for every 0 <= x < 2^31 and 1 <= d < 2^31 (checked at the
  edges and at random);
- for both plans and many shapes, the wave ranges cover every step exactly once, `wave_of_step`
  inverts them, every tile meets at most `pmax` parts, a tile's parts inside one workgroup are
  exactly the waves `lw0 .. lw0 + nl - 1` the split-tile hand-over counts, and a local leader
  with other local parts to collect holds the last part of its own range (so it never waits
  inside its step loop).
"""
from __future__ import annotations

import random

import pytest

WPB = 16


def div_magic(d: int):
    l = 0
    while (1 << l) < d:
        l += 1
    k = 31 + l
    return ((1 << k) + d - 1) // d, k


def udiv(x: int, mk) -> int:
    m, k = mk
    assert 0 <= x < 2**31 and m < 2**32
    return (x * m) >> k


def test_magic_division_exact():
    rng = random.Random(0)
    ds = [1, 2, 3, 5, 7, 16, 17, 255, 256, 1000, 65535, 65536, 2**20 + 1, 2**30 - 1, 2**30, 2**30 + 1,
          2**31 - 1] + [rng.randrange(1, 2**31) for _ in range(200)]
    for d in ds:
        mk = div_magic(d)
        xs = {0, 1, d - 1, d, d + 1, 2**31 - 1, (2**31 - 1) // d * d, (2**31 - 1) // d * d - 1}
        xs |= {rng.randrange(0, 2**31) for _ in range(200)}
        for x in xs:
            if 0 <= x < 2**31:
                assert udiv(x, mk) == x // d, (x, d)


def plan(nt: int, nc: int, cus: int = 256, lds_fits: bool = True) -> dict:
    ts = nt * nc
    T = (nt + cus - 1) // cus
    gA = (nt + T - 1) // T
    lA = (T * nc + WPB - 1) // WPB
    gB = max(1, min(cus, ts // WPB))
    lB = (ts + gB * WPB - 1) // (gB * WPB)
    if lA <= lB and lds_fits:
        return dict(grid=gA, wg_tiles=T, wgs=T * nc, wl=lA, pmax=0, ts=ts, nc=nc, nt=nt)
    grid = ((ts + lB - 1) // lB + WPB - 1) // WPB
    return dict(grid=grid, wg_tiles=0, wgs=0, wl=lB, pmax=nc // lB + 2, ts=ts, nc=nc, nt=nt)


def ranges(P):
    """The kernel's wave ranges: [(wave id, s_begin, s_end)] for the non-empty ones."""
    out = []
    for b in range(P["grid"]):
        for w in range(WPB):
            g = b * WPB + w
            if P["wg_tiles"]:
                lim = min((b + 1) * P["wgs"], P["ts"])
                sb = b * P["wgs"] + w * P["wl"]
            else:
                lim = P["ts"]
                sb = g * P["wl"]
            se = min(sb + P["wl"], lim)
            if sb < lim:
                out.append((g, sb, se))
    return out


def wave_of_step(P, s):
    ml = div_magic(P["wl"])
    if P["wg_tiles"] == 0:
        return udiv(s, ml)
    b = udiv(s, div_magic(P["wgs"]))
    return b * WPB + udiv(s - b * P["wgs"], ml)


def check_plan(P):
    ts, nc = P["ts"], P["nc"]
    owner = [-1] * ts
    last = {}
    for g, sb, se in ranges(P):
        for s in range(sb, se):
            assert owner[s] == -1
            owner[s] = g
        last[g] = se - 1
    assert all(o >= 0 for o in owner)
    for s in range(ts):
        assert wave_of_step(P, s) == owner[s]
    for t in range(P["nt"]):
        gr, gl = owner[t * nc], owner[t * nc + nc - 1]
        holders = set(owner[t * nc:(t + 1) * nc])
        ngrp = gl // WPB - gr // WPB + 1
        if P["wg_tiles"]:
            assert ngrp == 1
        else:
            assert len(holders) <= P["pmax"] and ngrp <= P["pmax"]
        for b in range(gr // WPB, gl // WPB + 1):
            b0 = b * WPB
            lw0 = max(gr, b0)
            nl = min(gl, b0 + WPB - 1) - lw0 + 1
            assert {w for w in holders if w // WPB == b} == set(range(lw0, lw0 + nl))
            if nl > 1:
                assert last[lw0] // nc == t


SHAPES = [(320, 50), (320, 10), (448, 10), (3200, 10), (768, 16), (256, 24), (1, 64), (1, 128),
          (3, 17), (64, 8), (2817, 40), (64, 96), (32, 64), (5, 1), (1, 1), (17, 3), (1, 200)]


@pytest.mark.parametrize("nt,nc", SHAPES)
@pytest.mark.parametrize("lds_fits", [True, False])
def test_plan_invariants(nt, nc, lds_fits):
    check_plan(plan(nt, nc, lds_fits=lds_fits))


def test_plan_invariants_random_shapes():
    rng = random.Random(1)
    for _ in range(60):
        nt, nc = rng.randint(1, 3000), rng.randint(1, 120)
        check_plan(plan(nt, nc, lds_fits=rng.random() < 0.7))
