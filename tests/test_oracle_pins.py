"""Pins of the fp64 oracle against what the paper and mathematics fix.

Each ``pin_*`` function checks one part of the oracle against something other than
itself: values the paper prints (golden fixtures with citations), closed forms,
invariants, library routines for special cases, exact rational arithmetic, and brute
force over every code of tiny codebooks. ``test_mutants_are_caught`` plants plausible
mistakes in a copy of the oracle and requires that some pin fails for each.
"""
from __future__ import annotations

import itertools
import types
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import sph as O
from tests.conftest import read_golden


def _ns(**override):
    ns = types.SimpleNamespace(**{k: getattr(O, k) for k in dir(O) if not k.startswith("__")})
    for k, v in override.items():
        setattr(ns, k, v)
    return ns


# A codebook of exactly-unit, non-negative 8-D directions: the 8 axes and the 56 first
# 4-subsets of coordinates at 1/2 (4 * 1/4 = 1). All values are exact in fp16.
def exact_unit_codebook(entries=64):
    rows = [np.eye(8)[j] for j in range(8)]
    for sub in itertools.combinations(range(8), 4):
        v = np.zeros(8)
        v[list(sub)] = 0.5
        rows.append(v)
    return synth.f16_bits(np.array(rows[:entries]))


# ------------------------------------------------------------------------- pins

def pin_worked_radius(o):
    """Sec. 1: radius of (1,..,1) is 2*sqrt(2); with one coordinate at 5 it is 4*sqrt(2)."""
    for coords, mult in read_golden("worked_radius.txt"):
        w = np.array([float(t) for t in coords.split()])
        r_sph, _ = o.spherical_coordinates(w)
        _, _, r_dec, _ = o.decompose(w)
        want = float(mult) * np.sqrt(2.0)
        assert abs(r_sph - want) < 1e-14 and abs(r_dec - want) < 1e-14


def pin_spherical_roundtrip(o):
    """Eq. 1 round trip through the textbook inverse, and the angle ranges."""
    g = np.random.default_rng(1)
    w = g.standard_normal((500, 8))
    r, phi = o.spherical_coordinates(w)
    assert np.allclose(o.from_spherical(r, phi), w, atol=1e-12)
    assert np.all(phi[:, :6] >= 0) and np.all(phi[:, :6] <= np.pi)
    assert np.allclose(r, np.linalg.norm(w, axis=1), rtol=1e-14)


def pin_bit_budget(o):
    """Storage figures of Sec. 1, 3.1, 3.2, 4.1, App. B, Tab. 7 and Tab. 12."""
    for key, args, want, _src in read_golden("bit_budget.txt"):
        a = dict(t.split("=") for t in args.split())
        a = {k: int(v) for k, v in a.items()}
        want = float(want)
        if key == "dir_bits":
            got = o.dir_bits_for(a["B"], a["dim"])
        elif key == "codebook_bytes":
            got = o.codebook_bytes(a["D"], a["dim"], bool(a["signed"]))
        elif key == "codebook_bytes_tab7":
            got = o.codebook_bytes(o.dir_bits_for(a["B"], a["dim"]), a["dim"])
        elif key == "payload":
            got = o.payload_bits_per_weight(a["B"], a["V"])
        elif key == "extra_payload_pct":
            got = 100.0 * (o.payload_bits_per_weight(a["B"], a["V"]) / a["B"] - 1.0)
        else:
            raise AssertionError(key)
        assert abs(got - want) < 1e-12, (key, args, got, want)


def pin_decompose(o):
    """Eq. 3: w = r * s (.) d exactly up to rounding, d on the positive unit sphere, sign of
    zero is +, and the zero vector gets r = 0 and d = 0."""
    g = np.random.default_rng(2)
    w = g.standard_normal((300, 8)) * np.exp(g.standard_normal((300, 1)))
    neg, wp, r, d = o.decompose(w)
    s = np.where(neg, -1.0, 1.0)
    assert np.allclose(r[:, None] * s * d, w, rtol=1e-14, atol=1e-300)
    assert np.all(d >= 0) and np.allclose(np.linalg.norm(d, axis=1), 1.0, atol=1e-14)
    assert np.array_equal(wp, np.abs(w))
    neg0, _, r0, d0 = o.decompose(np.array([0.0, -0.0, 1.0, 0, 0, 0, 0, -2.0]))
    assert list(neg0) == [False, False, False, False, False, False, False, True]
    _, _, rz, dz = o.decompose(np.zeros(8))
    assert rz == 0 and np.all(dz == 0)


def pin_assign(o):
    """Eq. 5: the direction of a codebook entry is assigned to that entry; the cosine
    argmax is the nearest entry in angle (checked by brute-force arccos); ties -> lowest."""
    g = np.random.default_rng(3)
    cb = synth.random_codebook(6, g)
    c = O.f16_to_f64(cb)
    own = c / np.linalg.norm(c, axis=1, keepdims=True)
    assert np.array_equal(o.assign_directions(own, c), np.arange(64))
    d = np.abs(g.standard_normal((400, 8)))
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    z = o.assign_directions(d, c)
    cn = c / np.linalg.norm(c, axis=1, keepdims=True)
    ang = np.arccos(np.clip(d @ cn.T, -1, 1))
    # Entries are not exactly unit after fp16; the cosine argmax may differ from the angle
    # argmin only when two angles agree to within the norm error.
    best = ang.min(axis=1)
    assert np.all(ang[np.arange(400), z] <= best + 2e-3)
    dup = np.vstack([c[:3], c[1:2], c[3:]])
    assert o.assign_directions(own[1:2], dup)[0] == 1


def pin_ls_radius(o):
    """Eq. 6: <w_+, c> is the least-squares scale along a unit c (checked with lstsq on
    exactly-unit entries) and never exceeds ||w_+|| (Cauchy-Schwarz)."""
    g = np.random.default_rng(4)
    c = O.f16_to_f64(exact_unit_codebook(64))
    for _ in range(50):
        wp = np.abs(g.standard_normal(8))
        cz = c[g.integers(0, 64)]
        alpha = np.linalg.lstsq(cz[:, None], wp, rcond=None)[0][0]
        assert abs(o.ls_radius(wp, cz) - alpha) < 1e-13
        assert o.ls_radius(wp, cz) <= np.linalg.norm(wp) + 1e-15
        assert o.ls_radius(wp, cz) >= 0


def pin_radius_quant(o):
    """Eq. 7 on a grid: radii min + j*Delta get levels j and their own (min, Delta) back;
    values outside [min, max] clip; a zero step gives level 0; V = 3 has 8 levels."""
    for v_bits, lo, step in ((4, 0.5, 0.125), (3, 0.25, 0.0625), (2, 1.0, 0.5), (8, 0.0, 2**-6)):
        grid = lo + np.arange(16) % (1 << v_bits) * step
        grid[0], grid[-1] = lo, lo + ((1 << v_bits) - 1) * step
        gmin, gstep = o.group_offset_step(grid[None, :], v_bits)
        assert O.f16_to_f64(gmin)[0] == lo and O.f16_to_f64(gstep)[0] == step
        q = o.quantize_radius(grid[None, :], gmin, gstep, v_bits)[0]
        want = np.arange(16) % (1 << v_bits)
        want[-1] = (1 << v_bits) - 1
        assert np.array_equal(q, want), (v_bits, q, want)
        out = o.quantize_radius(np.array([[lo - 5 * step, lo + ((1 << v_bits) + 50) * step]]), gmin, gstep, v_bits)
        assert list(out[0]) == [0, (1 << v_bits) - 1]
        r_hat = o.dequantize_radius(q[None, :].astype(np.uint8),
                                    np.array([gmin]), np.array([gstep]))[0]
        assert np.array_equal(r_hat, grid)
    gmin, gstep = o.group_offset_step(np.full((1, 16), 0.75), 4)
    assert O.f16_to_f64(gstep)[0] == 0
    assert np.all(o.quantize_radius(np.full((1, 16), 0.75), gmin, gstep, 4) == 0)


def pin_decode_norm_and_sign(o):
    """Eq. 4: ||w^|| = r^ ||c_z|| and sign(w^_j) = s_j wherever c_z,j > 0."""
    g = np.random.default_rng(5)
    cb = synth.random_codebook(6, g)
    codes = synth.uniform_codes(8, 256, 6, 4, g)
    codes["gmin"], codes["gstep"] = synth.row_scale_group_params(8, 256, 4, g)
    w = o.decode(codes, cb).reshape(8, 32, 8)
    c = O.f16_to_f64(cb)
    r_hat = o.dequantize_radius(codes["q"], codes["gmin"], codes["gstep"])
    norms = np.linalg.norm(c[codes["dir"].astype(int)], axis=-1)
    assert np.allclose(np.linalg.norm(w, axis=-1), r_hat * norms, rtol=1e-14)
    bits = (codes["signs"][..., None] >> np.arange(8)) & 1
    assert np.all((w < 0) == (bits == 1))


def pin_decode_one_hot(o):
    """Eq. 4 with the axis codebook c_k = e_(k mod 8): every vector has one non-zero,
    +-r^ at coordinate z mod 8 (written out by hand below)."""
    g = np.random.default_rng(6)
    cb = synth.f16_bits(np.eye(8)[np.arange(16) % 8])
    n, k = 3, 256
    codes = synth.uniform_codes(n, k, 4, 4, g)
    codes["gmin"], codes["gstep"] = synth.row_scale_group_params(n, k, 4, g)
    w = o.decode(codes, cb)
    for r in range(n):
        for v in range(k // 8):
            s = int(codes["signs"][r, v])
            z = int(codes["dir"][r, v])
            grp = v // 16
            rh = O.f16_to_f64(codes["gmin"][r, grp]) + int(codes["q"][r, v]) * \
                O.f16_to_f64(codes["gstep"][r, grp])
            want = np.zeros(8)
            j = z % 8
            want[j] = -rh if (s >> j) & 1 else rh
            assert np.array_equal(w[r, 8 * v:8 * v + 8], want)


def pin_gemm_exact_rational(o):
    """Y = W^ x against exact rational arithmetic (every fp16 input is a dyadic rational),
    one scalar term at a time; the oracle must agree within a few fp64 roundings."""
    g = np.random.default_rng(7)
    n, k, m = 3, 256, 2
    cb = synth.random_codebook(6, g)
    codes = synth.uniform_codes(n, k, 6, 4, g)
    codes["gmin"], codes["gstep"] = synth.row_scale_group_params(n, k, 4, g)
    codes["gmin"][1, 0] = synth.f16_bits([-0.375])[0]      # a negative offset is accepted too
    x = synth.activations(m, k, g)
    y = o.gemm(codes, cb, x)
    fr = lambda b: Fraction(float(O.f16_to_f64(b)))  # noqa: E731
    for b in range(m):
        for r in range(n):
            acc = Fraction(0)
            bound = 0.0
            for col in range(k):
                v, j = divmod(col, 8)
                grp = col // 128
                radius = fr(codes["gmin"][r, grp]) + int(codes["q"][r, v]) * fr(codes["gstep"][r, grp])
                sgn = -1 if (int(codes["signs"][r, v]) >> j) & 1 else 1
                term = radius * sgn * fr(cb[int(codes["dir"][r, v]), j]) * fr(x[b, col])
                acc += term
                bound += abs(float(term))
            assert abs(y[b, r] - float(acc)) <= 8 * k * 2.0**-53 * bound + 1e-300


def pin_gemm_special_cases(o):
    """x = e_col returns column col of W^; a zero step with the exact direction
    (1/2,1/2,1/2,1/2,0,0,0,0) and positive signs gives y = min/2 * (sum of x_j, j<4 per vector)."""
    g = np.random.default_rng(8)
    n, k = 5, 384
    cb = synth.random_codebook(4, g)
    codes = synth.uniform_codes(n, k, 4, 4, g)
    codes["gmin"], codes["gstep"] = synth.row_scale_group_params(n, k, 4, g)
    w = o.decode(codes, cb)
    for col in (0, 7, 8, 200, 383):
        e = np.zeros((1, k))
        e[0, col] = 1.0
        assert np.array_equal(o.gemm(codes, cb, synth.f16_bits(e))[0], w[:, col])
    half = np.zeros((16, 8))
    half[:, :4] = 0.5
    codes2 = {"signs": np.zeros((n, k // 8), np.uint8), "dir": codes["dir"],
              "q": codes["q"], "gmin": codes["gmin"],
              "gstep": np.zeros_like(codes["gstep"])}
    x = synth.activations(2, k, g)
    xf = O.f16_to_f64(x)
    y = o.gemm(codes2, synth.f16_bits(half), x)
    mins = O.f16_to_f64(codes["gmin"])[:, 0]
    want = mins[None, :] * 0.5 * xf.reshape(2, k // 8, 8)[:, :, :4].sum(axis=(1, 2))[:, None]
    assert np.allclose(y, want, rtol=1e-13)


def _all_codes(dir_bits, radius_bits, k=128):
    combos = np.array(list(itertools.product(range(256), range(1 << dir_bits),
                                             range(1 << radius_bits))), dtype=np.int64)
    nvec = combos.shape[0]
    per_row = k // 8
    n = -(-nvec // per_row)
    pad = n * per_row - nvec
    combos = np.vstack([combos, np.zeros((pad, 3), np.int64)])
    return {"signs": combos[:, 0].astype(np.uint8).reshape(n, per_row),
            "dir": combos[:, 1].astype(np.uint16).reshape(n, per_row),
            "q": combos[:, 2].astype(np.uint8).reshape(n, per_row)}


def pin_encode_roundtrip_bruteforce(o):
    """decode then encode returns the same codes, for every (sign byte, direction, level)
    of tiny codebooks (D = 2, 4, 6; V = 4 and 3) with fixed group parameters."""
    for d_bits, v_bits in ((2, 4), (4, 4), (6, 4), (4, 3)):
        g = np.random.default_rng(10 + d_bits)
        cb = synth.random_codebook(d_bits, g)
        assert np.all(O.f16_to_f64(cb) > 0)
        codes = _all_codes(d_bits, v_bits)
        n = codes["q"].shape[0]
        gmin = np.full((n, 1), synth.f16_bits(0.5), np.uint16)
        gstep = np.full((n, 1), synth.f16_bits(0.1), np.uint16)
        codes["gmin"], codes["gstep"] = gmin, gstep
        w = o.decode(codes, cb)
        back = o.encode(w, cb, v_bits, params=(gmin, gstep))
        for key in ("signs", "dir", "q"):
            assert np.array_equal(back[key], codes[key]), (d_bits, v_bits, key)


def pin_encode_group_params_recovered(o):
    """With exactly-unit directions and every group using both extreme levels, the
    data-derived (min, Delta) of Eq. 7 are the ones that generated the radii, and the codes
    come back (signs canonicalised to + where the direction coordinate is 0)."""
    g = np.random.default_rng(20)
    cb = exact_unit_codebook(64)
    c = O.f16_to_f64(cb)
    n, k, v_bits = 6, 512, 4
    codes = synth.uniform_codes(n, k, 6, v_bits, g)
    q = codes["q"].reshape(n, k // 128, 16)
    q[..., 0], q[..., 5] = 0, 15
    codes["q"] = q.reshape(n, k // 8)
    lo = np.array([0.5, 0.25, 1.0, 2.0, 0.125, 0.75])
    codes["gmin"] = synth.f16_bits(np.repeat(lo[:, None], k // 128, axis=1))
    codes["gstep"] = synth.f16_bits(np.repeat((lo / 8)[:, None], k // 128, axis=1))
    back = o.encode(o.decode(codes, cb), cb, v_bits)
    zero = c[codes["dir"].astype(int)] == 0
    bits = (codes["signs"][..., None] >> np.arange(8)) & 1
    canon = ((bits * ~zero) << np.arange(8)).sum(axis=-1).astype(np.uint8)
    assert np.array_equal(back["signs"], canon)
    for key in ("dir", "q", "gmin", "gstep"):
        assert np.array_equal(back[key], codes[key]), key


def pin_vector_dims(o):
    """Tab. 7's 4-D and 16-D vectors through the same encoder and decoder: every (4 sign bits,
    direction, level) code of a 4-entry 4-D codebook with 3 radius bits comes back from
    decode then encode; 16-D codes (16 sign bits, 14-bit direction, 6 radius bits) come back
    likewise; decoded vectors have norm r^ ||c_z|| and the code's signs; and with exactly-unit
    4-D axes and both extreme levels in every 32-vector group, Eq. 7's parameters are recovered."""
    g = np.random.default_rng(30)
    cb4 = synth.random_codebook(2, g, dim=4)
    combos = np.array(list(itertools.product(range(16), range(4), range(8))), dtype=np.int64)
    n4 = combos.shape[0] // 32
    codes = {"signs": combos[:, 0].astype(np.uint8).reshape(n4, 32),
             "dir": combos[:, 1].astype(np.uint16).reshape(n4, 32),
             "q": combos[:, 2].astype(np.uint8).reshape(n4, 32),
             "gmin": np.full((n4, 1), synth.f16_bits(0.5), np.uint16),
             "gstep": np.full((n4, 1), synth.f16_bits(0.1), np.uint16)}
    w = o.decode(codes, cb4)
    assert w.shape == (n4, 128)
    back = o.encode(w, cb4, 3, params=(codes["gmin"], codes["gstep"]))
    for key in ("signs", "dir", "q"):
        assert np.array_equal(back[key], codes[key]), ("4d", key)
    cb16 = synth.random_codebook(14, g, dim=16)
    n16 = 6
    c16 = {"signs": g.integers(0, 1 << 16, (n16, 16)).astype(np.uint16),
           "dir": g.integers(0, 1 << 14, (n16, 16)).astype(np.uint16),
           "q": g.integers(0, 64, (n16, 16)).astype(np.uint8),
           "gmin": np.full((n16, 2), synth.f16_bits(0.25), np.uint16),
           "gstep": np.full((n16, 2), synth.f16_bits(0.03125), np.uint16)}
    w16 = o.decode(c16, cb16)
    assert w16.shape == (n16, 256)
    back = o.encode(w16, cb16, 6, params=(c16["gmin"], c16["gstep"]))
    for key in ("signs", "dir", "q"):
        assert np.array_equal(back[key], c16[key]), ("16d", key)
    rh = 0.25 + c16["q"] * 0.03125
    cz = O.f16_to_f64(cb16)[c16["dir"].astype(np.int64)]
    v = w16.reshape(n16, 16, 16)
    assert np.allclose(np.linalg.norm(v, axis=2), rh * np.linalg.norm(cz, axis=2), rtol=1e-14)
    sbits = (c16["signs"][..., None].astype(np.int64) >> np.arange(16)) & 1
    assert np.array_equal(np.signbit(v), sbits.astype(bool))
    axes = synth.f16_bits(np.eye(4))
    n, k = 5, 256
    cg = synth.uniform_codes(n, k, 2, 3, g)
    cg["signs"] = g.integers(0, 16, (n, k // 4)).astype(np.uint8)
    cg["dir"] = g.integers(0, 4, (n, k // 4)).astype(np.uint16)
    q = g.integers(0, 8, (n, k // 4)).reshape(n, 2, 32)
    q[..., 3], q[..., 17] = 0, 7
    cg["q"] = q.reshape(n, k // 4).astype(np.uint8)
    lo = np.array([0.5, 0.25, 1.0, 2.0, 0.125])
    cg["gmin"] = synth.f16_bits(np.repeat(lo[:, None], 2, axis=1))
    cg["gstep"] = synth.f16_bits(np.repeat((lo / 4)[:, None], 2, axis=1))
    back = o.encode(o.decode(cg, axes), axes, 3)
    zero = np.eye(4)[cg["dir"].astype(int)] == 0
    bits = (cg["signs"][..., None] >> np.arange(4)) & 1
    canon = ((bits * ~zero) << np.arange(4)).sum(axis=-1).astype(np.uint8)
    assert np.array_equal(back["signs"], canon)
    for key in ("dir", "q", "gmin", "gstep"):
        assert np.array_equal(back[key], cg[key]), ("4d groups", key)


def pin_w2_layout(o):
    """Sec. 3.4 / App. D / Fig. 3b field positions, on hand-worked words; plus a bit-exact
    pack/unpack round trip on random codes."""
    rows = read_golden("w2_layout.txt")
    for fields, want in rows:
        vals = fields.split()
        if len(vals) == 3:
            s, d, q = int(vals[0], 0), int(vals[1]), int(vals[2])
            sig = np.zeros((1, 16), np.uint8)
            dd = np.zeros((1, 16), np.uint16)
            qq = np.zeros((1, 16), np.uint8)
            sig[0, 0], dd[0, 0], qq[0, 0] = s, d, q
            base, _ = o.paper_pack_w2(sig, dd, qq)
            assert int(base[0, 0]) == int(want, 16), (fields, hex(int(base[0, 0])))
        else:
            qq = np.array([[int(t) for t in vals]], np.uint8)
            _, aux = o.paper_pack_w2(np.zeros((1, 16), np.uint8), np.zeros((1, 16), np.uint16), qq)
            assert int(aux[0, 0]) == int(want, 16), (fields, hex(int(aux[0, 0])))
    g = np.random.default_rng(30)
    codes = synth.uniform_codes(7, 512, 6, 4, g)
    base, aux = o.paper_pack_w2(codes["signs"], codes["dir"], codes["q"])
    assert base.dtype == np.uint16 and aux.shape == (7, 4)
    s, d, q = o.paper_unpack_w2(base, aux)
    assert np.array_equal(s, codes["signs"]) and np.array_equal(d, codes["dir"])
    assert np.array_equal(q, codes["q"])


def pin_angular_codebook(o):
    """Eq. 9/10: unit norm and strictly positive entries for any logits; the angles that
    give the uniform direction (1/sqrt 8, ...) produce it; theta = 0 gives the first axis."""
    g = np.random.default_rng(40)
    phi = g.standard_normal((1000, 7)) * 4
    th = o.angles_from_logits(phi)
    assert np.all(th > 0) and np.all(th < np.pi / 2)
    c = o.angular_codebook(th)
    assert np.allclose(np.linalg.norm(c, axis=1), 1.0, atol=1e-14)
    assert np.all(c > 0)
    theta_u = np.array([np.arccos(1 / np.sqrt(8 - i)) for i in range(7)])
    assert np.allclose(o.angular_codebook(theta_u), np.full(8, 1 / np.sqrt(8)), atol=1e-15)
    assert np.allclose(o.angular_codebook(np.zeros(7)), np.eye(8)[0])


def pin_angular_backward(o):
    """Eq. 9-10 gradient against central finite differences of sum(g * c(phi)) in fp64, and the
    inverse map: phi -> c -> phi and c -> phi -> c round trips; an axis direction (zero tail)
    gives finite logits whose codebook entry is within 2e-4 of the axis."""
    g = np.random.default_rng(41)
    phi = g.standard_normal((6, 7)) * 2
    gc = g.standard_normal((6, 8))
    d = o.angular_codebook_backward(phi, gc)
    h = 1e-6
    for a in range(6):
        for j in range(7):
            p, m = phi[a].copy(), phi[a].copy()
            p[j] += h
            m[j] -= h
            fd = (gc[a] @ o.angular_codebook(o.angles_from_logits(p))
                  - gc[a] @ o.angular_codebook(o.angles_from_logits(m))) / (2 * h)
            assert abs(fd - d[a, j]) <= 1e-8 * (1 + abs(fd)), (a, j, fd, d[a, j])
    c = o.angular_codebook(o.angles_from_logits(phi))
    assert np.allclose(o.logits_from_codebook(c), phi, atol=1e-12)
    cr = np.abs(g.standard_normal((50, 8))) + 0.05
    cr /= np.linalg.norm(cr, axis=1, keepdims=True)
    assert np.allclose(o.angular_codebook(o.angles_from_logits(o.logits_from_codebook(cr))), cr, atol=1e-12)
    ax = o.logits_from_codebook(np.eye(8)[0])
    assert np.all(np.isfinite(ax)) and np.all(np.abs(ax) < 14)
    assert np.allclose(o.angular_codebook(o.angles_from_logits(ax)), np.eye(8)[0], atol=2e-4)


def pin_fake_quant_radius(o):
    """Softplus closed forms; radii on an fp16-exact grid (offset 0.5, step 1/8, V = 4) are
    reproduced exactly with their levels; a constant group has step 0 and r^ = fp16(r); in
    general r^ sits within half a stored step (plus the fp16 rounding of offset and step) of r."""
    assert abs(o.softplus(0.0) - np.log(2.0)) < 1e-16 and abs(o.softplus(50.0) - 50.0) < 1e-15
    assert abs(o.softplus(-40.0) - np.exp(-40.0)) < 1e-30
    lv = np.tile(np.arange(16), 2)
    r = 0.5 + lv / 8.0
    rho = np.log(np.expm1(r))[None, :]
    _r, rh, q = o.fake_quant_radius(rho, 4)
    assert np.array_equal(q[0], lv) and np.array_equal(rh[0], r)
    _r, rh, q = o.fake_quant_radius(np.full((1, 16), 0.3), 3)
    assert np.all(q == 0) and np.all(rh == O.f16_to_f64(O.f64_to_f16(o.softplus(0.3))))
    g = np.random.default_rng(42)
    rho = g.standard_normal((7, 64)) * 2
    for v in (2, 3, 4):
        r, rh, q = o.fake_quant_radius(rho, v)
        rg = r.reshape(7, 4, 16)
        lo, hi = rg.min(axis=2), rg.max(axis=2)
        lo16 = O.f16_to_f64(O.f64_to_f16(lo))
        st16 = O.f16_to_f64(O.f64_to_f16((hi - lo) / (2**v - 1)))
        bound = 0.5 * st16 + np.abs(lo16 - lo) + (2**v - 1) * np.abs(st16 - (hi - lo) / (2**v - 1)) + 1e-15
        assert np.all(np.abs(rh - r).reshape(7, 4, 16) <= bound[..., None])
        assert q.min() >= 0 and q.max() <= 2**v - 1


def pin_fake_quant_backward(o):
    """Straight-through gradients: dL/dcodebook equals exact finite differences (L is linear in
    the codebook), dL/drho equals central differences of the unrounded surrogate
    sum(g * softplus(rho) s (.) c_z), and W^'s vectors have norm r^ ||c_z|| and the code's signs."""
    g = np.random.default_rng(43)
    n, k, D, V = 3, 256, 4, 3
    rho = g.standard_normal((n, k // 8))
    signs = g.integers(0, 256, (n, k // 8)).astype(np.uint8)
    z = g.integers(0, 1 << D, (n, k // 8))
    phi = g.standard_normal((1 << D, 7))
    c = o.angular_codebook(o.angles_from_logits(phi))
    gw = g.standard_normal((n, k))
    w = o.fake_quant_weights(rho, signs, z, c, V)
    _r, rh, _q = o.fake_quant_radius(rho, V)
    assert np.allclose(np.linalg.norm(w.reshape(n, -1, 8), axis=2), rh * np.linalg.norm(c[z], axis=2), atol=1e-14)
    assert np.array_equal(np.signbit(w.reshape(n, -1, 8)) & (rh[..., None] > 0),
                          (O.sign_factors(signs) < 0) & (rh[..., None] > 0))
    d_rho, d_c = o.fake_quant_backward(rho, signs, z, c, gw, V)
    L0 = np.sum(gw * w)
    for (a, j) in ((0, 0), (3, 5), (int(z[1, 7]), 2)):
        cp = c.copy()
        cp[a, j] += 1.0
        assert abs(np.sum(gw * o.fake_quant_weights(rho, signs, z, cp, V)) - L0 - d_c[a, j]) < 1e-9
    sf = O.sign_factors(signs)

    def surrogate(rr):
        return np.sum(gw.reshape(n, -1, 8) * (o.softplus(rr)[..., None] * sf * c[z]))
    h = 1e-6
    for (a, b) in ((0, 0), (1, 13), (2, 31)):
        p, m = rho.copy(), rho.copy()
        p[a, b] += h
        m[a, b] -= h
        fd = (surrogate(p) - surrogate(m)) / (2 * h)
        assert abs(fd - d_rho[a, b]) <= 1e-7 * (1 + abs(fd))


def pin_init_rho(o):
    """softplus(init_rho) is Eq. 6's radius <|w|, c_z>, floored at 1e-6 for a zero vector."""
    g = np.random.default_rng(44)
    w = g.standard_normal((2, 128)) * 0.05
    w[1, :8] = 0
    cb = synth.random_codebook(4, synth.rng(45))
    c = O.f16_to_f64(cb)
    z = g.integers(0, 16, (2, 16))
    rt = np.sum(np.abs(w.reshape(2, 16, 8)) * c[z], axis=2)
    got = o.softplus(o.init_rho(w, z, c))
    assert np.allclose(got[rt > 0], rt[rt > 0], rtol=1e-12)
    assert abs(got[1, 0] - 1e-6) < 1e-18


def pin_sample_by_squared_radius(o):
    """Sec. 3.1's r^2-proportional sampling: its definition on a tiny input (uniforms chosen away
    from the cumulative boundaries), zero radii never drawn, equal radii give floor(u * N), and
    drawn frequencies follow r^2 / sum r^2."""
    r = np.array([0.0, 1.0, 2.0, 0.0, 3.0])                 # r^2 = 0, 1, 4, 0, 9; total 14
    u = np.array([0.0, 0.5, 0.9, 1.5, 4.9, 5.1, 13.9]) / 14
    assert np.array_equal(o.sample_by_squared_radius(r, u), [1, 1, 1, 2, 2, 4, 4])
    one = np.zeros(50)
    one[17] = 0.3
    g = np.random.default_rng(53)
    assert np.all(o.sample_by_squared_radius(one, g.random(200)) == 17)
    n = 1000
    uu = (np.arange(n) + 0.5) / n
    assert np.array_equal(o.sample_by_squared_radius(np.full(n, 0.7), uu), np.arange(n))
    rr = np.array([1.0, 2.0, 3.0, 4.0])
    idx = o.sample_by_squared_radius(rr, g.random(200000))
    freq = np.bincount(idx, minlength=4) / idx.size
    p = rr**2 / np.sum(rr**2)
    assert np.all(np.abs(freq - p) < 4 * np.sqrt(p * (1 - p) / idx.size))


def pin_spherical_kmeans(o):
    """Spherical k-means (Sec. 3.1): exact centres are a fixed point with the objective equal to
    the sample count; one update moves a centre to the normalised sum of its two directions and
    leaves centres without directions in place; on random data the centres stay on S^7_+, the
    summed cosine never decreases, and no unit vector beats a centre on its own cluster."""
    cb = exact_unit_codebook(16)
    c0 = O.f16_to_f64(cb)
    c, obj = o.spherical_kmeans(np.repeat(c0, 3, axis=0), cb, 3)
    assert np.allclose(c, c0, atol=1e-15) and all(abs(v - 48) < 1e-12 for v in obj)
    a = np.array([1.0, 0.2, 0, 0, 0, 0, 0, 0])
    b = np.array([1.0, 0, 0.3, 0, 0, 0, 0, 0])
    a, b = a / np.linalg.norm(a), b / np.linalg.norm(b)
    c, _ = o.spherical_kmeans(np.stack([a, b]), cb, 1)
    assert np.allclose(c[0], (a + b) / np.linalg.norm(a + b), atol=1e-15)
    assert np.array_equal(c[1:], c0[1:])
    g = np.random.default_rng(51)
    d = np.abs(g.standard_normal((3000, 8)))
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    cbr = synth.random_codebook(5, synth.rng(52))
    c, obj = o.spherical_kmeans(d, cbr, 8)
    assert np.all(c >= 0) and np.allclose(np.linalg.norm(c, axis=1), 1.0, atol=1e-12)
    assert all(y >= x - 1e-9 for x, y in zip(obj, obj[1:]))
    # one update from the fp16 start: each new centre beats random unit vectors on the
    # directions that were assigned to it (the maximiser of the summed cosine)
    c1, _ = o.spherical_kmeans(d, cbr, 1)
    z0 = np.argmax(d @ O.f16_to_f64(cbr).T, axis=1)
    v = np.abs(g.standard_normal((200, 8)))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    for kk in np.unique(z0)[:8]:
        dk = d[z0 == kk]
        best = np.sum(dk @ c1[kk])
        assert np.all(np.sum(dk @ v.T, axis=0) <= best + 1e-9)


def pin_kmeans_codebook(o):
    """The codebook of a matrix whose vectors all point one way (any signs and radii): the centre
    nearest that direction moves onto it (in fp16), every other centre stays, and the objective is
    the sample count."""
    g = np.random.default_rng(54)
    dirn = np.abs(g.standard_normal(8))
    dirn /= np.linalg.norm(dirn)
    scale = g.uniform(0.5, 2.0, (32, 16, 1)) * np.where(g.random((32, 16, 8)) < 0.5, -1.0, 1.0)
    w = (scale * dirn).reshape(32, 128)
    cb = synth.random_codebook(6, synth.rng(55))
    out, obj = o.kmeans_codebook(w, cb, g.random(500), iters=3)
    k0 = int(np.argmax(O.f16_to_f64(cb) @ dirn))
    assert np.array_equal(out[k0], O.f64_to_f16(dirn))
    others = np.arange(64) != k0
    assert np.array_equal(out[others], cb[others])
    assert abs(obj[-1] - 500) < 1e-9


def pin_rel_err(o):
    """The comparison metric: zero on equal inputs, scale invariant, floored by row RMS."""
    y = np.array([[1.0, -2.0, 0.0, 4.0]])
    assert o.rel_err(y, y) == 0
    assert abs(o.rel_err(y * 1.001, y) - 1e-3) < 1e-12
    z = y.copy()
    z[0, 2] = 1e-3
    rms = np.sqrt(np.mean(y * y))
    assert abs(o.rel_err(z, y) - 1e-3 / rms) < 1e-15


PINS = [pin_worked_radius, pin_spherical_roundtrip, pin_bit_budget, pin_decompose,
        pin_assign, pin_ls_radius, pin_radius_quant, pin_decode_norm_and_sign,
        pin_decode_one_hot, pin_gemm_exact_rational, pin_gemm_special_cases,
        pin_encode_roundtrip_bruteforce, pin_encode_group_params_recovered, pin_vector_dims, pin_w2_layout,
        pin_angular_codebook, pin_angular_backward, pin_fake_quant_radius, pin_fake_quant_backward,
        pin_init_rho, pin_sample_by_squared_radius, pin_spherical_kmeans, pin_kmeans_codebook,
        pin_rel_err]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin(_ns())


# ----------------------------------------------------------------- planted mistakes

def _mut_sign_order(signs, dim=8):
    b = np.asarray(signs).astype(np.uint32)[..., None]
    bit = (b >> np.arange(dim - 1, -1, -1, dtype=np.uint32)) & 1      # reversed bit order
    return 1.0 - 2.0 * bit.astype(np.float64)


def _mut_drop_min(q, gmin, gstep):
    return O.dequantize_radius(q, np.zeros_like(gmin), gstep)   # dropped offset term


def _mut_level_off_by_one(q, gmin, gstep):
    return O.dequantize_radius(np.asarray(q) + 1, gmin, gstep)


def _mut_decode_transposed(codes, cb):
    c = O.f16_to_f64(cb)
    r_hat = O.dequantize_radius(codes["q"], codes["gmin"], codes["gstep"])
    s = O.sign_factors(codes["signs"])
    cz = c[np.asarray(codes["dir"], dtype=np.int64)][..., ::-1]  # coordinates reversed
    n, nv = r_hat.shape
    return (r_hat[..., None] * s * cz).reshape(n, nv * 8)


def _mut_step_denominator(r_tilde, v_bits):
    r_tilde = np.asarray(r_tilde, dtype=np.float64)
    lo, hi = r_tilde.min(axis=-1), r_tilde.max(axis=-1)
    return O.f64_to_f16(lo), O.f64_to_f16((hi - lo) / (1 << v_bits))   # 2**V, not 2**V - 1


def _mut_ls_norm(wp, cz):
    return np.linalg.norm(np.asarray(wp, np.float64), axis=-1)     # radius instead of Eq. 6


def _mut_aux_order(signs, dir_idx, q):
    base, aux = O.paper_pack_w2(signs, dir_idx, np.asarray(q))
    base = (np.asarray(base, np.uint32) & 0x3FFF) | (((np.asarray(q, np.uint32) >> 2) & 3) << 14)
    lo = np.asarray(q, np.uint32) & 3
    n, nv = lo.shape
    aux = np.bitwise_or.reduce(lo.reshape(n, nv // 16, 16) << (2 * np.arange(16)), axis=-1)
    return base.astype(np.uint16), aux.astype(np.uint32)             # low/high bits swapped


def _mut_assign_last_tie(d, cb, chunk=4096):
    d = np.asarray(d, dtype=np.float64).reshape(-1, 8)
    c = np.asarray(cb, dtype=np.float64)
    sc = d @ c.T
    return (c.shape[0] - 1 - np.argmax(sc[:, ::-1], axis=1)).astype(np.int64)


def _mut_gemm_x_transposed(codes, cb, x_bits, row_chunk=256):
    x = O.f16_to_f64(x_bits)
    if x.ndim == 1:
        x = x[None, :]
    w = O.decode(codes, cb)
    xr = x.reshape(x.shape[0], -1, 8)[:, :, ::-1].reshape(x.shape)  # x read reversed per vector
    return xr @ w.T


def _mut_sample_by_radius(r, u):
    return O.sample_by_squared_radius(np.sqrt(np.abs(np.asarray(r, np.float64))), u)   # r, not r^2


def _mut_kmeans_mean(d, init_bits, iters):
    c = O.f16_to_f64(init_bits)
    d = np.asarray(d, dtype=np.float64).reshape(-1, 8)
    obj = []
    for _ in range(iters):
        z = O.assign_directions(d, c)
        obj.append(float(np.sum(np.sum(d * c[z], axis=1))))
        cnt = np.bincount(z, minlength=c.shape[0])
        s = np.zeros_like(c)
        np.add.at(s, z, d)
        c = np.where(cnt[:, None] > 0, s / np.maximum(cnt, 1)[:, None], c)   # mean, not normalised
    z = O.assign_directions(d, c)
    obj.append(float(np.sum(np.sum(d * c[z], axis=1))))
    return c, obj


def _mut_kmeans_empty_zero(d, init_bits, iters):
    c = O.f16_to_f64(init_bits)
    d = np.asarray(d, dtype=np.float64).reshape(-1, 8)
    obj = []
    for _ in range(iters):
        z = O.assign_directions(d, c)
        obj.append(float(np.sum(np.sum(d * c[z], axis=1))))
        s = np.zeros_like(c)
        np.add.at(s, z, d)
        norm = np.linalg.norm(s, axis=1)
        c = s / np.where(norm > 0, norm, 1.0)[:, None]                       # empty -> zero centre
    z = O.assign_directions(d, c)
    obj.append(float(np.sum(np.sum(d * c[z], axis=1))))
    return c, obj


def _mut_angular_backward_no_sigmoid(phi, grad_c, eps=1e-4):
    sg = 1.0 / (1.0 + np.exp(-np.asarray(phi, dtype=np.float64)))
    return O.angular_codebook_backward(phi, grad_c, eps) / (sg * (1 - sg))


def _mut_angular_backward_same_index(phi, grad_c, eps=1e-4):
    # the j = i term taken with the sign of the later terms
    phi = np.asarray(phi, dtype=np.float64)
    th = O.angles_from_logits(phi, eps)
    g = np.asarray(grad_c, dtype=np.float64)
    base = O.angular_codebook_backward(phi, grad_c, eps)
    c = O.angular_codebook(th)
    sg = 1.0 / (1.0 + np.exp(-phi))
    extra = 2 * g[..., :7] * c[..., :7] * np.tan(th) * (np.pi / 2 - 2 * eps) * sg * (1 - sg)
    return base + extra


def _mut_logits_swapped(c, eps=1e-4):
    c = np.asarray(c, dtype=np.float64)
    tail = np.sqrt(np.cumsum((c * c)[..., ::-1], axis=-1)[..., ::-1])
    theta = np.arctan2(c[..., :7], tail[..., 1:])
    t = np.clip((theta - eps) / (np.pi / 2 - 2 * eps), 1e-6, 1 - 1e-6)
    return np.log(t) - np.log1p(-t)


def _mut_fq_backward_no_sigmoid(rho, signs, dir_idx, codebook, grad_w, radius_bits):
    d_rho, d_c = O.fake_quant_backward(rho, signs, dir_idx, codebook, grad_w, radius_bits)
    return d_rho * (1.0 + np.exp(-np.asarray(rho, dtype=np.float64))), d_c


def _mut_fq_backward_no_radius(rho, signs, dir_idx, codebook, grad_w, radius_bits):
    d_rho, _ = O.fake_quant_backward(rho, signs, dir_idx, codebook, grad_w, radius_bits)
    n, nv = np.asarray(rho).shape
    g = np.asarray(grad_w, dtype=np.float64).reshape(n, nv, 8)
    d_c = np.zeros_like(np.asarray(codebook, dtype=np.float64))
    np.add.at(d_c, np.asarray(dir_idx).reshape(-1), (O.sign_factors(signs) * g).reshape(-1, 8))
    return d_rho, d_c


def _mut_fq_radius_no_f16(rho, radius_bits):
    r = O.softplus(rho)
    n, nv = r.shape
    rg = r.reshape(n, nv // 16, 16)
    lo = rg.min(axis=-1, keepdims=True)
    st = (rg.max(axis=-1, keepdims=True) - lo) / (2**radius_bits - 1)
    q = np.clip(np.rint((rg - lo) / np.where(st > 0, st, 1)), 0, 2**radius_bits - 1)
    return r, (lo + q * st).reshape(n, nv), q.reshape(n, nv).astype(np.uint8)


MUTANTS = {
    "sign_bit_order": dict(sign_factors=_mut_sign_order),
    "dropped_group_offset": dict(dequantize_radius=_mut_drop_min),
    "level_off_by_one": dict(dequantize_radius=_mut_level_off_by_one),
    "codebook_coords_reversed": dict(decode=_mut_decode_transposed),
    "step_denominator": dict(group_offset_step=_mut_step_denominator),
    "ls_radius_is_norm": dict(ls_radius=_mut_ls_norm),
    "aux_bits_swapped": dict(paper_pack_w2=_mut_aux_order),
    "assign_ties_last": dict(assign_directions=_mut_assign_last_tie),
    "gemm_activation_order": dict(gemm=_mut_gemm_x_transposed),
    "sample_by_radius": dict(sample_by_squared_radius=_mut_sample_by_radius),
    "kmeans_mean_not_normalised": dict(spherical_kmeans=_mut_kmeans_mean),
    "kmeans_empty_centre_zero": dict(spherical_kmeans=_mut_kmeans_empty_zero),
    "angular_backward_no_sigmoid": dict(angular_codebook_backward=_mut_angular_backward_no_sigmoid),
    "angular_backward_same_index_sign": dict(angular_codebook_backward=_mut_angular_backward_same_index),
    "logits_swapped_atan2": dict(logits_from_codebook=_mut_logits_swapped),
    "fake_quant_backward_no_sigmoid": dict(fake_quant_backward=_mut_fq_backward_no_sigmoid),
    "fake_quant_backward_no_radius": dict(fake_quant_backward=_mut_fq_backward_no_radius),
    "fake_quant_radius_unrounded_params": dict(fake_quant_radius=_mut_fq_radius_no_f16),
}


def _rebind(ns):
    """Make the mutated helpers visible to the functions that call them (decode, encode,
    gemm use module globals): run pins against thin wrappers built on the namespace."""
    def decode(codes, cb):
        c = O.f16_to_f64(cb)
        dim = c.shape[-1]
        r_hat = ns.dequantize_radius(codes["q"], codes["gmin"], codes["gstep"])
        s = ns.sign_factors(codes["signs"], dim)
        vec = r_hat[..., None] * s * c[np.asarray(codes["dir"], dtype=np.int64)]
        n, nv = r_hat.shape
        return vec.reshape(n, nv * dim)

    def encode(w, cb, v_bits, params=None):
        w = np.asarray(w, dtype=np.float64)
        n, k = w.shape
        c = O.f16_to_f64(cb)
        dim = c.shape[-1]
        vecs = w.reshape(n, k // dim, dim)
        neg, wp, _r, d = ns.decompose(vecs)
        z = ns.assign_directions(d, c).reshape(n, k // dim)
        rt = ns.ls_radius(wp, c[z]).reshape(n, k // 128, 128 // dim)
        if params is None:
            gmin, gstep = ns.group_offset_step(rt, v_bits)
        else:
            gmin = np.broadcast_to(np.asarray(params[0], np.uint16), (n, k // 128)).copy()
            gstep = np.broadcast_to(np.asarray(params[1], np.uint16), (n, k // 128)).copy()
        q = ns.quantize_radius(rt, gmin, gstep, v_bits).reshape(n, k // dim)
        return {"signs": O.signs_to_bits(neg), "dir": z.astype(np.uint16), "q": q,
                "gmin": gmin, "gstep": gstep}

    def gemm(codes, cb, x_bits, row_chunk=256):
        x = O.f16_to_f64(x_bits)
        if x.ndim == 1:
            x = x[None, :]
        return x @ ns.decode(codes, cb).T

    def kmeans_codebook(w, init_bits, u, iters=20):
        w = np.asarray(w, dtype=np.float64)
        n, k = w.shape
        _neg, _wp, r, d = ns.decompose(w.reshape(n, k // 8, 8))
        idx = ns.sample_by_squared_radius(r, u)
        c, obj = ns.spherical_kmeans(d.reshape(-1, 8)[idx], init_bits, iters)
        return O.f64_to_f16(c), obj

    if ns.kmeans_codebook is O.kmeans_codebook:
        ns.kmeans_codebook = kmeans_codebook
    if ns.decode is O.decode:
        ns.decode = decode
    if ns.encode is O.encode:
        ns.encode = encode
    if ns.gemm is O.gemm:
        ns.gemm = gemm
    return ns


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutants_are_caught(name):
    ns = _rebind(_ns(**MUTANTS[name]))
    failed = []
    for pin in PINS:
        try:
            pin(ns)
        except (AssertionError, ValueError, IndexError):
            failed.append(pin.__name__)
    assert failed, f"no pin caught mutant {name}"


def test_unmutated_rebind_passes():
    """The wrapper used for mutants is itself faithful: with no mutation every pin passes."""
    ns = _rebind(_ns())
    for pin in PINS:
        pin(ns)


def test_synthetic_codebook_on_positive_sphere():
    """Generated codebooks lie on S^7_+ up to fp16 rounding (each coordinate within 2^-11
    relative), as the representation requires (Sec. 3.1)."""
    for d_bits in (4, 6, 8, 13):
        c = O.f16_to_f64(synth.random_codebook(d_bits, synth.rng(d_bits)))
        assert np.all(c >= 0)
        assert np.all(np.abs(np.linalg.norm(c, axis=1) - 1.0) <= 2.0**-10)
