"""CPU checks of the C-ABI library: it loads, exports every function include/sph.h declares, and
its host-side validation returns the documented status codes before any HIP call is made.
No call here launches a kernel or copies memory."""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import pytest

import synth
import paper_2609_24875_amd as pkg
from paper_2609_24875_amd import sph as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sph.h")

needs_lib = pytest.mark.skipif(not os.path.exists(pkg.LIB_PATH), reason="libsph.so not built")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sph_[a-z_]+)\s*\(", text)))


def test_header_declares_binding_exports():
    assert declared_functions() == sorted(pkg.EXPORTS)


@needs_lib
def test_library_exports_every_declared_symbol():
    lib = pkg.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_read_probe_is_separate_from_the_library():
    """The benchmark's streaming-read probe is its own library: libsph exports no probe symbol,
    and the probe exports its one entry point."""
    from paper_2609_24875_amd import build as Bd
    if os.path.exists(pkg.LIB_PATH):
        assert not hasattr(ctypes.CDLL(pkg.LIB_PATH), "sph_probe_stream_read")
    if not os.path.exists(Bd.PROBE_OUT):
        pytest.skip("libsph_probe.so not built")
    assert hasattr(ctypes.CDLL(Bd.PROBE_OUT), "sph_probe_stream_read")


@needs_lib
def test_status_strings():
    for code in range(9):
        assert pkg.status_str(code) and pkg.status_str(code) != "unknown status"
    assert pkg.status_str(99) == "unknown status"


@needs_lib
@pytest.mark.parametrize("d,v,ok", [(6, 4, True), (13, 3, True), (4, 4, True), (8, 8, True),
                                    (6, 2, True), (5, 3, True), (6, 3, True), (7, 2, True),
                                    (8, 2, True), (13, 4, True), (7, 3, False), (8, 4, False),
                                    (13, 5, False), (2, 4, False), (16, 4, False)])
def test_format_supported(d, v, ok):
    assert pkg.format_supported(d, v) == ok


@needs_lib
def test_packed_bytes_accounts_for_every_stream():
    # W2 4096 x 12288: records 36 B per 16 rows x 8 columns; params 4 B per 16 rows x 128 cols.
    n, k = 4096, 12288
    got = pkg.packed_bytes(6, 4, n, k)
    codes = (n // 16) * (k // 8) * 36           # 36 B per (16 rows x 8 columns) record
    params = n * (k // 128) * 4                  # fp16 (offset, step) per row and group
    tables = 2 * 64 * 16 * 8 + 64 * 16          # nibble tables + raw codebook
    assert codes + params + tables <= got <= codes + params + tables + 5 * 256
    # padding to 16-row tiles
    assert pkg.packed_bytes(6, 4, 17, 128) == pkg.packed_bytes(6, 4, 32, 128)


@needs_lib
def test_packed_bytes_w3_four_radius_bits():
    # 8 sign + 13 direction + 4 radius bits: sign bytes and (z | low 3 bits of q) words as for 3
    # radius bits, plus one 16-bit word of high radius bits per record.
    n, k = 4096, 12288
    got = pkg.packed_bytes(13, 4, n, k)
    codes = (n // 16) * (k // 8) * (16 + 32 + 2)
    params = n * (k // 128) * 4
    tables = (16 << 13) * 2                     # codebook table + raw codebook
    assert codes + params + tables <= got <= codes + params + tables + 6 * 256


@needs_lib
@pytest.mark.parametrize("n,k", [(0, 128), (-1, 128), (16, 0), (16, 100), (16, 130), (1 << 25, 128)])
def test_packed_bytes_shape_errors(n, k):
    with pytest.raises(pkg.SphError) as e:
        pkg.packed_bytes(6, 4, n, k)
    assert e.value.status == 2


def _codes(n=20, k=256, D=6, V=4, seed=0):
    g = synth.rng(seed)
    c = synth.uniform_codes(n, k, D, V, g)
    c["gmin"], c["gstep"] = synth.row_scale_group_params(n, k, V, g)
    return c, synth.random_codebook(D, g)


def _pack_status(codes, cb, D=6, V=4, buf=0x10000, nbytes=1 << 30, fmt=None):
    lib = pkg.load_library()
    fmt = fmt or B.make_format(D, V)
    n, nv = codes["signs"].shape
    arrs = [np.ascontiguousarray(codes[key]) for key in ("signs", "dir", "q", "gmin", "gstep")]
    cb = np.ascontiguousarray(cb)
    w = B.CWeights()
    return lib.sph_pack_weights(ctypes.byref(fmt), n, nv * 8, *[a.ctypes.data for a in arrs],
                                cb.ctypes.data, buf, nbytes, None, ctypes.byref(w))


@needs_lib
def test_pack_validation_errors():
    codes, cb = _codes()
    assert _pack_status(codes, cb, fmt=B.make_format(6, 4, vec_dim=4)) == 3
    assert _pack_status(codes, cb, fmt=B.make_format(6, 4, group_size=64)) == 3
    assert _pack_status(codes, cb, fmt=B.make_format(7, 4)) == 3
    bad = dict(codes, dir=codes["dir"].copy())
    bad["dir"][3, 5] = 64
    assert _pack_status(bad, cb) == 4
    bad = dict(codes, q=codes["q"].copy())
    bad["q"][0, 0] = 16
    assert _pack_status(bad, cb) == 4
    for key, val in (("gstep", 0xBC00), ("gstep", 0x7C00), ("gmin", 0x7E00)):
        bad = dict(codes, **{key: codes[key].copy()})
        bad[key][1, 1] = val                   # -1.0, +inf, NaN
        assert _pack_status(bad, cb) == 5, (key, hex(val))
    bcb = cb.copy()
    bcb[2, 3] = 0x8000 | bcb[2, 3]             # negative entry
    assert _pack_status(codes, bcb) == 5
    bcb = cb.copy()
    bcb[1, 0] = 0x4001                         # just above 2: not a unit direction's coordinate
    assert _pack_status(codes, bcb) == 5
    bcb[1, 0] = 0x4000                         # exactly 2 passes validation (then the size check)
    assert _pack_status(codes, bcb, nbytes=100) == 6
    assert _pack_status(codes, cb, nbytes=100) == 6
    assert _pack_status(codes, cb, buf=0x10001) == 2
    assert _pack_status(codes, cb, buf=0) == 1


@needs_lib
def test_compute_calls_reject_bad_descriptor_before_any_hip_call():
    lib = pkg.load_library()
    w = B.CWeights()                           # never filled by sph_pack_weights
    assert lib.sph_gemv(ctypes.byref(w), 0x10000, 0x20000, 1, None, 0, None) == 8
    assert lib.sph_gemm_small(ctypes.byref(w), 0x10000, 4, 256, 0x20000, 256, 1, None, 0, None) == 8
    assert lib.sph_unpack(ctypes.byref(w), 0x1000, 0x2000, 0x3000, None) == 8
    assert lib.sph_gemv(None, 0x10000, 0x20000, 1, None, 0, None) == 1
    out = ctypes.c_size_t(0)
    assert lib.sph_workspace_bytes(ctypes.byref(w), 1, ctypes.byref(out)) == 8


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(pkg.SphLibraryMissing):
        _load_fresh(str(tmp_path / "missing.so"))


def _load_fresh(path):
    saved = B._lib
    B._lib = None
    try:
        return B.load_library(path)
    finally:
        B._lib = saved


@needs_lib
def test_encode_validation_errors_before_any_hip_call():
    lib = pkg.load_library()
    f = B.make_format(6, 4)
    W, CB, S, D, Q, GM, GS = 0x10000, 0x20000, 0x30000, 0x40000, 0x50000, 0x60000, 0x70000

    def st(fmt=f, n=16, k=128, w=W, ldw=128, cb=CB, s=S, d=D, q=Q, gm=GM, gs=GS):
        return lib.sph_encode(ctypes.byref(fmt) if fmt is not None else None, n, k, w, ldw, cb,
                              s, d, q, gm, gs, None)
    assert st(fmt=None) == 1 and st(w=0) == 1 and st(cb=0) == 1 and st(gs=0) == 1
    assert st(fmt=B.make_format(7, 4)) == 3 and st(fmt=B.make_format(6, 4, vec_dim=4)) == 3
    assert st(k=100) == 2 and st(n=0) == 2
    assert st(ldw=120) == 2 and st(ldw=130) == 2       # ldw < k, ldw not a multiple of 4
    assert st(w=0x10008) == 2 and st(d=0x40001) == 2    # misaligned weights / direction indices


@needs_lib
def test_kmeans_workspace_and_validation():
    lib = pkg.load_library()
    f = B.make_format(6, 4)
    n, k, ns = 1024, 4096, 65536
    nb = pkg.kmeans_workspace_bytes(6, 4, n, k, ns)
    nvec = n * k // 8
    # running r^2 per vector; per sample a direction (64 B), an assignment (4 B), an objective
    # part per 256 samples, and a (cosine, index) pair per codebook split; per centre the fp64
    # centre (64 B) and, per sample chunk, its fixed-point sum (8 components x 3 limbs x 8 B)
    for D, V in ((6, 4), (13, 3)):
        ncb = 1 << D
        chunks = -(-128 // -(-ncb // 512))
        nb = pkg.kmeans_workspace_bytes(D, V, n, k, ns)
        assert nb >= nvec * 8 + ns * (64 + 4 + 12) + ncb * (64 + 192 * chunks)
        assert nb <= (nvec * 8 + ns * 80 + 12 * (ns + 2**20) + ncb * (64 + 192 * chunks) + 10 * 256
                      + (nvec // 2048 + ns // 256 + 2) * 8)
    with pytest.raises(pkg.SphError) as e:
        pkg.kmeans_workspace_bytes(6, 4, n, k, 0)
    assert e.value.status == 2

    def st(ns=1000, iters=5, ws_bytes=1 << 40, ws=0x100000, u=0x10000, ldw=k):
        return lib.sph_kmeans_codebook(ctypes.byref(f), n, k, 0x20000, ldw, u, ns, iters, 0x30000,
                                       0x40000, 0x50000, 0x60000, ws, ws_bytes, None)
    assert st(u=0) == 1 and st(ws=0) == 1
    assert st(ns=0) == 2 and st(ns=(1 << 24) + 1) == 2 and st(iters=-1) == 2 and st(iters=10001) == 2
    assert st(ws=0x100080) == 2 and st(u=0x10004) == 2 and st(ldw=k - 4) == 2
    assert st(ws_bytes=pkg.kmeans_workspace_bytes(6, 4, n, k, 1000) - 1) == 6


@needs_lib
def test_direction_groups_host_counting_sort():
    z = np.random.default_rng(5).integers(0, 64, 10000).astype(np.uint16)
    perm, off = B.direction_groups(6, z)
    assert np.array_equal(perm, np.argsort(z, kind="stable"))
    assert np.array_equal(off, np.concatenate([[0], np.cumsum(np.bincount(z, minlength=64))]))
    with pytest.raises(pkg.SphError) as e:
        B.direction_groups(4, z)                # indices >= 16
    assert e.value.status == 4


@needs_lib
def test_training_entry_points_validate_before_any_hip_call():
    lib = pkg.load_library()
    f = B.make_format(6, 4)
    assert lib.sph_angular_codebook(0, 0x1000, 1e-4, 0x2000, None) == 2
    assert lib.sph_angular_codebook(14, 0x1000, 1e-4, 0x2000, None) == 2
    assert lib.sph_angular_codebook(6, 0x1000, 0.3, 0x2000, None) == 2
    assert lib.sph_angular_codebook(6, None, 1e-4, 0x2000, None) == 1
    assert lib.sph_angular_logits(6, 0x1000, 1e-4, None, None) == 1
    P = 0x10000
    assert lib.sph_fake_quant_forward(ctypes.byref(f), 16, 100, P, P, P, P, P, 128, None, None, None, None, None) == 2
    assert lib.sph_fake_quant_forward(ctypes.byref(f), 16, 128, P, P, P, P, P, 120, None, None, None, None, None) == 2
    assert lib.sph_fake_quant_forward(ctypes.byref(f), 16, 128, P, P, P, P, P, 128, None, P, None, None, None) == 1
    assert lib.sph_fake_quant_forward(ctypes.byref(f), 16, 128, P, P, P, P, P + 8, 128, None, None, None, None,
                                      None) == 2
    assert lib.sph_fake_quant_forward(ctypes.byref(B.make_format(7, 4)), 16, 128, P, P, P, P, P, 128, None, None,
                                      None, None, None) == 3
    nb = ctypes.c_size_t(0)
    assert lib.sph_fake_quant_backward_workspace_bytes(13, ctypes.byref(nb)) == 0 and nb.value == 8192 * 32
    assert lib.sph_fake_quant_backward_workspace_bytes(6, ctypes.byref(nb)) == 0 and nb.value == 64 * 16 * 32
    assert lib.sph_fake_quant_backward(ctypes.byref(f), 16, 128, P, P, P, P, P, P, 128, P, P, P, P, P,
                                       64 * 16 * 32 - 1, None) == 6
    assert lib.sph_fake_quant_backward(ctypes.byref(f), 16, 128, P, P, P, P, P, P, 128, P, P, P, P, None,
                                       1 << 20, None) == 1


@needs_lib
def test_vector_size_variants_supported_and_sized():
    assert pkg.format_supported(2, 3, 4) and pkg.format_supported(14, 6, 16)
    assert not pkg.format_supported(6, 4, 4) and not pkg.format_supported(13, 3, 16)
    assert not pkg.format_supported(2, 3, 8) and not pkg.format_supported(2, 3, 2)
    n, k = 4096, 4096
    # 4-D: one byte per vector, one dword of high radius bits and one of parameters per group
    got = pkg.packed_bytes(2, 3, n, k, 4)
    base = n * k // 4 + n * (k // 128) * 8 + 64 * 8 + 4 * 4 * 2
    assert base <= got <= base + 5 * 256
    # 16-D: one dword per vector, two dwords per group, the 512 KiB codebook
    got = pkg.packed_bytes(14, 6, n, k, 16)
    base = n * k // 16 * 4 + n * (k // 128) * 8 + (1 << 14) * 16 * 2
    assert base <= got <= base + 5 * 256
    # payload 2.25 bits per weight plus 0.25 of fp16 group parameters, besides the codebook
    assert (got - (1 << 14) * 32) * 8 / (n * k) <= 2.5 + 1e-3


@needs_lib
def test_vector_size_pack_validation():
    g = synth.rng(9)
    codes = synth.uniform_codes(16, 128, 2, 3, g, dim=4)
    codes["gmin"], codes["gstep"] = synth.row_scale_group_params(16, 128, 3, g)
    cb = synth.random_codebook(2, g, dim=4)
    lib = pkg.load_library()

    def st(c, fmt=B.make_format(2, 3, 4)):
        arrs = [np.ascontiguousarray(c[key]) for key in ("signs", "dir", "q", "gmin", "gstep")]
        w = B.CWeights()
        return lib.sph_pack_weights(ctypes.byref(fmt), 16, 128, *[a.ctypes.data for a in arrs], cb.ctypes.data,
                                    0x10000, 1 << 30, None, ctypes.byref(w))
    bad = dict(codes, signs=codes["signs"].copy())
    bad["signs"][2, 3] = 16                     # only 4 sign bits
    assert st(bad) == 4
    bad = dict(codes, q=codes["q"].copy())
    bad["q"][0, 0] = 8
    assert st(bad) == 4
    enc = ctypes.c_int
    f4 = B.make_format(2, 3, 4)
    assert lib.sph_encode(ctypes.byref(f4), 16, 128, 0x10000, 128, 0x20000, 0x30000, 0x40000, 0x50000,
                          0x60000, 0x70000, None) == 3     # the encoder is 8-D only


def test_noalloc_scratch_size_matches_header():
    with open(os.path.join(os.path.dirname(__file__), "..", "include", "sph.h")) as f:
        m = re.search(r"#define SPH_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", f.read())
    assert m and int(m.group(1)) << int(m.group(2)) == B.NOALLOC_SCRATCH_BYTES


@needs_lib
def test_noalloc_rejects_bad_arguments_before_any_hip_call():
    lib = pkg.load_library()
    w = B.CWeights()                           # never filled by sph_pack_weights
    assert lib.sph_gemm_small_noalloc(ctypes.byref(w), 0x10000, 4, 256, 0x20000, 256, 1, None) == 8
    assert lib.sph_gemm_small_noalloc(None, 0x10000, 4, 256, 0x20000, 256, 1, None) == 1
    assert lib.sph_gemm_small_noalloc(ctypes.byref(w), None, 4, 256, 0x20000, 256, 1, None) == 1
