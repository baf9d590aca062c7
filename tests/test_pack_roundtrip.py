"""The library's host packer (csrc/sph_pack.cpp) under AddressSanitizer and UndefinedBehavior-
Sanitizer, on the CPU: tests/native/pack_roundtrip.cpp packs seeded logical codes into a blob of
exactly the size the layout reports, checks that nothing lands outside the streams, that padded
rows of the last 16-row tile are zero and that the tables follow from the codebook, and decodes
every field back with its own reader of the layout; the decoded codes must equal the input bit
for bit. Every format, at ragged row counts (1, 17, 87 rows: a partial tile, one full and one
partial, several) and one or two 128-weight groups."""
from __future__ import annotations

import os
import shutil
import subprocess

import numpy as np
import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = [os.path.join(ROOT, "tests", "native", "pack_roundtrip.cpp"),
       os.path.join(ROOT, "paper_2609_24875_amd", "csrc", "sph_pack.cpp")]

# (vec_dim, dir_bits, radius_bits): every layout kind, and every built-in pair of the W2 budget
FORMATS = [(8, 6, 4), (8, 6, 3), (8, 7, 2), (8, 4, 4), (8, 5, 3), (8, 6, 2), (8, 8, 8), (8, 8, 2),
           (8, 13, 3), (8, 13, 4), (4, 2, 3), (16, 14, 6)]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    out = str(tmp_path_factory.mktemp("native") / "pack_roundtrip")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), *SRC, "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0 and "sanitize" in res.stderr and "cannot find" in res.stderr:
        pytest.skip("sanitizer runtime not available")
    assert res.returncode == 0, res.stderr
    return out


def _codes(vec, d, v, n, k, seed):
    g = synth.rng(seed, n, k, d, v)
    codes = synth.uniform_codes(n, k, d, v, g, dim=vec)
    codes["gmin"], codes["gstep"] = synth.varied_group_params(n, k, v, g)
    cb = synth.random_codebook(d, g, dim=vec)
    return codes, cb


@pytest.mark.parametrize("vec,d,v", FORMATS)
@pytest.mark.parametrize("n", [1, 17, 87])
@pytest.mark.parametrize("k", [128, 256])
def test_host_pack_roundtrip_sanitized(driver, tmp_path, vec, d, v, n, k):
    codes, cb = _codes(vec, d, v, n, k, 5)
    sign_t = np.uint16 if vec == 16 else np.uint8
    arrays = [np.ascontiguousarray(codes["signs"], dtype=sign_t),
              np.ascontiguousarray(codes["dir"], dtype=np.uint16),
              np.ascontiguousarray(codes["q"], dtype=np.uint8),
              np.ascontiguousarray(codes["gmin"], dtype=np.uint16),
              np.ascontiguousarray(codes["gstep"], dtype=np.uint16)]
    inp, outp = tmp_path / "in.bin", tmp_path / "out.bin"
    with open(inp, "wb") as f:
        f.write(np.array([vec, d, v], dtype=np.int32).tobytes())
        f.write(np.array([n, k], dtype=np.int64).tobytes())
        for a in arrays:
            f.write(a.tobytes())
        f.write(np.ascontiguousarray(cb, dtype=np.uint16).tobytes())
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=90",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1:exitcode=91")
    res = subprocess.run([driver, str(inp), str(outp)], capture_output=True, text=True, env=env, timeout=120)
    assert res.returncode == 0, res.stderr
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, res.stderr
    raw = open(outp, "rb").read()
    pos = 0
    for a in arrays:
        b = np.frombuffer(raw, dtype=a.dtype, count=a.size, offset=pos).reshape(a.shape)
        pos += a.nbytes
        assert np.array_equal(b, a)
    assert pos == len(raw)


def test_roundtrip_driver_catches_a_corrupted_code(driver, tmp_path):
    """The driver's own check is live: an out-of-range direction index is refused by the
    library's validation before packing (exit status 10, message on stderr)."""
    codes, cb = _codes(8, 6, 4, 17, 128, 6)
    codes["dir"][3, 2] = 1 << 6
    inp = tmp_path / "in.bin"
    with open(inp, "wb") as f:
        f.write(np.array([8, 6, 4], dtype=np.int32).tobytes())
        f.write(np.array([17, 128], dtype=np.int64).tobytes())
        for name, t in (("signs", np.uint8), ("dir", np.uint16), ("q", np.uint8), ("gmin", np.uint16),
                        ("gstep", np.uint16)):
            f.write(np.ascontiguousarray(codes[name], dtype=t).tobytes())
        f.write(np.ascontiguousarray(cb, dtype=np.uint16).tobytes())
    res = subprocess.run([driver, str(inp), str(tmp_path / "out.bin")], capture_output=True, text=True, timeout=60)
    assert res.returncode == 10 and "codes rejected" in res.stderr
