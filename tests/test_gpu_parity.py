"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Bars: unpacked codes bit-exact; outputs within rel_err <= 2e-3 (max |y - y*| over
max(|y*|, row RMS of y*)), the tolerance the target states for fp32 accumulation against the
fp64 oracle. Every path forms exact fp16 products (the signed directions, and on the matrix
cores the level times the direction split exactly into two fp16 words) and rounds only its fp32
radius and sums. Each path is also held, output by output, to the a-priori bound its arithmetic
gives.

Group parameters (Eq. 7) are drawn independently for every group of every row, with negative
offsets, zero steps and magnitudes over eight binary orders, so that a wrong group or row index
in any kernel mode changes the result.
"""
from __future__ import annotations

import numpy as np
import pytest

import synth
from oracle import sph as O

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_24875_amd as pkg  # noqa: E402

DEV = torch.device("cuda:0")
TOL = 2e-3
FMTS = ["W2", "W3", "W2_cfg", "W3_cfg", "W2_16", "W3_25", "W2_63", "W2_72", "W2_82"]
PARAMS = {"varied": synth.varied_group_params, "row": synth.row_scale_group_params,
          "extreme": synth.extreme_group_params}


def to_dev_f16(bits: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.float16)


def uniform_case(fmt, n, k, seed, params="varied"):
    """Uniform random codes with group parameters of the given kind (see ``PARAMS``)."""
    D, V = synth.FORMATS[fmt]
    g = synth.rng(seed, n, k, synth.STREAM_CODES)
    codes = synth.uniform_codes(n, k, D, V, g)
    codes["gmin"], codes["gstep"] = PARAMS[params](n, k, V, g)
    cb = synth.random_codebook(D, synth.rng(seed, n, k, synth.STREAM_CODEBOOK))
    return D, V, codes, cb


def encoded_case(fmt, n, k, seed):
    D, V = synth.FORMATS[fmt]
    cb = synth.random_codebook(D, synth.rng(seed, n, k, synth.STREAM_CODEBOOK))
    w = synth.outlier_gaussian_weights(n, k, synth.rng(seed, n, k, synth.STREAM_WEIGHTS))
    return D, V, O.encode(w, cb, V), cb


def radius_bound(codes, cb, x, rows=512):
    """sum_k (|min| + q step) |c| |x_k| per output (decoded a block of rows at a time): the scale
    of fp32 summation error, sum |w^ x|, with each radius replaced by the sum of the magnitudes of
    its two terms (Eq. 7); the two agree when offsets are non-negative. The matrix-core paths for
    batches above 8 form offset * sum <t, x> and step * sum q <t, x> separately, so their fp32
    rounding scales with these terms even where a negative offset cancels part of the radius."""
    xa = np.abs(O.f16_to_f64(x))
    dim = np.asarray(cb).shape[-1]
    n = np.asarray(codes["q"]).shape[0]
    out = np.empty((xa.shape[0], n))
    for a in range(0, n, rows):
        blk = {name: np.asarray(v)[a:a + rows] for name, v in codes.items()}
        mag = dict(blk, gmin=O.f64_to_f16(np.abs(O.f16_to_f64(blk["gmin"]))))
        mag["signs"] = np.zeros_like(blk["signs"])
        out[:, a:a + rows] = xa @ np.abs(O.decode(mag, cb)).T
    return out


def sum_bound(codes, cb, x, k):
    """Error bound of every path: exact fp16 products, fp32 radius and fp32 sums (k 2^-23 is a
    loose cover for the rounding of sums of at most k + 3 terms)."""
    return k * 2.0**-23 * radius_bound(codes, cb, x)


@pytest.mark.parametrize("fmt", FMTS)
def test_unpack_bit_exact(fmt):
    D, V, codes, cb = uniform_case(fmt, 87, 640, 1)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    back = pkg.unpack(w)
    for key in ("signs", "dir", "q"):
        assert np.array_equal(back[key], codes[key]), key


@pytest.mark.parametrize("fmt", FMTS)
# 4224 = 33 groups of 128 leaves a ragged last step (32 vector positions per batch-1 step);
# 8320 weights per row span several wave ranges
@pytest.mark.parametrize("n,k", [(87, 640), (16, 128), (1, 256), (300, 2048), (300, 4224), (40, 8320)])
def test_gemv_parity(fmt, n, k):
    D, V, codes, cb = uniform_case(fmt, n, k, 2)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(1, k, synth.rng(2, n, k, synth.STREAM_X))
    y = pkg.gemv(w, to_dev_f16(x)[0]).cpu().numpy()
    ref = O.gemv(codes, cb, x)
    assert O.rel_err(y, ref) <= TOL
    # exact products + fp32 sums: |error| <= K * 2^-23 * sum|w x| (a loose a-priori bound)
    assert np.all(np.abs(y - ref) <= sum_bound(codes, cb, x, k)[0] + 1e-30)
    y16 = pkg.gemv(w, to_dev_f16(x)[0], out_dtype=torch.float16).cpu().numpy().astype(np.float64)
    assert np.array_equal(y16, y.astype(np.float16).astype(np.float64))


@pytest.mark.parametrize("fmt", ["W2", "W3", "W2_cfg", "W3_cfg"])
def test_gemv_parity_encoded(fmt):
    D, V, codes, cb = encoded_case(fmt, 70, 1024, 3)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(1, 1024, synth.rng(3, 0, 0, synth.STREAM_X))
    y = pkg.gemv(w, to_dev_f16(x)[0]).cpu().numpy()
    assert O.rel_err(y, O.gemv(codes, cb, x)) <= TOL


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("m", [2, 3, 4, 5, 8, 9, 16, 17, 24, 32])
def test_gemm_small_parity(fmt, m):
    n, k = 75, 1152
    D, V, codes, cb = uniform_case(fmt, n, k, 4)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(4, m, k, synth.STREAM_X))
    y = pkg.gemm_small(w, to_dev_f16(x)).cpu().numpy()
    ref = O.gemm(codes, cb, x)
    err = O.rel_err(y, ref)
    assert err <= TOL, err
    assert np.all(np.abs(y - ref) <= sum_bound(codes, cb, x, k) + 1e-30)


def test_gemm_small_strided_and_fp16_out():
    D, V, codes, cb = uniform_case("W2", 48, 512, 5)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    for m in (2, 3, 20):
        x = synth.activations(m, 512, synth.rng(5, m, 0, synth.STREAM_X))
        big = torch.zeros((m, 512 + 64), dtype=torch.float16, device=DEV)
        big[:, :512] = to_dev_f16(x)
        out = torch.full((m, 64), 7.0, dtype=torch.float16, device=DEV)
        pkg.gemm_small(w, big[:, :512], out=out[:, :48])
        ref = O.gemm(codes, cb, x)
        assert O.rel_err(out[:, :48].float().cpu().numpy(), ref) <= TOL
        assert torch.all(out[:, 48:] == 7.0)            # nothing written past n


def test_unit_activation_returns_decoded_column():
    """x = e_c picks column c of W^: every weight the kernel rebuilds is checked (Eq. 4). Batches
    1..8 return its fp32 rounding exactly (the per-row radius scale of the benchmark description
    makes every radius exact in fp32, and each product is rounded once); the factored paths above
    batch 8 round the offset and step terms separately, within 2^-23 of their magnitudes."""
    D, V, codes, cb = uniform_case("W2", 33, 256, 6, params="row")
    w = pkg.pack(D, V, codes, cb, device=DEV)
    dense = O.decode(codes, cb)
    eye = np.eye(256)
    for c0 in range(0, 256, 64):
        x = synth.f16_bits(eye[c0:c0 + 64])                        # 64 unit vectors at once
        xd = to_dev_f16(x)
        for i in range(0, 64, 9):
            y1 = pkg.gemv(w, xd[i]).cpu().numpy()
            assert np.array_equal(y1, dense[:, c0 + i].astype(np.float32))
        ref = dense[:, c0:c0 + 64].T
        for m in (2, 3, 8):
            y = pkg.gemm_small(w, xd[:m]).cpu().numpy()
            assert np.array_equal(y, ref[:m].astype(np.float32)), m
        for m, call in ((16, pkg.gemm_small), (32, pkg.gemm_small), (64, pkg.gemm)):
            y = call(w, xd[:m]).cpu().numpy()
            assert np.all(np.abs(y - ref[:m]) <= 2.0**-22 * radius_bound(codes, cb, x[:m])), m


def test_deterministic():
    D, V, codes, cb = uniform_case("W2", 500, 4096, 7)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = to_dev_f16(synth.activations(1, 4096, synth.rng(7)))[0]
    a = pkg.gemv(w, x).clone()
    b = pkg.gemv(w, x).clone()
    assert torch.equal(a, b)


def test_concurrent_streams():
    """Two decode calls whose split tiles meet in the global workspace, launched back to back on
    two streams so that their workgroups share the GPU, each with its own workspace: both match
    the oracle and the results of the same calls made one after the other."""
    cases = []
    for i, (fmt, n, k) in enumerate((("W2", 5120, 25600), ("W3", 4096, 12288))):
        D, V, codes, cb = uniform_case(fmt, n, k, 50 + i)
        w = pkg.pack(D, V, codes, cb, device=DEV)
        x = synth.activations(1, k, synth.rng(50 + i, synth.STREAM_X))
        cases.append((w, codes, cb, x, to_dev_f16(x)[0]))
    serial = [pkg.gemv(w, xd).cpu().numpy() for w, _, _, _, xd in cases]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [torch.empty(c[0].n, dtype=torch.float32, device=DEV) for c in cases]
    torch.cuda.synchronize()
    for _ in range(20):
        for (w, _, _, _, xd), s, o in zip(cases, streams, outs):
            with torch.cuda.stream(s):
                pkg.gemv(w, xd, out=o, stream=s)
    torch.cuda.synchronize()
    for (w, codes, cb, x, _), o, ref_bits in zip(cases, outs, serial):
        y = o.cpu().numpy()
        assert np.array_equal(y, ref_bits)
        assert O.rel_err(y, O.gemv(codes, cb, x)) <= TOL


def test_bad_arguments_raise():
    D, V, codes, cb = uniform_case("W2", 16, 128, 8)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = torch.zeros((2, 128), dtype=torch.float16, device=DEV)
    with pytest.raises(TypeError):
        pkg.gemm_small(w, x.float())                                  # fp32 activations
    with pytest.raises(ValueError):
        pkg.gemm_small(w, torch.zeros((2, 64), dtype=torch.float16, device=DEV))  # short rows
    with pytest.raises(ValueError):
        pkg.gemv(w, torch.zeros(256, dtype=torch.float16, device=DEV)[::2])        # strided x
    with pytest.raises(TypeError):
        pkg.gemm_small(w, x, out=torch.empty((2, 16), dtype=torch.bfloat16, device=DEV))
    with pytest.raises(ValueError):
        pkg.gemm_small(w, x, out=torch.empty((2, 8), dtype=torch.float32, device=DEV))
    with pytest.raises(ValueError):
        pkg.gemm_small(w, x, out=torch.empty((16, 2), dtype=torch.float32, device=DEV).t())


def test_bad_batch_raises():
    D, V, codes, cb = uniform_case("W2", 16, 128, 8)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = torch.zeros((33, 128), dtype=torch.float16, device=DEV)
    with pytest.raises(pkg.SphError):
        pkg.gemm_small(w, x)


# ----------------------------------------------------------------- special cases (Eq. 4, 7)

def run_any(w, x):
    """The library call for a batch of activation rows: sph_gemv, sph_gemm_small or sph_gemm."""
    xd = to_dev_f16(x)
    m = x.shape[0]
    if m == 1:
        return pkg.gemv(w, xd[0]).cpu().numpy()[None, :]
    return (pkg.gemm_small(w, xd) if m <= 32 else pkg.gemm(w, xd)).cpu().numpy()


def check_bounds(y, ref, codes, cb, x, k):
    bound = sum_bound(codes, cb, x, k)
    assert np.all(np.abs(y - ref) <= bound + 1e-30), float(np.max(np.abs(y - ref) - bound))


ALL_FMTS = FMTS + ["V4", "V16"]


@pytest.mark.parametrize("fmt", ALL_FMTS)
@pytest.mark.parametrize("m", [1, 2, 4, 16, 64])
def test_one_hot_codebook_is_sparse_dot(fmt, m):
    """A codebook of unit axes, c_z = e_(z mod dim): Eq. 4 keeps one coordinate per vector, so
    y[b, n] = sum_v r^_(n,v) s_(n,v,j) x[b, dim v + j] with j = z mod dim, a sparse dot product
    written out here with numpy indexing (independent of the oracle's decoder)."""
    n, k = 90, 1152
    D, V = synth.FORMATS[fmt]
    dim = synth.fmt_dim(fmt)
    g = synth.rng(31, n, k, m, synth.STREAM_CODES)
    codes = synth.uniform_codes(n, k, D, V, g, dim=dim)
    codes["gmin"], codes["gstep"] = synth.varied_group_params(n, k, V, g)
    cb = synth.f16_bits(np.eye(dim)[np.arange(1 << D) % dim])
    w = pkg.pack(D, V, codes, cb, device=DEV, vec_dim=dim)
    x = synth.activations(m, k, synth.rng(31, m, synth.STREAM_X))
    xf = O.f16_to_f64(x)
    nv = k // dim
    lo = np.repeat(O.f16_to_f64(codes["gmin"]), 128 // dim, axis=1)
    st = np.repeat(O.f16_to_f64(codes["gstep"]), 128 // dim, axis=1)
    radius = lo + codes["q"].astype(np.float64) * st
    j = codes["dir"].astype(np.int64) % dim
    neg = (codes["signs"].astype(np.int64) >> j) & 1
    col = dim * np.arange(nv)[None, :] + j                         # [n, nv] column picked
    ref = np.einsum("nv,bnv->bn", radius * (1.0 - 2.0 * neg), xf[:, col])
    y = run_any(w, x)
    assert O.rel_err(y, ref) <= TOL
    check_bounds(y, ref, codes, cb, x, k)


@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("m", [1, 2, 4, 16, 64])
def test_zero_step_uniform_codebook_closed_form(fmt, m):
    """Every step zero and every codebook entry fp16(1/sqrt(8)): Eq. 7 gives r^ = min_G for
    every vector, so y[b, n] = c * sum_G min_(n,G) * sum_(i in G) s_(n,i) x[b, i] (a per-group
    signed sum of activations), whatever the levels and direction indices hold."""
    n, k = 75, 1024
    D, V = synth.FORMATS[fmt]
    g = synth.rng(32, n, k, m, synth.STREAM_CODES)
    codes = synth.uniform_codes(n, k, D, V, g)
    gmin, _ = synth.varied_group_params(n, k, V, g)
    codes["gmin"], codes["gstep"] = gmin, np.zeros_like(gmin)
    c16 = float(np.float16(1.0 / np.sqrt(8.0)))
    cb = synth.f16_bits(np.full((1 << D, 8), c16))
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(32, m, synth.STREAM_X))
    xf = O.f16_to_f64(x)
    bits = (codes["signs"][..., None].astype(np.int64) >> np.arange(8)) & 1
    sgn = (1.0 - 2.0 * bits).reshape(n, k)                         # s[n, i]
    per_group = np.einsum("bgi,ngi->bng", xf.reshape(m, k // 128, 128), sgn.reshape(n, k // 128, 128))
    ref = c16 * np.einsum("bng,ng->bn", per_group, O.f16_to_f64(gmin))
    y = run_any(w, x)
    assert O.rel_err(y, ref) <= TOL
    check_bounds(y, ref, codes, cb, x, k)


@pytest.mark.parametrize("fmt", ["W2", "W3", "W3_cfg", "W2_cfg", "V4", "V16"])
@pytest.mark.parametrize("m", [1, 2, 4, 8, 16, 32, 64])
def test_extreme_radii(fmt, m):
    """Radii past the fp16 range (offsets near 2^15 plus up to 15 steps of up to 2^15) and among
    the fp16 subnormals, alone and mixed within a row: every batch size stays finite and within
    its bound, output by output. The matrix-core paths scale each row's rebuilt weights by a
    power of two before rounding them to fp16."""
    n, k = 96, 1280
    D, V = synth.FORMATS[fmt]
    dim = synth.fmt_dim(fmt)
    g = synth.rng(33, n, k, synth.STREAM_CODES)
    codes = synth.uniform_codes(n, k, D, V, g, dim=dim)
    codes["gmin"], codes["gstep"] = synth.extreme_group_params(n, k, V, g)
    cb = synth.random_codebook(D, synth.rng(33, synth.STREAM_CODEBOOK), dim=dim)
    w = pkg.pack(D, V, codes, cb, device=DEV, vec_dim=dim)
    x = synth.activations(m, k, synth.rng(33, m, synth.STREAM_X))
    ref = O.gemm(codes, cb, x)
    y = run_any(w, x)
    assert np.all(np.isfinite(y))
    assert O.rel_err(y, ref) <= TOL
    check_bounds(y, ref, codes, cb, x, k)


# --------------------------------------------------------------- full-size workloads

FULL = [
    ("W2", 1024, 1024, "row", 1),            # the 1024x1024 workload's recipe: every output checked
    ("W2", 4096, 4096, "encoded", 1),        # encoded outlier-laden weights
    ("W2", 7168, 5120, "varied", 1),         # 32B-class fused q/k/v, batch 1
    ("W2", 5120, 25600, "varied", 1),        # 32B-class down, batch 1
    ("W3", 12288, 4096, "varied", 1),        # 8B-class gate/up, W3
    ("W3", 4096, 12288, "varied", 1),        # 8B-class down, W3
    ("W2", 25600, 5120, "varied", 8),        # 32B-class gate/up, batch 8
    ("W2", 5120, 25600, "varied", 4),        # 32B-class down, batch 4
    ("W2", 12288, 4096, "varied", 32),       # matrix-core path
    ("W3", 4096, 12288, "varied", 16),
    # batches 9..16 on matrices of about 10^8 weights or more run on the prefill kernel (16 batch
    # rows per workgroup); just below the bound they stay in the tile mode
    ("W3", 24576, 4096, "varied", 16),       # 96 * 2^20 weights: tile mode
    ("W2", 24576, 4096, "varied", 16),       # the same in the staged-activation tile mode
    ("W2", 32768, 4096, "varied", 12),       # 128 * 2^20: prefill
    ("W2", 24576, 4096, "varied", 12),       # below 120 * 2^20: tile mode
    ("W2", 5120, 25600, "varied", 9),        # 125 * 2^20, just above the bound: prefill
]


@pytest.mark.parametrize("fmt,n,k,kind,m", FULL)
def test_full_size_sampled(fmt, n, k, kind, m):
    if kind == "encoded":
        D, V, codes, cb = encoded_case(fmt, n, k, 9)
    else:
        D, V, codes, cb = uniform_case(fmt, n, k, 9, params=kind)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(9, m, k, synth.STREAM_X))
    y = run_any(w, x)
    g = np.random.default_rng(n + k)
    rows = np.unique(np.concatenate([[0, n - 1], g.integers(0, n, 48)]))
    if n * k <= 1 << 21:
        rows = np.arange(n)
    ref = O.gemm_rows(codes, cb, x, rows)
    # Row RMS for the metric's floor is taken over the sampled outputs.
    assert O.rel_err(y[:, rows], ref) <= TOL


# Encoded outlier-laden matrices at the benchmark configurations' full sizes, every output
# compared: the 32B-class gate/up (fused) and down projections at batch 1, 2, 4 and 8 (and the
# gate/up at 16, on the prefill kernel); the 12288x4096 and 4096x12288 projections in both
# formats at batch 1, 16 and 32; and the remaining layer shapes of the two decode steps.
ENCODED_FULL = (
    [("W2", 51200, 5120, m) for m in (1, 2, 4, 8, 16)]
    + [("W2", 5120, 25600, m) for m in (1, 2, 4, 8)]
    + [(f, n, k, m) for f in ("W2", "W3") for (n, k) in ((12288, 4096), (4096, 12288)) for m in (1, 16, 32)]
    # the other launches of the two decode steps: the 32B-class fused q/k/v and o projections at
    # batch 1, 2, 4 and 8; the 8B-class W3 fused q/k/v, o, a lone k/v and the fused gate/up at batch 1
    + [("W2", n, 5120, m) for n in (7168, 5120) for m in (1, 2, 4, 8)]
    + [("W3", n, 4096, 1) for n in (6144, 4096, 1024, 24576)]
)
_ENCODED = {}


def encoded_full(fmt, n, k):
    """Codes of an outlier-laden Gaussian matrix encoded by the oracle's encoder (Eq. 3, 5-7) in
    blocks of rows (each row is encoded on its own, so blocking changes nothing), activations
    for the largest batch used with it, and the oracle's outputs for all of them. Cached for the
    module, since several batch sizes share one matrix."""
    key = (fmt, n, k)
    if key not in _ENCODED:
        D, V = synth.FORMATS[fmt]
        cb = synth.random_codebook(D, synth.rng(21, n, k, synth.STREAM_CODEBOOK))
        rows = max(16, (1 << 22) // k)
        parts = []
        for i, a in enumerate(range(0, n, rows)):
            wblk = synth.outlier_gaussian_weights(min(rows, n - a), k, synth.rng(21, n, k, i, synth.STREAM_WEIGHTS))
            parts.append(O.encode(wblk, cb, V))
        codes = {name: np.concatenate([p[name] for p in parts]) for name in parts[0]}
        mmax = max(m for f, nn, kk, m in ENCODED_FULL if (f, nn, kk) == key)
        x = synth.activations(mmax, k, synth.rng(21, n, k, synth.STREAM_X))
        w = pkg.pack(D, V, codes, cb, device=DEV)
        _ENCODED[key] = (codes, cb, x, O.gemm(codes, cb, x), w)
    return _ENCODED[key]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("fmt,n,k,m", ENCODED_FULL)
def test_full_size_encoded_every_output(fmt, n, k, m):
    codes, cb, x, ref, w = encoded_full(fmt, n, k)
    y = run_any(w, x[:m])
    assert O.rel_err(y, ref[:m]) <= TOL
    check_bounds(y, ref[:m], codes, cb, x[:m], k)


# ------------------------------------------------------------------ prefill (batch > 32)

@pytest.mark.parametrize("fmt", FMTS)
@pytest.mark.parametrize("n,k,m", [(87, 640, 33), (300, 2048, 100), (16, 128, 64), (1, 256, 129)])
def test_prefill_gemm_parity(fmt, n, k, m):
    D, V, codes, cb = uniform_case(fmt, n, k, 5)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(5, n, k, m, synth.STREAM_X))
    y = pkg.gemm(w, to_dev_f16(x)).cpu().numpy()
    ref = O.gemm(codes, cb, x)
    if n >= 16:    # with one output per row the row-RMS floor of rel_err is |y*| itself
        assert O.rel_err(y, ref) <= TOL
    assert np.all(np.abs(y - ref) <= sum_bound(codes, cb, x, k) + 1e-30)


@pytest.mark.parametrize("fmt", ["W2", "W3"])
def test_prefill_gemm_fp16_out_strided_repeatable(fmt):
    n, k, m = 200, 1024, 80
    D, V, codes, cb = uniform_case(fmt, n, k, 6)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(6, n, k, m, synth.STREAM_X))
    xbuf = torch.zeros((m, k + 64), dtype=torch.float16, device=DEV)
    xbuf[:, :k] = to_dev_f16(x)
    ybuf = torch.full((m, n + 8), float("nan"), dtype=torch.float32, device=DEV)
    y1 = pkg.gemm(w, xbuf[:, :k], out=ybuf[:, :n]).cpu().numpy()
    y2 = pkg.gemm(w, xbuf[:, :k]).cpu().numpy()
    assert np.array_equal(y1, y2)
    assert torch.isnan(ybuf[:, n:]).all()
    y16 = pkg.gemm(w, xbuf[:, :k], out_dtype=torch.float16).cpu().numpy()
    assert np.array_equal(y16, y2.astype(np.float16))
    assert O.rel_err(y2, O.gemm(codes, cb, x)) <= TOL


@pytest.mark.parametrize("fmt", ["W2", "W3"])
def test_prefill_gemm_full_size_sampled_rows(fmt):
    """The paper's 256-token prefill on a full 12288 x 4096 projection, compared on sampled output
    rows; and the 4096 x 12288 down projection, whose smaller grid splits K."""
    for (n, k) in ((12288, 4096), (4096, 12288)):
        D, V, codes, cb = uniform_case(fmt, n, k, 7)
        w = pkg.pack(D, V, codes, cb, device=DEV)
        m = 256
        x = synth.activations(m, k, synth.rng(7, n, k, m, synth.STREAM_X))
        y = pkg.gemm(w, to_dev_f16(x)).cpu().numpy()
        rows = np.sort(np.random.default_rng(7).choice(n, 48, replace=False))
        rows[0], rows[-1] = 0, n - 1
        ref = O.gemm_rows(codes, cb, x, rows)
        assert O.rel_err(y[:, rows], ref) <= TOL


# ------------------------------------------------------------------ 4-D and 16-D vectors (Tab. 7)

DIM_FMTS = ["V4", "V16"]


def dim_case(fmt, n, k, seed):
    D, V = synth.FORMATS[fmt]
    dim = synth.fmt_dim(fmt)
    g = synth.rng(seed, n, k, dim, synth.STREAM_CODES)
    codes = synth.uniform_codes(n, k, D, V, g, dim=dim)
    codes["gmin"], codes["gstep"] = synth.varied_group_params(n, k, V, g)
    cb = synth.random_codebook(D, synth.rng(seed, n, k, dim, synth.STREAM_CODEBOOK), dim=dim)
    return D, V, dim, codes, cb


@pytest.mark.parametrize("fmt", DIM_FMTS)
def test_vector_size_unpack_bit_exact(fmt):
    D, V, dim, codes, cb = dim_case(fmt, 87, 640, 11)
    w = pkg.pack(D, V, codes, cb, device=DEV, vec_dim=dim)
    back = pkg.unpack(w)
    for key in ("signs", "dir", "q"):
        assert np.array_equal(back[key], codes[key]), key


@pytest.mark.parametrize("fmt", DIM_FMTS)
@pytest.mark.parametrize("n,k", [(87, 640), (16, 128), (1, 256), (300, 8192), (40, 4224)])
def test_vector_size_gemv_parity(fmt, n, k):
    D, V, dim, codes, cb = dim_case(fmt, n, k, 12)
    w = pkg.pack(D, V, codes, cb, device=DEV, vec_dim=dim)
    x = synth.activations(1, k, synth.rng(12, n, k, synth.STREAM_X))
    y = pkg.gemv(w, to_dev_f16(x)[0]).cpu().numpy()
    ref = O.gemv(codes, cb, x)
    if n >= 16:
        assert O.rel_err(y, ref) <= TOL
    assert np.all(np.abs(y - ref) <= sum_bound(codes, cb, x, k)[0] + 1e-30)


@pytest.mark.parametrize("fmt", DIM_FMTS)
@pytest.mark.parametrize("m", [2, 5, 17, 32, 100])
def test_vector_size_batched_parity(fmt, m):
    n, k = 75, 1152
    D, V, dim, codes, cb = dim_case(fmt, n, k, 13)
    w = pkg.pack(D, V, codes, cb, device=DEV, vec_dim=dim)
    x = synth.activations(m, k, synth.rng(13, m, k, synth.STREAM_X))
    y = pkg.gemm(w, to_dev_f16(x)).cpu().numpy()
    ref = O.gemm(codes, cb, x)
    assert O.rel_err(y, ref) <= TOL
    assert np.all(np.abs(y - ref) <= sum_bound(codes, cb, x, k) + 1e-30)


@pytest.mark.parametrize("fmt", DIM_FMTS)
def test_vector_size_full_size_sampled(fmt):
    n, k = 12288, 4096
    D, V, dim, codes, cb = dim_case(fmt, n, k, 14)
    w = pkg.pack(D, V, codes, cb, device=DEV, vec_dim=dim)
    x = synth.activations(1, k, synth.rng(14, synth.STREAM_X))
    y = pkg.gemv(w, to_dev_f16(x)[0]).cpu().numpy()
    rows = np.unique(np.concatenate([[0, n - 1], np.random.default_rng(14).integers(0, n, 48)]))
    ref = O.gemm_rows(codes, cb, x, rows)[0]
    assert O.rel_err(y[rows], ref) <= TOL


def test_graph_capture_replays():
    """A decode call whose split tiles meet in the workspace, captured into a HIP graph on a stream
    that has made one eager call (so its workspace exists before the capture): every replay, with
    other eager work and synchronizations between them, gives the eager result bit for bit. A
    capture on a stream without a workspace is refused rather than recording an allocation."""
    D, V, codes, cb = uniform_case("W2", 1024, 25600, 17)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    assert pkg.workspace_bytes(w, 1) > 0
    x = to_dev_f16(synth.activations(1, 25600, synth.rng(17, synth.STREAM_X)))[0]
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y_eager = pkg.gemv(w, x).clone()
    torch.cuda.synchronize()
    y = torch.empty_like(y_eager)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        pkg.gemv(w, x, out=y)
    for i in range(4):
        y.fill_(float("nan"))
        pkg.gemv(w, x)                      # eager work on the default stream between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager), i
    y_np = y.cpu().numpy()
    assert O.rel_err(y_np, O.gemv(codes, cb, synth.activations(1, 25600, synth.rng(17, synth.STREAM_X)))) <= TOL
    s2 = torch.cuda.Stream()
    with pytest.raises(RuntimeError, match="capture stream"):
        with torch.cuda.graph(torch.cuda.CUDAGraph(), stream=s2):
            pkg.gemv(w, x, out=y)
    torch.cuda.synchronize()


@pytest.mark.parametrize("fmt", ["W2", "W3"])
@pytest.mark.parametrize("m", [1, 2, 4, 8, 16])
@pytest.mark.parametrize("n,k", [(16, 65536), (48, 12288), (200, 20480)])
def test_split_tiles_over_workgroups(fmt, m, n, k):
    """Long rows spread over many short wave ranges: a tile's parts meet inside a workgroup, across
    two workgroups (one atomic exchange per value) and across three or more (slots and a counter;
    n = 16 with k = 65536 puts the one tile over 8 to 32 workgroups). Every batch mode is checked
    against the oracle, the workspace is zero after each call, and a second call is bitwise equal."""
    D, V, codes, cb = uniform_case(fmt, n, k, 16)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(16, m, k, synth.STREAM_X))
    xd = to_dev_f16(x)
    call = (lambda: pkg.gemv(w, xd[0])[None]) if m == 1 else (lambda: pkg.gemm_small(w, xd))
    y1 = call().cpu().numpy()
    for ws in w.workspaces.values():
        assert int(torch.count_nonzero(ws)) == 0
    y2 = call().cpu().numpy()
    assert np.array_equal(y1, y2)
    ref = O.gemm(codes, cb, x)
    assert O.rel_err(y1, ref) <= TOL
    assert np.all(np.abs(y1 - ref) <= sum_bound(codes, cb, x, k) + 1e-30)


@pytest.mark.parametrize("m", [17, 24, 32, 40])
def test_batch_workspace_left_zero(m):
    """The split-K partials of the batched kernels are cleared by the call that used them, so one
    zero-filled workspace serves every later call."""
    D, V, codes, cb = uniform_case("W2", 64, 4096, 15)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, 4096, synth.rng(15, m, synth.STREAM_X))
    y1 = pkg.gemm(w, to_dev_f16(x)).cpu().numpy()
    for (mm, _stream), ws in w.workspaces.items():
        if mm == m:
            assert int(torch.count_nonzero(ws)) == 0
    y2 = pkg.gemm(w, to_dev_f16(x)).cpu().numpy()
    assert np.array_equal(y1, y2)
    assert O.rel_err(y1, O.gemm(codes, cb, x)) <= TOL


# ---------------------------------------------------------- seeded random shapes, every output

def _random_cases(count=80, seed=11):
    """Seeded (format, n, k, m) draws across every kernel mode and both work plans: rows 1..3000,
    k up to 64 groups, batches 1..48 (the 8-D formats and the 4-D / 16-D ones)."""
    g = np.random.default_rng(seed)
    fmts = ALL_FMTS
    out = []
    for i in range(count):
        fmt = fmts[i % len(fmts)]
        n = int(g.integers(1, 3001))
        k = 128 * int(g.integers(1, 65))
        m = int(g.choice([1, 1, 2, 3, 4, 7, 8, 9, 12, 16, 17, 31, 33, 48]))
        while n * k * m > 24 << 20:   # keep the fp64 oracle within seconds
            n = max(1, n // 2)
        out.append((fmt, n, k, m))
    return out


@pytest.mark.parametrize("fmt,n,k,m", _random_cases())
def test_random_shapes_every_output(fmt, n, k, m):
    """Per-group radius parameters, ragged row counts and chunk counts: every output against the
    oracle (Eq. 4, Eq. 7), within the relative bar and the a-priori bound."""
    if fmt in DIM_FMTS:
        D, V, dim, codes, cb = dim_case(fmt, n, k, 23)
        w = pkg.pack(D, V, codes, cb, device=DEV, vec_dim=dim)
    else:
        D, V, codes, cb = uniform_case(fmt, n, k, 23)
        w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(23, n, k, m, synth.STREAM_X))
    y = run_any(w, x)
    ref = O.gemm(codes, cb, x)
    assert np.all(np.isfinite(y))
    if n >= 16:   # the relative metric's row-RMS floor needs a few rows
        assert O.rel_err(y, ref) <= TOL, (fmt, n, k, m)
    check_bounds(y, ref, codes, cb, x, k)
