"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Bars: unpacked codes bit-exact; outputs within rel_err <= 2e-3 (max |y - y*| over
max(|y*|, row RMS of y*)), the tolerance the target states for fp32 accumulation against the
fp64 oracle. The batch-1 vector-ALU path forms exact fp16 products and only rounds its fp32
sums; the batched paths (matrix cores) round each rebuilt weight to fp16 first. Each path is
also held to the a-priori bound its arithmetic gives.
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


def to_dev_f16(bits: np.ndarray):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(DEV).view(torch.float16)


def uniform_case(fmt, n, k, seed):
    D, V = synth.FORMATS[fmt]
    g = synth.rng(seed, n, k, synth.STREAM_CODES)
    codes = synth.uniform_codes(n, k, D, V, g)
    codes["gmin"], codes["gstep"] = synth.row_scale_group_params(n, k, V, g)
    cb = synth.random_codebook(D, synth.rng(seed, n, k, synth.STREAM_CODEBOOK))
    return D, V, codes, cb


def encoded_case(fmt, n, k, seed):
    D, V = synth.FORMATS[fmt]
    cb = synth.random_codebook(D, synth.rng(seed, n, k, synth.STREAM_CODEBOOK))
    w = synth.outlier_gaussian_weights(n, k, synth.rng(seed, n, k, synth.STREAM_WEIGHTS))
    return D, V, O.encode(w, cb, V), cb


def apriori_bound(codes, cb, x):
    """sum_k |w^_nk x_k| per output: the scale of fp32 summation error."""
    w = np.abs(O.decode(codes, cb))
    return np.abs(O.f16_to_f64(x)) @ w.T


def f16_weight_bound(codes, cb, x, k):
    """Error bound of the matrix-core paths: every weight is rebuilt as fp16(fp16(r) * t), at most
    2^-10 (+ fp32 radius rounding) relative error or half an fp16 subnormal step (2^-25) away
    from w^, then summed in fp32."""
    xa = np.abs(O.f16_to_f64(x))
    return (2.0**-10 + 2.0**-20 + k * 2.0**-23) * apriori_bound(codes, cb, x) + 2.0**-25 * xa.sum(axis=1)[:, None]


@pytest.mark.parametrize("fmt", FMTS)
def test_unpack_bit_exact(fmt):
    D, V, codes, cb = uniform_case(fmt, 87, 640, 1)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    back = pkg.unpack(w)
    for key in ("signs", "dir", "q"):
        assert np.array_equal(back[key], codes[key]), key


@pytest.mark.parametrize("fmt", FMTS)
# rows of at most 4096 weights take 8 rows per lane at batch 1, longer ones 16 (for the formats
# that have both): 4224 = 33 groups of 128 also leaves a ragged last step
@pytest.mark.parametrize("n,k", [(87, 640), (16, 128), (1, 256), (300, 2048), (300, 4224), (40, 8320)])
def test_gemv_parity(fmt, n, k):
    D, V, codes, cb = uniform_case(fmt, n, k, 2)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(1, k, synth.rng(2, n, k, synth.STREAM_X))
    y = pkg.gemv(w, to_dev_f16(x)[0]).cpu().numpy()
    ref = O.gemv(codes, cb, x)
    assert O.rel_err(y, ref) <= TOL
    # exact products + fp32 sums: |error| <= K * 2^-23 * sum|w x| (a loose a-priori bound)
    bound = apriori_bound(codes, cb, x)[0]
    assert np.all(np.abs(y - ref) <= k * 2.0**-23 * bound + 1e-30)
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
    assert np.all(np.abs(y - ref) <= f16_weight_bound(codes, cb, x, k) + 1e-30)
    if m == 2 and D < 13:
        # batch 2 runs on the vector ALUs with exact products, like batch 1
        assert np.all(np.abs(y - ref) <= k * 2.0**-23 * apriori_bound(codes, cb, x) + 1e-30)


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
    """x = e_c picks column c of W^: every weight the kernel rebuilds is checked (Eq. 4). The
    batch-1 and batch-2 paths return it exactly (in fp32); the matrix-core paths return its fp16
    rounding."""
    D, V, codes, cb = uniform_case("W2", 33, 256, 6)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    dense = O.decode(codes, cb)
    eye = np.eye(256)
    for c0 in range(0, 256, 32):
        x = synth.f16_bits(eye[c0:c0 + 8])                         # 8 unit vectors at once
        xd = to_dev_f16(x)
        for i in range(8):
            y1 = pkg.gemv(w, xd[i]).cpu().numpy()
            assert np.array_equal(y1, dense[:, c0 + i].astype(np.float32))
        y = pkg.gemm_small(w, xd).cpu().numpy()
        ref = dense[:, c0:c0 + 8].T
        assert np.all(np.abs(y - ref) <= (2.0**-10 + 2.0**-20) * np.abs(ref) + 2.0**-25)
        y2 = pkg.gemm_small(w, xd[2:4]).cpu().numpy()
        assert np.array_equal(y2, ref[2:4].astype(np.float32))


def test_deterministic():
    D, V, codes, cb = uniform_case("W2", 500, 4096, 7)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = to_dev_f16(synth.activations(1, 4096, synth.rng(7)))[0]
    a = pkg.gemv(w, x).clone()
    b = pkg.gemv(w, x).clone()
    assert torch.equal(a, b)


def test_bad_batch_raises():
    D, V, codes, cb = uniform_case("W2", 16, 128, 8)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = torch.zeros((33, 128), dtype=torch.float16, device=DEV)
    with pytest.raises(pkg.SphError):
        pkg.gemm_small(w, x)


# --------------------------------------------------------------- full-size workloads

FULL = [
    ("W2", 1024, 1024, "uniform", 1),        # smallest workload: every output checked
    ("W2", 4096, 4096, "encoded", 1),        # encoded outlier-laden weights
    ("W2", 7168, 5120, "uniform", 1),        # 32B-class fused q/k/v, batch 1 (16 rows per lane)
    ("W2", 5120, 25600, "uniform", 1),       # 32B-class down, batch 1
    ("W3", 12288, 4096, "uniform", 1),       # 8B-class gate/up, W3
    ("W3", 4096, 12288, "uniform", 1),       # 8B-class down, W3
    ("W2", 25600, 5120, "uniform", 8),       # 32B-class gate/up, batch 8
    ("W2", 5120, 25600, "uniform", 4),       # 32B-class down, batch 4
    ("W2", 12288, 4096, "uniform", 32),      # matrix-core path
    ("W3", 4096, 12288, "uniform", 16),
]


@pytest.mark.parametrize("fmt,n,k,kind,m", FULL)
def test_full_size_sampled(fmt, n, k, kind, m):
    D, V, codes, cb = (uniform_case if kind == "uniform" else encoded_case)(fmt, n, k, 9)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(9, m, k, synth.STREAM_X))
    xd = to_dev_f16(x)
    y = (pkg.gemv(w, xd[0])[None, :] if m == 1 else pkg.gemm_small(w, xd)).cpu().numpy()
    g = np.random.default_rng(n + k)
    rows = np.unique(np.concatenate([[0, n - 1], g.integers(0, n, 48)]))
    if n * k <= 1 << 21:
        rows = np.arange(n)
    ref = O.gemm_rows(codes, cb, x, rows)
    # Row RMS for the metric's floor is taken over the sampled outputs.
    assert O.rel_err(y[:, rows], ref) <= TOL


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
    assert np.all(np.abs(y - ref) <= f16_weight_bound(codes, cb, x, k))


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
    codes["gmin"], codes["gstep"] = synth.row_scale_group_params(n, k, V, g)
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
    bound = apriori_bound(codes, cb, x)[0]
    assert np.all(np.abs(y - ref) <= k * 2.0**-23 * bound + 1e-30)


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
    assert np.all(np.abs(y - ref) <= f16_weight_bound(codes, cb, x, k) + 1e-30)


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


@pytest.mark.parametrize("m", [17, 24, 32, 40])
def test_batch_workspace_left_zero(m):
    """The split-K partials of the batched kernels are cleared by the call that used them, so one
    zero-filled workspace serves every later call."""
    D, V, codes, cb = uniform_case("W2", 64, 4096, 15)
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, 4096, synth.rng(15, m, synth.STREAM_X))
    y1 = pkg.gemm(w, to_dev_f16(x)).cpu().numpy()
    ws = w.workspaces.get(m)
    if ws is not None:
        assert int(torch.count_nonzero(ws)) == 0
    y2 = pkg.gemm(w, to_dev_f16(x)).cpu().numpy()
    assert np.array_equal(y1, y2)
    assert O.rel_err(y1, O.gemm(codes, cb, x)) <= TOL
