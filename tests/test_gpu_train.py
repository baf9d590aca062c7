"""GPU parity of the fine-tuning kernels (angular codebook, straight-through fake quantisation)
through the C ABI against the fp64 oracle, and an end-to-end check of the pseudo-quantised module.

Bars: the angular codebook and all gradients are fp32 computations compared with fp64 within
bounds derived from fp32 rounding of their sums; the fake quantisation decides its levels in fp64
like the oracle, so levels and fp16 group parameters are compared exactly (a level may differ
only where the oracle's (r - min)/step sits within 1e-12 of a rounding boundary), and the stored
fp32 weights within one fp32 rounding.
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
from paper_2609_24875_amd import sph as B  # noqa: E402
from paper_2609_24875_amd import train as T  # noqa: E402

DEV = torch.device("cuda:0")
EPS = B.ANGLE_EPS


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    return (t if dtype is None else t.to(dtype)).to(DEV)


def case(fmt, n, k, seed):
    D, V = synth.FORMATS[fmt]
    g = np.random.default_rng(seed)
    rho = (g.standard_normal((n, k // 8)) - 3.0).astype(np.float32)
    signs = g.integers(0, 256, (n, k // 8)).astype(np.uint8)
    z = g.integers(0, 1 << D, (n, k // 8)).astype(np.uint16)
    phi = (g.standard_normal((1 << D, 7)) * 1.5).astype(np.float32)
    return D, V, rho, signs, z, phi


@pytest.mark.parametrize("D", [4, 6, 13])
def test_angular_codebook_parity(D):
    phi = (np.random.default_rng(D).standard_normal((1 << D, 7)) * 3).astype(np.float32)
    c = B.angular_codebook(D, dev(phi)).cpu().numpy()
    ref = O.angular_codebook(O.angles_from_logits(phi.astype(np.float64), EPS))
    assert np.max(np.abs(c - ref)) <= 2e-6
    assert np.all(c >= 0) and np.allclose(np.linalg.norm(c.astype(np.float64), axis=1), 1.0, atol=4e-6)
    gc = np.random.default_rng(D + 1).standard_normal((1 << D, 8)).astype(np.float32)
    gp = B.angular_codebook_backward(D, dev(phi), dev(gc)).cpu().numpy()
    gref = O.angular_codebook_backward(phi.astype(np.float64), gc.astype(np.float64), EPS)
    # each term of the sums is bounded by |g| (|c| <= 1, |cot| and |tan| <= 1/eps at the ends)
    scale = np.abs(gc).sum(axis=1, keepdims=True) * (1 + np.abs(np.tan(O.angles_from_logits(phi.astype(np.float64), EPS))))
    assert np.all(np.abs(gp - gref) <= 2e-6 * scale)


def test_angular_logits_round_trip():
    D = 6
    cb = synth.random_codebook(D, synth.rng(61))
    c32 = O.f16_to_f64(cb).astype(np.float32)
    phi = B.angular_logits(D, dev(c32)).cpu().numpy()
    ref = O.logits_from_codebook(c32.astype(np.float64), EPS)
    inner = (np.abs(ref) < 6)
    assert np.all(np.abs(phi - ref)[inner] <= 1e-3 * (1 + np.abs(ref[inner])))
    back = B.angular_codebook(D, dev(phi)).cpu().numpy()
    assert np.max(np.abs(back - c32)) <= 2e-4      # clamped angles give up to ~eps


@pytest.mark.parametrize("fmt", ["W2", "W3", "W2_cfg", "W3_cfg", "W2_16"])
@pytest.mark.parametrize("n,k", [(40, 384), (1, 128), (300, 2048)])
def test_fake_quant_forward_parity(fmt, n, k):
    D, V, rho, signs, z, phi = case(fmt, n, k, 62)
    c = B.angular_codebook(D, dev(phi))
    w, r_hat, codes = B.fake_quant_forward(D, V, dev(rho), dev(signs), dev(z.view(np.int16)), c, want_codes=True)
    c64 = c.cpu().numpy().astype(np.float64)
    r, rh_ref, q_ref = O.fake_quant_radius(rho.astype(np.float64), V)
    q = codes["q"].cpu().numpy()
    rg = r.reshape(n, -1, 16)
    lo16, st16 = O.group_offset_step(rg, V)
    assert np.array_equal(codes["gmin"].cpu().numpy().view(np.uint16), lo16)
    assert np.array_equal(codes["gstep"].cpu().numpy().view(np.uint16), st16)
    bad = q != q_ref
    if bad.any():
        x = ((rg - O.f16_to_f64(lo16)[..., None]) / O.f16_to_f64(st16)[..., None]).reshape(n, -1)
        assert np.all(np.abs(np.abs(x - np.floor(x)) - 0.5)[bad] < 1e-12)
    ok = ~bad
    assert np.array_equal(r_hat.cpu().numpy()[ok], rh_ref.astype(np.float32)[ok])
    w_ref = O.fake_quant_weights(rho.astype(np.float64), signs, z, c64, V)
    okw = np.repeat(ok, 8, axis=1)
    wg = w.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(wg - w_ref)[okw] <= (2.0**-24 + 2.0**-50) * np.abs(w_ref)[okw] + 1e-38)


@pytest.mark.parametrize("fmt", ["W2", "W3", "W2_cfg"])
def test_fake_quant_backward_parity(fmt):
    n, k = 96, 512
    D, V, rho, signs, z, phi = case(fmt, n, k, 63)
    c = B.angular_codebook(D, dev(phi))
    c64 = c.cpu().numpy().astype(np.float64)
    w, r_hat = B.fake_quant_forward(D, V, dev(rho), dev(signs), dev(z.view(np.int16)), c)
    gw = np.random.default_rng(64).standard_normal((n, k)).astype(np.float32)
    perm, off = B.direction_groups(D, z)
    args = (D, V, dev(rho), dev(signs), dev(z.view(np.int16)), c, r_hat, dev(gw), dev(perm), dev(off))
    g_rho, g_cb = B.fake_quant_backward(*args)
    g_rho2, g_cb2 = B.fake_quant_backward(*args)
    assert torch.equal(g_rho, g_rho2) and torch.equal(g_cb, g_cb2)
    d_rho, d_c = O.fake_quant_backward(rho.astype(np.float64), signs, z, c64, gw.astype(np.float64), V)
    sig = 1 / (1 + np.exp(-rho.astype(np.float64)))
    sc_rho = sig * np.sum(np.abs(gw.reshape(n, -1, 8)) * c64[z.astype(np.int64)], axis=2)
    assert np.all(np.abs(g_rho.cpu().numpy() - d_rho) <= 4e-7 * sc_rho + 1e-30)
    _r, rh, _q = O.fake_quant_radius(rho.astype(np.float64), V)
    sc_c = np.zeros_like(c64)
    np.add.at(sc_c, z.reshape(-1).astype(np.int64), (rh[..., None] * np.abs(gw.reshape(n, -1, 8))).reshape(-1, 8))
    assert np.all(np.abs(g_cb.cpu().numpy() - d_c) <= 2e-6 * sc_c + 1e-30)


def test_fake_quant_init_rho_parity():
    D, V = synth.FORMATS["W2"]
    n, k = 64, 512
    w32 = synth.outlier_gaussian_weights(n, k, synth.rng(65, n, k, synth.STREAM_WEIGHTS)).astype(np.float32)
    w32[3, :8] = 0
    cb = synth.random_codebook(D, synth.rng(65, synth.STREAM_CODEBOOK))
    c32 = O.f16_to_f64(cb).astype(np.float32)
    z = np.random.default_rng(65).integers(0, 1 << D, (n, k // 8)).astype(np.uint16)
    rho = B.fake_quant_init_rho(D, V, dev(w32), dev(z.view(np.int16)), dev(c32)).cpu().numpy()
    ref = O.init_rho(w32.astype(np.float64), z, c32.astype(np.float64))
    # compare the radii the parameters stand for: softplus(rho) against Eq. 6's radius
    assert np.allclose(O.softplus(rho.astype(np.float64)), O.softplus(ref), rtol=2e-6, atol=1e-12)


def test_module_trains_and_finalizes_to_the_decode_path():
    """A synthetic layer: teacher y = x W^T with dense outlier-laden W; the pseudo-quantised module
    (W2, k-means codebook) is tuned with Adam on (rho, phi); its loss falls; its finalised codes
    decode (oracle) to the module's weight up to the fp16 rounding of the codebook, and the packed
    codes run through sph_gemm_small within the decode path's tolerance."""
    D, V = synth.FORMATS["W2"]
    n, k, m = 256, 1024, 512
    w32 = synth.outlier_gaussian_weights(n, k, synth.rng(66, n, k, synth.STREAM_WEIGHTS)).astype(np.float32)
    wd = dev(w32)
    init = dev(synth.random_codebook(D, synth.rng(66, synth.STREAM_CODEBOOK)).view(np.int16))
    u = dev(synth.rng(66, 4096, synth.STREAM_CODES).random(4096))
    mod = T.make_module(wd, D, V, init_codebook=init, kmeans_uniforms=u, kmeans_iters=10)
    x = torch.from_numpy(np.random.default_rng(67).standard_normal((m, k)).astype(np.float32)).to(DEV)
    y_t = x @ wd.t()
    opt = torch.optim.Adam([mod.rho, mod.phi], lr=2e-3)
    losses = []
    for _ in range(60):
        opt.zero_grad()
        loss = torch.mean((mod(x) - y_t) ** 2)
        loss.backward()
        opt.step()
        losses.append(float(loss.detach()))
    assert np.all(np.isfinite(losses)) and losses[-1] < 0.95 * losses[0], losses[::10]
    codes, cb16, w_hat = mod.finalize()
    w_dec = O.decode(codes, cb16)
    wh = w_hat.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(w_dec - wh) <= 2.0**-11 * np.abs(wh) + 1e-7)
    pw = pkg.pack(D, V, codes, cb16, device=DEV)
    x16 = synth.f16_bits(x[:32].cpu().numpy())
    y = pkg.gemm_small(pw, dev(x16.view(np.int16)).view(torch.float16)).cpu().numpy()
    assert O.rel_err(y, O.gemm(codes, cb16, x16)) <= 2e-3
