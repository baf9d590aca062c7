"""Plain fp64 CPU reference of SPHQuant's representation and its decode-and-multiply.

TEST INFRASTRUCTURE ONLY. Only the test-suite, the smoke check of ``__graft_entry__`` and
the CPU-baseline leg of ``bench.py`` may import this module; the library never does. It
shares no code with the HIP path: it reads the logical codes (see ``synth``) and
computes with NumPy in fp64, step by step in the paper's order and notation.

References are to the SPHQuant paper: Sec. 1 (introduction, worked radius example),
Sec. 3.1 (spherical quantisation, Eq. 3-7), Sec. 3.3 (angular codebook, Eq. 9-10, and the
softplus radius with straight-through fake quantisation), App. A (the layer-wise procedure),
Sec. 3.4 and App. D (W2 packed layout and fused decode), App. B (payload accounting),
Tab. 7 (codebook sizes by vector dimension).

Every function here is pinned by a test in ``tests/test_oracle_pins.py`` against values
the paper prints, closed forms, invariants or brute force; none is "parity unpinned".
"""
from __future__ import annotations

import numpy as np

VEC = 8                # Sec. 3.1: rows are cut along d_in into contiguous 8-D vectors (the
                       # encoder, decoder and GEMM also take 4-D and 16-D codebooks, Tab. 7:
                       # the vector size is the codebook's second dimension)
GROUP = 128            # Sec. 3.1: a radius group is 128 consecutive scalars of one row
VPG = GROUP // VEC     # = 16 vectors per group
EPS = 1e-12            # Eq. 3's epsilon (its value is not printed; reading: 1e-12 in fp64)


# ----------------------------------------------------------------------------- helpers

def f16_to_f64(bits) -> np.ndarray:
    """fp16 bit patterns (uint16) -> exact fp64 values."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def f64_to_f16(a) -> np.ndarray:
    """fp64 -> nearest fp16, returned as bit patterns (uint16)."""
    return np.asarray(a, dtype=np.float64).astype(np.float16).view(np.uint16)


# ------------------------------------------------------------- bit budget (Sec. 3.1, App. B)

def dir_bits_for(bits_per_weight: int, dim: int = VEC) -> int:
    """Direction-index width. Sec. 3.1 gives 7B bits to the 7 angular degrees of freedom of
    an 8-D vector and spends 8 of them on the sign bits, K_dir = 7B - 8. For a k-D vector the
    same accounting reads (k-1)B - k (this generalisation is what Tab. 7's codebook sizes
    imply: 32 B, 1 KiB and 512 KiB for 4-D, 8-D and 16-D at B = 2)."""
    return (dim - 1) * bits_per_weight - dim


def codebook_bytes(dir_bits: int, dim: int = VEC, signed: bool = False) -> int:
    """fp16 storage of a 2**dir_bits-entry codebook; a signed-direction codebook needs 2**dim
    times more entries (Sec. 3.1)."""
    entries = (1 << dir_bits) * ((1 << dim) if signed else 1)
    return entries * dim * 2


def payload_bits_per_weight(bits_per_weight: int, radius_bits: int) -> float:
    """Encoded payload of an 8-D vector code, (7B + V)/8 bits per weight (App. B). Excludes
    group parameters and the codebook."""
    return (7 * bits_per_weight + radius_bits) / 8.0


# --------------------------------------------------------- spherical coordinates (Eq. 1)

def spherical_coordinates(w) -> tuple[np.ndarray, np.ndarray]:
    """Eq. 1: radius r = ||w||_2 and the k-1 angles of a k-D vector (last axis)."""
    w = np.asarray(w, dtype=np.float64)
    k = w.shape[-1]
    r = np.sqrt(np.sum(w * w, axis=-1))
    phi = np.empty(w.shape[:-1] + (k - 1,))
    for i in range(k - 2):
        tail = np.sqrt(np.sum(w[..., i:] ** 2, axis=-1))
        with np.errstate(invalid="ignore", divide="ignore"):
            c = np.where(tail > 0, w[..., i] / np.where(tail > 0, tail, 1.0), 1.0)
        phi[..., i] = np.arccos(np.clip(c, -1.0, 1.0))
    phi[..., k - 2] = np.arctan2(w[..., k - 1], w[..., k - 2])
    return r, phi


def from_spherical(r, phi) -> np.ndarray:
    """Inverse of Eq. 1 (standard hyperspherical parameterisation)."""
    r = np.asarray(r, dtype=np.float64)
    phi = np.asarray(phi, dtype=np.float64)
    k = phi.shape[-1] + 1
    out = np.empty(phi.shape[:-1] + (k,))
    sprod = np.ones(phi.shape[:-1])
    for i in range(k - 1):
        out[..., i] = sprod * np.cos(phi[..., i])
        sprod = sprod * np.sin(phi[..., i])
    out[..., k - 1] = sprod
    return r[..., None] * out


# ------------------------------------------------------------------ encoder (Eq. 3, 5-7)

def decompose(w):
    """Eq. 3 on the last axis: signs, positive-orthant vector, radius and unit direction.

    Returns (neg, w_plus, r, d) with neg[..., j] True where w_j < 0. Reading: a zero (or
    negative zero) coordinate counts as positive, since sign(0) is not defined by Eq. 3."""
    w = np.asarray(w, dtype=np.float64)
    neg = w < 0
    w_plus = np.abs(w)
    r = np.sqrt(np.sum(w_plus * w_plus, axis=-1))
    d = w_plus / np.maximum(r, EPS)[..., None]
    return neg, w_plus, r, d


def assign_directions(d, codebook, chunk: int = 4096) -> np.ndarray:
    """Eq. 5: z_i = argmax_k <d_i, c_k>; ties go to the lowest index (reading)."""
    c = np.asarray(codebook, dtype=np.float64)
    d = np.asarray(d, dtype=np.float64).reshape(-1, c.shape[-1])
    z = np.empty(d.shape[0], dtype=np.int64)
    for a in range(0, d.shape[0], chunk):
        z[a:a + chunk] = np.argmax(d[a:a + chunk] @ c.T, axis=1)
    return z


def ls_radius(w_plus, c_z) -> np.ndarray:
    """Eq. 6: pre-quantisation radius <w_+, c_z> (the least-squares scale along a unit c_z).
    Reading: the stored fp16 codebook entry is used as is, not renormalised."""
    return np.sum(np.asarray(w_plus, np.float64) * np.asarray(c_z, np.float64), axis=-1)


def group_offset_step(r_tilde, radius_bits: int):
    """Eq. 7's per-group offset and step: min over the group, (max - min)/(2**V - 1).
    ``r_tilde`` is [..., groups, 16]; returns fp16 bit patterns (reading: both stored as fp16).
    """
    r_tilde = np.asarray(r_tilde, dtype=np.float64)
    lo = r_tilde.min(axis=-1)
    hi = r_tilde.max(axis=-1)
    step = (hi - lo) / ((1 << radius_bits) - 1)
    return f64_to_f16(lo), f64_to_f16(step)


def quantize_radius(r_tilde, gmin_bits, gstep_bits, radius_bits: int) -> np.ndarray:
    """Eq. 7: q = clip(round((r~ - min)/Delta), 0, 2**V - 1) with the stored (fp16) group
    parameters. ``r_tilde`` is [..., groups, 16], params [..., groups]. Readings: round half
    to even; a zero step gives q = 0."""
    r_tilde = np.asarray(r_tilde, dtype=np.float64)
    lo = f16_to_f64(gmin_bits)[..., None]
    step = f16_to_f64(gstep_bits)[..., None]
    safe = np.where(step > 0, step, 1.0)
    t = np.where(step > 0, np.rint((r_tilde - lo) / safe), 0.0)
    return np.clip(t, 0, (1 << radius_bits) - 1).astype(np.uint8)


def signs_to_bits(neg) -> np.ndarray:
    """Pack the negative-flags of a vector (last axis) into an integer, bit j <-> coordinate j:
    a byte for 4-D and 8-D vectors, 16 bits for 16-D vectors."""
    neg = np.asarray(neg, dtype=bool)
    dim = neg.shape[-1]
    weights = (1 << np.arange(dim)).astype(np.uint32)
    bits = (neg.astype(np.uint32) * weights).sum(axis=-1)
    return bits.astype(np.uint8 if dim <= 8 else np.uint16)


def encode(w, codebook_bits, radius_bits: int, params=None) -> dict:
    """Spherical quantisation of a weight matrix W[n][k] (Sec. 3.1; App. A steps 4-6, 10,
    with a fixed codebook instead of k-means and without fine-tuning).

    Per 8-D vector: Eq. 3 decomposition, Eq. 5 direction, Eq. 6 radius, Eq. 7 group
    quantisation. ``params`` = (gmin_bits, gstep_bits) forces the group parameters; by
    default they come from the data as in Eq. 7. Returns the logical codes."""
    w = np.asarray(w, dtype=np.float64)
    n, k = w.shape
    if k % GROUP:
        raise ValueError("k must be a multiple of 128")
    c = f16_to_f64(codebook_bits)
    dim = c.shape[-1]
    vecs = w.reshape(n, k // dim, dim)
    neg, w_plus, _r, d = decompose(vecs)
    z = assign_directions(d, c).reshape(n, k // dim)
    r_tilde = ls_radius(w_plus, c[z])
    rg = r_tilde.reshape(n, k // GROUP, GROUP // dim)
    if params is None:
        gmin, gstep = group_offset_step(rg, radius_bits)
    else:
        gmin = np.broadcast_to(np.asarray(params[0], np.uint16), (n, k // GROUP)).copy()
        gstep = np.broadcast_to(np.asarray(params[1], np.uint16), (n, k // GROUP)).copy()
    q = quantize_radius(rg, gmin, gstep, radius_bits).reshape(n, k // dim)
    return {"signs": signs_to_bits(neg), "dir": z.astype(np.uint16), "q": q,
            "gmin": gmin, "gstep": gstep}


# ------------------------------------------- codebook initialisation (Sec. 3.1, Sec. 4.1)

def sample_by_squared_radius(r, u) -> np.ndarray:
    """Sec. 3.1: vector indices drawn with probability proportional to r_i^2, by the inverse of
    the cumulative distribution: sample j takes the first i whose running sum of r^2 exceeds
    u_j * (total r^2). The uniforms u_j in [0, 1) are drawn by the caller. Readings: with
    replacement; the running sum is in storage order of the vectors (row-major)."""
    r2 = np.asarray(r, dtype=np.float64).reshape(-1) ** 2
    cdf = np.cumsum(r2)
    idx = np.searchsorted(cdf, np.asarray(u, dtype=np.float64) * cdf[-1], side="right")
    return np.minimum(idx, r2.size - 1)


def spherical_kmeans(d, init_bits, iters: int):
    """Spherical k-means on unit directions d [N, 8] from the fp16 codebook ``init_bits``
    (Sec. 3.1, App. A step 6). Each iteration assigns every direction to its nearest centre by
    cosine (Eq. 5, ties to the lowest index) and moves each centre to the normalised sum of its
    directions, the unit vector with the largest summed cosine to them; a centre with no
    directions stays where it is (reading). Returns the centres (fp64) and the objective, the
    summed cosine of each iteration's assignment and finally of the returned centres."""
    c = f16_to_f64(init_bits)
    d = np.asarray(d, dtype=np.float64).reshape(-1, VEC)
    obj = []
    for _ in range(iters):
        z = assign_directions(d, c)
        obj.append(float(np.sum(np.sum(d * c[z], axis=1))))
        s = np.zeros_like(c)
        np.add.at(s, z, d)
        norm = np.linalg.norm(s, axis=1)
        c = np.where(norm[:, None] > 0, s / np.where(norm > 0, norm, 1.0)[:, None], c)
    z = assign_directions(d, c)
    obj.append(float(np.sum(np.sum(d * c[z], axis=1))))
    return c, obj


def kmeans_codebook(w, init_bits, u, iters: int = 20):
    """Radius-weighted spherical k-means codebook of a weight matrix W[n][k] (Sec. 3.1; Sec. 4.1
    uses 65,536 samples and 20 iterations): Eq. 3 decomposition of the rows' 8-D vectors,
    directions sampled by r^2 (one per uniform in ``u``), k-means from ``init_bits``. Returns the
    fp16 codebook (reading: centres rounded to fp16 for storage) and the objective trace."""
    w = np.asarray(w, dtype=np.float64)
    n, k = w.shape
    _neg, _wp, r, d = decompose(w.reshape(n, k // VEC, VEC))
    idx = sample_by_squared_radius(r, u)
    c, obj = spherical_kmeans(d.reshape(-1, VEC)[idx], init_bits, iters)
    return f64_to_f16(c), obj


# ---------------------------------------------------------------- decoder (Eq. 4 and 7)

def sign_factors(signs, dim: int = VEC) -> np.ndarray:
    """Sign bits of a vector -> the +-1 factors s of Eq. 3/4, shape [..., dim]."""
    b = np.asarray(signs).astype(np.uint32)[..., None]
    bit = (b >> np.arange(dim, dtype=np.uint32)) & 1
    return 1.0 - 2.0 * bit.astype(np.float64)


def dequantize_radius(q, gmin_bits, gstep_bits) -> np.ndarray:
    """Eq. 7: r^ = min_G + q * Delta_G, per vector; params are per group of 128 weights (16
    vectors of 8-D, 32 of 4-D, 8 of 16-D)."""
    q = np.asarray(q, dtype=np.float64)
    n, nv = q.shape
    vpg = nv // np.asarray(gmin_bits).shape[1]
    lo = np.repeat(f16_to_f64(gmin_bits), vpg, axis=1)[:, :nv]
    step = np.repeat(f16_to_f64(gstep_bits), vpg, axis=1)[:, :nv]
    return lo + q * step


def decode(codes: dict, codebook_bits) -> np.ndarray:
    """Eq. 4: w^ = r^ * s (.) c_z, assembled into the dense fp64 matrix W^[n][k]."""
    c = f16_to_f64(codebook_bits)
    dim = c.shape[-1]
    r_hat = dequantize_radius(codes["q"], codes["gmin"], codes["gstep"])
    s = sign_factors(codes["signs"], dim)
    vec = r_hat[..., None] * s * c[np.asarray(codes["dir"], dtype=np.int64)]
    n, nv = r_hat.shape
    return vec.reshape(n, nv * dim)


def _rows(codes: dict, a: int, b: int) -> dict:
    return {key: np.asarray(v)[a:b] for key, v in codes.items()}


def gemm(codes: dict, codebook_bits, x_bits, row_chunk: int = 256) -> np.ndarray:
    """Y[m][n] = sum_k W^[n][k] * x[m][k] in fp64 (the linear layer y = W x of Sec. 3.4 with
    fp16 activations), decoding W^ a block of rows at a time."""
    x = f16_to_f64(x_bits)
    if x.ndim == 1:
        x = x[None, :]
    n = np.asarray(codes["q"]).shape[0]
    y = np.empty((x.shape[0], n))
    for a in range(0, n, row_chunk):
        b = min(n, a + row_chunk)
        y[:, a:b] = x @ decode(_rows(codes, a, b), codebook_bits).T
    return y


def gemv(codes: dict, codebook_bits, x_bits) -> np.ndarray:
    """Batch-1 case of ``gemm``: y[n]."""
    return gemm(codes, codebook_bits, np.asarray(x_bits).reshape(1, -1))[0]


def gemm_rows(codes: dict, codebook_bits, x_bits, rows) -> np.ndarray:
    """``gemm`` restricted to a list of output rows: Y[m][len(rows)]."""
    rows = np.asarray(rows, dtype=np.int64)
    sub = {key: np.asarray(v)[rows] for key, v in codes.items()}
    x = f16_to_f64(x_bits)
    if x.ndim == 1:
        x = x[None, :]
    return x @ decode(sub, codebook_bits).T


# ---------------------------------------------- the W2 packed layout (Sec. 3.4, App. D)

def paper_pack_w2(signs, dir_idx, q):
    """Sec. 3.4 / App. D / Fig. 3b, W2 (D = 6, V = 4).

    One 16-bit base word per vector: bits [7:0] sign bits, [13:8] direction index,
    [15:14] the low two bits of the radius level. One 32-bit word per 128-weight group holds
    the two extra (high) radius bits of its 16 vectors; reading: vector i of the group sits at
    bits [2i+1:2i]."""
    signs = np.asarray(signs, dtype=np.uint32)
    dir_idx = np.asarray(dir_idx, dtype=np.uint32)
    q = np.asarray(q, dtype=np.uint32)
    if dir_idx.max(initial=0) >= 64 or q.max(initial=0) >= 16:
        raise ValueError("W2 codes out of range")
    base = (signs | (dir_idx << 8) | ((q & 3) << 14)).astype(np.uint16)
    n, nv = q.shape
    hi = ((q >> 2) & 3).reshape(n, nv // VPG, VPG)
    shifts = (2 * np.arange(VPG)).astype(np.uint32)
    aux = np.bitwise_or.reduce(hi << shifts, axis=-1).astype(np.uint32)
    return base, aux


def paper_unpack_w2(base, aux):
    """Inverse of ``paper_pack_w2``."""
    base = np.asarray(base, dtype=np.uint32)
    aux = np.asarray(aux, dtype=np.uint32)
    n, nv = base.shape
    signs = (base & 0xFF).astype(np.uint8)
    dir_idx = ((base >> 8) & 0x3F).astype(np.uint16)
    shifts = (2 * np.arange(VPG)).astype(np.uint32)
    hi = ((aux[..., None] >> shifts) & 3).reshape(n, nv)
    q = ((base >> 14) & 3) | (hi << 2)
    return signs, dir_idx, q.astype(np.uint8)


# --------------------------------------------------- angular codebook (Eq. 9 and Eq. 10)

def angles_from_logits(phi, eps: float = 1e-4) -> np.ndarray:
    """Eq. 10: theta_j = eps + (pi/2 - 2 eps) * sigmoid(phi_j), which keeps every angle
    strictly inside (0, pi/2). The value of eps is not printed; 1e-4 is the reading."""
    phi = np.asarray(phi, dtype=np.float64)
    return eps + (np.pi / 2 - 2 * eps) / (1.0 + np.exp(-phi))


def angular_codebook(theta) -> np.ndarray:
    """Eq. 9: a unit 8-D direction from seven hyperspherical angles,
    c_1 = cos t_1, c_i = (prod_{j<i} sin t_j) cos t_i for 2 <= i <= 7, c_8 = prod sin t_j."""
    theta = np.asarray(theta, dtype=np.float64)
    out = np.empty(theta.shape[:-1] + (VEC,))
    sprod = np.ones(theta.shape[:-1])
    for i in range(VEC - 1):
        out[..., i] = sprod * np.cos(theta[..., i])
        sprod = sprod * np.sin(theta[..., i])
    out[..., VEC - 1] = sprod
    return out


def logits_from_codebook(c, eps: float = 1e-4) -> np.ndarray:
    """Inverse of Eq. 9-10 for a positive unit direction: theta_i = atan2(||c_{i+1..8}||, c_i)
    (the angle between c's tail from coordinate i on and axis i), then phi = logit of
    t = (theta - eps) / (pi/2 - 2 eps). Reading: t is clamped to [1e-6, 1 - 1e-6], so an angle
    at or beyond the interval's ends (a zero coordinate) gives a finite phi (|phi| <= 13.8)."""
    c = np.asarray(c, dtype=np.float64)
    tail = np.sqrt(np.cumsum((c * c)[..., ::-1], axis=-1)[..., ::-1])   # ||c_{i..8}||
    theta = np.arctan2(tail[..., 1:], c[..., :VEC - 1])
    t = np.clip((theta - eps) / (np.pi / 2 - 2 * eps), 1e-6, 1 - 1e-6)
    return np.log(t) - np.log1p(-t)


def angular_codebook_backward(phi, grad_c, eps: float = 1e-4) -> np.ndarray:
    """Gradient of a loss L through Eq. 10 and Eq. 9: given dL/dc [..., 8], returns dL/dphi
    [..., 7]. With c_i = (prod_{j<i} sin t_j) cos t_i, dc_i/dt_j = c_i cot t_j for j < i,
    -(prod_{k<i} sin t_k) sin t_i for j = i (i <= 7), 0 for j > i; and c_8 = prod sin t_j
    gives dc_8/dt_j = c_8 cot t_j. Then dt_j/dphi_j = (pi/2 - 2 eps) s (1 - s), s = sigmoid."""
    phi = np.asarray(phi, dtype=np.float64)
    g = np.asarray(grad_c, dtype=np.float64)
    th = angles_from_logits(phi, eps)
    c = angular_codebook(th)
    sprod = np.ones(phi.shape[:-1])
    dth = np.zeros(phi.shape)
    for j in range(VEC - 1):
        later = np.sum(g[..., j + 1:] * c[..., j + 1:], axis=-1)        # sum over i > j
        dth[..., j] = later * np.cos(th[..., j]) / np.sin(th[..., j]) - g[..., j] * sprod * np.sin(th[..., j])
        sprod = sprod * np.sin(th[..., j])
    sg = 1.0 / (1.0 + np.exp(-phi))
    return dth * (np.pi / 2 - 2 * eps) * sg * (1.0 - sg)


# ------------------------------- pseudo-quantised module (Sec. 3.3, App. A steps 7-8)

def softplus(rho) -> np.ndarray:
    """Sec. 3.3's radius parameterisation r = softplus(rho) = log(1 + e^rho)."""
    return np.logaddexp(0.0, np.asarray(rho, dtype=np.float64))


def fake_quant_radius(rho, radius_bits: int):
    """Group-wise V-bit fake quantisation of r = softplus(rho) (Sec. 3.3, App. A step 8).
    ``rho`` is [n, k/8]; groups are 16 consecutive vectors of a row, with Eq. 7's offset (min)
    and step ((max - min) / (2^V - 1)). Readings: the offset and step are rounded to fp16, as
    the finalised codes store them, and the level is computed from the rounded values (as in
    ``encode``), half to even, 0 for a zero step. Returns (r, r_hat, q)."""
    r = softplus(rho)
    n, nv = r.shape
    rg = r.reshape(n, nv // VPG, VPG)
    lo16, st16 = group_offset_step(rg, radius_bits)
    q = quantize_radius(rg, lo16, st16, radius_bits)
    r_hat = f16_to_f64(lo16)[..., None] + q * f16_to_f64(st16)[..., None]
    return r, r_hat.reshape(n, nv), q.reshape(n, nv)


def fake_quant_weights(rho, signs, dir_idx, codebook, radius_bits: int) -> np.ndarray:
    """App. A step 8: W^ with w^_i = r^_i s_i (.) c_{z_i}, from radius parameters, fixed signs and
    direction indices and an fp64 codebook [2^D, 8] (e.g. from ``angular_codebook``)."""
    _r, r_hat, _q = fake_quant_radius(rho, radius_bits)
    c = np.asarray(codebook, dtype=np.float64)
    w = r_hat[..., None] * sign_factors(signs) * c[np.asarray(dir_idx, dtype=np.int64)]
    n, nv = r_hat.shape
    return w.reshape(n, nv * VEC)


def fake_quant_backward(rho, signs, dir_idx, codebook, grad_w, radius_bits: int):
    """Gradients of a loss L through ``fake_quant_weights`` given dL/dW^ [n, k]: the
    straight-through estimator treats the rounding of the radius as the identity
    (d r^ / d r = 1), so dL/drho_i = sigmoid(rho_i) * sum_j dL/dw^_ij s_ij c_{z_i, j}, and
    dL/dc_z = sum over vectors i with z_i = z of r^_i s_i (.) dL/dw^_i. Returns
    (dL/drho [n, k/8], dL/dcodebook [2^D, 8])."""
    rho = np.asarray(rho, dtype=np.float64)
    _r, r_hat, _q = fake_quant_radius(rho, radius_bits)
    c = np.asarray(codebook, dtype=np.float64)
    n, nv = rho.shape
    g = np.asarray(grad_w, dtype=np.float64).reshape(n, nv, VEC)
    sf = sign_factors(signs)
    z = np.asarray(dir_idx, dtype=np.int64)
    d_rhat = np.sum(g * sf * c[z], axis=-1)
    d_rho = d_rhat / (1.0 + np.exp(-rho))
    d_c = np.zeros_like(c)
    np.add.at(d_c, z.reshape(-1), (r_hat[..., None] * sf * g).reshape(-1, VEC))
    return d_rho, d_c


def init_rho(w, dir_idx, codebook) -> np.ndarray:
    """App. A steps 6-7: the pre-quantisation radius r~ = <|w_i|, c_{z_i}> (Eq. 6) mapped through
    the inverse of softplus, rho = log(e^r~ - 1). Reading: r~ is floored at 1e-6 so that rho is
    finite for a zero vector."""
    w = np.asarray(w, dtype=np.float64)
    n, k = w.shape
    c = np.asarray(codebook, dtype=np.float64)
    rt = ls_radius(np.abs(w.reshape(n, k // VEC, VEC)), c[np.asarray(dir_idx, dtype=np.int64)])
    rt = np.maximum(rt, 1e-6)
    return np.log(np.expm1(rt))


# ----------------------------------------------------------------- comparison metric

def rel_err(y, y_ref) -> float:
    """Max over outputs of |y - y*| / max(|y*|, rms of y* over its output row).

    Element-wise relative error is ill-posed where y* is near zero; the row RMS floors the
    denominator (reading of "max relative error")."""
    y = np.atleast_2d(np.asarray(y, dtype=np.float64))
    y_ref = np.atleast_2d(np.asarray(y_ref, dtype=np.float64))
    rms = np.sqrt(np.mean(y_ref * y_ref, axis=1, keepdims=True))
    den = np.maximum(np.abs(y_ref), rms)
    den = np.where(den > 0, den, 1.0)
    return float(np.max(np.abs(y - y_ref) / den)) if y.size else 0.0
