"""Python binding of libsph (include/sph.h): argument marshalling only.

Every step of the decode path runs in the HIP kernels of ``libsph.so``; PyTorch supplies device
memory and the current stream. There is no CPU fallback: if the library has not been built,
importing works but every call raises ``SphLibraryMissing``.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsph.so")

SPH_F16, SPH_F32 = 0, 1

STATUS = {
    0: "SPH_OK", 1: "SPH_ERR_NULL", 2: "SPH_ERR_SHAPE", 3: "SPH_ERR_UNSUPPORTED_FORMAT",
    4: "SPH_ERR_CODE_RANGE", 5: "SPH_ERR_BAD_VALUE", 6: "SPH_ERR_BUFFER_TOO_SMALL",
    7: "SPH_ERR_HIP", 8: "SPH_ERR_BAD_DESCRIPTOR",
}

# Every symbol include/sph.h declares.
EXPORTS = ("sph_packed_bytes", "sph_pack_weights", "sph_gemv", "sph_gemm_small",
           "sph_gemm_small_noalloc", "sph_gemm", "sph_workspace_bytes", "sph_unpack", "sph_encode", "sph_kmeans_workspace_bytes",
           "sph_kmeans_codebook", "sph_angular_codebook", "sph_angular_codebook_backward",
           "sph_angular_logits", "sph_direction_groups", "sph_fake_quant_init_rho",
           "sph_fake_quant_forward", "sph_fake_quant_backward_workspace_bytes",
           "sph_fake_quant_backward", "sph_format_supported", "sph_status_str")

FORMATS = {
    "W2": (6, 4), "W3": (13, 3), "W2_cfg": (4, 4), "W3_cfg": (8, 8), "W2_16": (6, 2),
}


# Size of the library's scratch array used by sph_gemm_small_noalloc (SPH_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = 16 << 20


class SphLibraryMissing(RuntimeError):
    pass


class SphError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {STATUS.get(status, status)} ({status})")


class CFormat(ctypes.Structure):
    _fields_ = [("vec_dim", ctypes.c_int32), ("dir_bits", ctypes.c_int32),
                ("radius_bits", ctypes.c_int32), ("group_size", ctypes.c_int32)]


class CWeights(ctypes.Structure):
    _fields_ = [("fmt", CFormat), ("n", ctypes.c_int64), ("k", ctypes.c_int64),
                ("d_base", ctypes.c_void_p), ("bytes", ctypes.c_size_t),
                ("off", ctypes.c_uint64 * 8), ("layout_version", ctypes.c_uint32),
                ("magic", ctypes.c_uint32)]


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libsph.so and declare its signatures. Raises SphLibraryMissing if not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise SphLibraryMissing(f"{path} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(path)
    P, I64, SZ, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t, ctypes.c_int
    pf, pw = ctypes.POINTER(CFormat), ctypes.POINTER(CWeights)
    lib.sph_packed_bytes.argtypes = [pf, I64, I64, ctypes.POINTER(SZ)]
    lib.sph_pack_weights.argtypes = [pf, I64, I64, P, P, P, P, P, P, P, SZ, P, pw]
    lib.sph_gemv.argtypes = [pw, P, P, I32, P, SZ, P]
    lib.sph_gemm_small.argtypes = [pw, P, I64, I64, P, I64, I32, P, SZ, P]
    lib.sph_gemm.argtypes = [pw, P, I64, I64, P, I64, I32, P, SZ, P]
    lib.sph_gemm_small_noalloc.argtypes = [pw, P, I64, I64, P, I64, I32, P]
    lib.sph_workspace_bytes.argtypes = [pw, I64, ctypes.POINTER(SZ)]
    lib.sph_unpack.argtypes = [pw, P, P, P, P]
    lib.sph_encode.argtypes = [pf, I64, I64, P, I64, P, P, P, P, P, P, P]
    lib.sph_kmeans_workspace_bytes.argtypes = [pf, I64, I64, I64, ctypes.POINTER(SZ)]
    lib.sph_kmeans_codebook.argtypes = [pf, I64, I64, P, I64, P, I64, ctypes.c_int32, P, P, P, P,
                                        P, SZ, P]
    F = ctypes.c_float
    lib.sph_angular_codebook.argtypes = [I32, P, F, P, P]
    lib.sph_angular_codebook_backward.argtypes = [I32, P, F, P, P, P]
    lib.sph_angular_logits.argtypes = [I32, P, F, P, P]
    lib.sph_direction_groups.argtypes = [I32, I64, P, P, P]
    lib.sph_fake_quant_init_rho.argtypes = [pf, I64, I64, P, I64, P, P, P, P]
    lib.sph_fake_quant_forward.argtypes = [pf, I64, I64, P, P, P, P, P, I64, P, P, P, P, P]
    lib.sph_fake_quant_backward_workspace_bytes.argtypes = [I32, ctypes.POINTER(SZ)]
    lib.sph_fake_quant_backward.argtypes = [pf, I64, I64, P, P, P, P, P, P, I64, P, P, P, P, P, SZ, P]
    lib.sph_format_supported.argtypes = [pf]
    lib.sph_format_supported.restype = I32
    lib.sph_status_str.argtypes = [I32]
    lib.sph_status_str.restype = ctypes.c_char_p
    for name in ("sph_packed_bytes", "sph_pack_weights", "sph_gemv", "sph_gemm_small",
                 "sph_gemm_small_noalloc", "sph_gemm", "sph_workspace_bytes", "sph_unpack", "sph_encode", "sph_kmeans_workspace_bytes",
                 "sph_kmeans_codebook", "sph_angular_codebook", "sph_angular_codebook_backward",
                 "sph_angular_logits", "sph_direction_groups", "sph_fake_quant_init_rho",
                 "sph_fake_quant_forward", "sph_fake_quant_backward_workspace_bytes",
                 "sph_fake_quant_backward"):
        getattr(lib, name).restype = I32
    _lib = lib
    return lib


def _check(st: int, what: str):
    if st != 0:
        raise SphError(st, what)


def make_format(dir_bits: int, radius_bits: int, vec_dim: int = 8, group_size: int = 128) -> CFormat:
    return CFormat(vec_dim, dir_bits, radius_bits, group_size)


def format_supported(dir_bits: int, radius_bits: int, vec_dim: int = 8) -> bool:
    return bool(load_library().sph_format_supported(ctypes.byref(make_format(dir_bits, radius_bits, vec_dim))))


def status_str(status: int) -> str:
    return load_library().sph_status_str(status).decode()


def packed_bytes(dir_bits: int, radius_bits: int, n: int, k: int, vec_dim: int = 8) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().sph_packed_bytes(ctypes.byref(make_format(dir_bits, radius_bits, vec_dim)),
                                           n, k, ctypes.byref(out)), "sph_packed_bytes")
    return out.value


def _stream_handle(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _host(a, dtype) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


@dataclass
class SphWeights:
    """A packed matrix: the device buffer (a torch uint8 tensor) and the C descriptor."""
    desc: CWeights
    buffer: object
    n: int
    k: int
    dir_bits: int
    radius_bits: int
    workspaces: dict = field(default_factory=dict)
    vec_dim: int = 8

    @property
    def nbytes(self) -> int:
        return int(self.desc.bytes)


def pack(dir_bits: int, radius_bits: int, codes: dict, codebook, device="cuda", stream=None,
         buffer=None, vec_dim: int = 8) -> SphWeights:
    """Pack logical codes (see ``synth``) into a device buffer (allocated unless ``buffer`` is
    given) with sph_pack_weights. ``vec_dim`` 4, 8 or 16; 16-D signs are uint16 per vector."""
    import torch
    lib = load_library()
    signs = _host(codes["signs"], np.uint8 if vec_dim <= 8 else np.uint16)
    n, nv = signs.shape
    k = nv * vec_dim
    dirs = _host(codes["dir"], np.uint16)
    q = _host(codes["q"], np.uint8)
    gmin = _host(codes["gmin"], np.uint16)
    gstep = _host(codes["gstep"], np.uint16)
    cb = _host(codebook, np.uint16)
    fmt = make_format(dir_bits, radius_bits, vec_dim)
    need = packed_bytes(dir_bits, radius_bits, n, k, vec_dim)
    if buffer is None:
        buffer = torch.empty(need, dtype=torch.uint8, device=device)
    w = CWeights()
    st = lib.sph_pack_weights(ctypes.byref(fmt), n, k, signs.ctypes.data, dirs.ctypes.data,
                              q.ctypes.data, gmin.ctypes.data, gstep.ctypes.data, cb.ctypes.data,
                              buffer.data_ptr(), buffer.numel(), _stream_handle(stream),
                              ctypes.byref(w))
    _check(st, "sph_pack_weights")
    return SphWeights(w, buffer, n, k, dir_bits, radius_bits, vec_dim=vec_dim)


def workspace_bytes(w: SphWeights, m: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().sph_workspace_bytes(ctypes.byref(w.desc), m, ctypes.byref(out)),
           "sph_workspace_bytes")
    return out.value


def _workspace(w: SphWeights, m: int, device, stream=None):
    """Zero-filled workspace for (w, m) on one stream, allocated once and kept with the weights
    (the library leaves it zero-filled after every call). Calls on different streams may run
    concurrently, so each stream gets its own."""
    import torch
    nb = workspace_bytes(w, m)
    if nb == 0:
        return None, 0
    key = (m, _stream_handle(stream))
    ws = w.workspaces.get(key)
    if ws is None or ws.numel() < nb:
        if torch.cuda.is_current_stream_capturing():
            # a zero-filled allocation here would put a fill into the graph ahead of every launch
            raise RuntimeError("no workspace for this (batch, stream) yet: make one call on the "
                               "capture stream before capturing a graph")
        ws = torch.zeros(nb, dtype=torch.uint8, device=device)
        w.workspaces[key] = ws
    return ws, nb


def _check_x(w: SphWeights, x, batched: bool):
    """x must be a device fp16 tensor on the weights' device with k columns, contiguous along k:
    [k] for gemv, [m][k] (any row stride) for the batched calls."""
    import torch
    if not isinstance(x, torch.Tensor) or x.dtype != torch.float16:
        raise TypeError("x must be a torch.float16 tensor")
    if x.device != w.buffer.device:
        raise ValueError(f"x is on {x.device}, the weights on {w.buffer.device}")
    if x.dim() != (2 if batched else 1) or x.shape[-1] != w.k or (x.numel() > 0 and x.stride(-1) != 1):
        raise ValueError(f"x must be {'[m][' if batched else '['}{w.k}] with unit stride along k, "
                         f"got shape {tuple(x.shape)} and strides {tuple(x.stride())}")


def _out(w: SphWeights, x, m: int, out, out_dtype, batched: bool):
    """The output tensor: a new one, or ``out`` checked to be fp16 or fp32 on x's device, [n] for
    gemv or [m][n] (any row stride) for the batched calls, contiguous along n."""
    import torch
    if out is None:
        shape = (m, w.n) if batched else (w.n,)
        return torch.empty(shape, dtype=out_dtype or torch.float32, device=x.device)
    if out.dtype not in (torch.float16, torch.float32):
        raise TypeError("out must be torch.float16 or torch.float32")
    if out_dtype is not None and out.dtype != out_dtype:
        raise TypeError("out_dtype differs from out.dtype")
    if out.device != x.device:
        raise ValueError(f"out is on {out.device}, x on {x.device}")
    want = (m, w.n) if batched else (w.n,)
    if tuple(out.shape) != want or out.stride(-1) != 1:
        raise ValueError(f"out must have shape {want} with unit stride along n, got "
                         f"{tuple(out.shape)} and strides {tuple(out.stride())}")
    return out


def _dtype_code(t) -> int:
    import torch
    return SPH_F16 if t.dtype == torch.float16 else SPH_F32


def gemv(w: SphWeights, x, out=None, out_dtype=None, stream=None):
    """y = W^ x for a device fp16 vector x[k] (sph_gemv)."""
    _check_x(w, x, batched=False)
    out = _out(w, x, 1, out, out_dtype, batched=False)
    ws, nb = _workspace(w, 1, x.device, stream)
    st = load_library().sph_gemv(ctypes.byref(w.desc), x.data_ptr(), out.data_ptr(), _dtype_code(out),
                                 ws.data_ptr() if ws is not None else None, nb, _stream_handle(stream))
    _check(st, "sph_gemv")
    return out


def gemm_small(w: SphWeights, x, out=None, out_dtype=None, stream=None):
    """Y = X W^T for device fp16 X[m][k], 1 <= m <= 32 (sph_gemm_small)."""
    _check_x(w, x, batched=True)
    m = x.shape[0]
    out = _out(w, x, m, out, out_dtype, batched=True)
    ws, nb = _workspace(w, m, x.device, stream)
    st = load_library().sph_gemm_small(ctypes.byref(w.desc), x.data_ptr(), m, x.stride(0),
                                       out.data_ptr(), out.stride(0), _dtype_code(out),
                                       ws.data_ptr() if ws is not None else None, nb,
                                       _stream_handle(stream))
    _check(st, "sph_gemm_small")
    return out


def gemm_small_noalloc(w: SphWeights, x, out, stream=None):
    """Y = X W^T like ``gemm_small``, through sph_gemm_small_noalloc: no workspace, no allocation
    (``out`` must be given). Calls on one GPU share the library's scratch array and must not
    overlap."""
    _check_x(w, x, batched=True)
    m = x.shape[0]
    out = _out(w, x, m, out, None, batched=True)
    st = load_library().sph_gemm_small_noalloc(ctypes.byref(w.desc), x.data_ptr(), m, x.stride(0),
                                               out.data_ptr(), out.stride(0), _dtype_code(out),
                                               _stream_handle(stream))
    _check(st, "sph_gemm_small_noalloc")
    return out


def gemm(w: SphWeights, x, out=None, out_dtype=None, stream=None):
    """Y = X W^T for device fp16 X[m][k], any 1 <= m <= 65536 (sph_gemm): the matrix-core prefill
    kernel above m = 32."""
    _check_x(w, x, batched=True)
    m = x.shape[0]
    out = _out(w, x, m, out, out_dtype, batched=True)
    ws, nb = _workspace(w, m, x.device, stream)
    st = load_library().sph_gemm(ctypes.byref(w.desc), x.data_ptr(), m, x.stride(0), out.data_ptr(),
                                 out.stride(0), _dtype_code(out),
                                 ws.data_ptr() if ws is not None else None, nb, _stream_handle(stream))
    _check(st, "sph_gemm")
    return out


def unpack(w: SphWeights, stream=None) -> dict:
    """Logical codes read back through the kernels' field extraction (sph_unpack)."""
    import torch
    dev = w.buffer.device
    nv = w.k // w.vec_dim
    s = torch.empty((w.n, nv), dtype=torch.uint8 if w.vec_dim <= 8 else torch.int16, device=dev)
    d = torch.empty((w.n, nv), dtype=torch.int16, device=dev)
    q = torch.empty((w.n, nv), dtype=torch.uint8, device=dev)
    st = load_library().sph_unpack(ctypes.byref(w.desc), s.data_ptr(), d.data_ptr(), q.data_ptr(),
                                   _stream_handle(stream))
    _check(st, "sph_unpack")
    torch.cuda.synchronize(dev)
    sg = s.cpu().numpy()
    return {"signs": sg if w.vec_dim <= 8 else sg.view(np.uint16), "dir": d.cpu().numpy().view(np.uint16),
            "q": q.cpu().numpy()}


def _dev_f32_matrix(w):
    import torch
    if w.dtype != torch.float32 or w.dim() != 2 or w.stride(1) != 1 or w.stride(0) % 4 != 0:
        raise ValueError("w must be a device fp32 matrix with unit column stride and a row stride "
                         "that is a multiple of 4")
    return w


def encode(dir_bits: int, radius_bits: int, w, codebook, stream=None) -> dict:
    """Spherical quantisation of a device fp32 matrix w[n][k] against a device fp16-bit codebook
    [2^D][8] (sph_encode). Returns device tensors: signs uint8, dir int16 (bits of uint16), q
    uint8 ([n][k/8]), gmin, gstep int16 (fp16 bits, [n][k/128])."""
    import torch
    w = _dev_f32_matrix(w)
    n, k = w.shape
    dev = w.device
    cb = codebook.contiguous()
    out = {"signs": torch.empty((n, k // 8), dtype=torch.uint8, device=dev),
           "dir": torch.empty((n, k // 8), dtype=torch.int16, device=dev),
           "q": torch.empty((n, k // 8), dtype=torch.uint8, device=dev),
           "gmin": torch.empty((n, k // 128), dtype=torch.int16, device=dev),
           "gstep": torch.empty((n, k // 128), dtype=torch.int16, device=dev)}
    st = load_library().sph_encode(ctypes.byref(make_format(dir_bits, radius_bits)), n, k,
                                   w.data_ptr(), w.stride(0), cb.data_ptr(),
                                   out["signs"].data_ptr(), out["dir"].data_ptr(),
                                   out["q"].data_ptr(), out["gmin"].data_ptr(),
                                   out["gstep"].data_ptr(), _stream_handle(stream))
    _check(st, "sph_encode")
    return out


def codes_to_host(codes: dict) -> dict:
    """Device codes from ``encode`` as numpy arrays with the dtypes ``pack`` takes."""
    h = {key: v.cpu().numpy() for key, v in codes.items()}
    for key in ("dir", "gmin", "gstep"):
        h[key] = h[key].view(np.uint16)
    return h


def kmeans_workspace_bytes(dir_bits: int, radius_bits: int, n: int, k: int, n_samples: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load_library().sph_kmeans_workspace_bytes(ctypes.byref(make_format(dir_bits, radius_bits)),
                                                     n, k, n_samples, ctypes.byref(out)),
           "sph_kmeans_workspace_bytes")
    return out.value


def kmeans_codebook(dir_bits: int, radius_bits: int, w, u, init, iters: int = 20, workspace=None,
                    stream=None):
    """Radius-weighted spherical k-means codebook of a device fp32 matrix w[n][k]
    (sph_kmeans_codebook). ``u``: device fp64 uniforms, one per sample; ``init``: device fp16-bit
    centres [2^D][8]. Returns (codebook int16 [2^D][8] of fp16 bits, objective fp64 [iters + 1],
    sample indices int64 [len(u)]), all on the device."""
    import torch
    w = _dev_f32_matrix(w)
    n, k = w.shape
    dev = w.device
    ns = u.numel()
    if u.dtype != torch.float64:
        raise ValueError("u must be fp64")
    nb = kmeans_workspace_bytes(dir_bits, radius_bits, n, k, ns)
    if workspace is None or workspace.numel() < nb:
        workspace = torch.empty(nb, dtype=torch.uint8, device=dev)
    cb = torch.empty((1 << dir_bits, 8), dtype=torch.int16, device=dev)
    obj = torch.empty(iters + 1, dtype=torch.float64, device=dev)
    idx = torch.empty(ns, dtype=torch.int64, device=dev)
    init = init.contiguous()
    u = u.contiguous()
    st = load_library().sph_kmeans_codebook(
        ctypes.byref(make_format(dir_bits, radius_bits)), n, k, w.data_ptr(), w.stride(0),
        u.data_ptr(), ns, iters, init.data_ptr(), cb.data_ptr(), obj.data_ptr(), idx.data_ptr(),
        workspace.data_ptr(), workspace.numel(), _stream_handle(stream))
    _check(st, "sph_kmeans_codebook")
    return cb, obj, idx


# ------------------------------------------------------------------ fine-tuning side

ANGLE_EPS = 1e-4


def _ptr(t):
    return t.data_ptr() if t is not None else None


def angular_codebook(dir_bits: int, phi, eps: float = ANGLE_EPS, out=None, stream=None):
    """Eq. 9-10 on the device: fp32 logits [2^D][7] -> fp32 codebook [2^D][8]."""
    import torch
    phi = phi.contiguous()
    if out is None:
        out = torch.empty((1 << dir_bits, 8), dtype=torch.float32, device=phi.device)
    _check(load_library().sph_angular_codebook(dir_bits, phi.data_ptr(), eps, out.data_ptr(),
                                               _stream_handle(stream)), "sph_angular_codebook")
    return out


def angular_codebook_backward(dir_bits: int, phi, grad_c, eps: float = ANGLE_EPS, stream=None):
    import torch
    phi, grad_c = phi.contiguous(), grad_c.contiguous()
    out = torch.empty_like(phi)
    _check(load_library().sph_angular_codebook_backward(dir_bits, phi.data_ptr(), eps, grad_c.data_ptr(),
                                                        out.data_ptr(), _stream_handle(stream)),
           "sph_angular_codebook_backward")
    return out


def angular_logits(dir_bits: int, codebook, eps: float = ANGLE_EPS, stream=None):
    """Inverse of Eq. 9-10 on the device: fp32 codebook [2^D][8] -> logits [2^D][7]."""
    import torch
    cb = codebook.contiguous()
    out = torch.empty((1 << dir_bits, 7), dtype=torch.float32, device=cb.device)
    _check(load_library().sph_angular_logits(dir_bits, cb.data_ptr(), eps, out.data_ptr(),
                                             _stream_handle(stream)), "sph_angular_logits")
    return out


def direction_groups(dir_bits: int, dir_idx) -> tuple:
    """Host: (perm int32[count], offsets int64[2^D + 1]) of the vectors sorted by direction."""
    d = np.ascontiguousarray(np.asarray(dir_idx).reshape(-1), dtype=np.uint16)
    perm = np.empty(d.size, dtype=np.int32)
    off = np.empty((1 << dir_bits) + 1, dtype=np.int64)
    _check(load_library().sph_direction_groups(dir_bits, d.size, d.ctypes.data, perm.ctypes.data,
                                               off.ctypes.data), "sph_direction_groups")
    return perm, off


def fake_quant_init_rho(dir_bits: int, radius_bits: int, w, dir_idx, codebook, stream=None):
    import torch
    w = _dev_f32_matrix(w)
    n, k = w.shape
    rho = torch.empty((n, k // 8), dtype=torch.float32, device=w.device)
    _check(load_library().sph_fake_quant_init_rho(
        ctypes.byref(make_format(dir_bits, radius_bits)), n, k, w.data_ptr(), w.stride(0),
        dir_idx.contiguous().data_ptr(), codebook.contiguous().data_ptr(), rho.data_ptr(),
        _stream_handle(stream)), "sph_fake_quant_init_rho")
    return rho


def fake_quant_forward(dir_bits: int, radius_bits: int, rho, signs, dir_idx, codebook,
                       want_codes: bool = False, stream=None):
    """W^ (fp32 [n][k]) and r^ (fp32 [n][k/8]); with ``want_codes`` also the finalised levels
    and fp16 group parameters."""
    import torch
    n, nv = rho.shape
    k = nv * 8
    dev = rho.device
    w = torch.empty((n, k), dtype=torch.float32, device=dev)
    r_hat = torch.empty((n, nv), dtype=torch.float32, device=dev)
    q = gmin = gstep = None
    if want_codes:
        q = torch.empty((n, nv), dtype=torch.uint8, device=dev)
        gmin = torch.empty((n, k // 128), dtype=torch.int16, device=dev)
        gstep = torch.empty((n, k // 128), dtype=torch.int16, device=dev)
    _check(load_library().sph_fake_quant_forward(
        ctypes.byref(make_format(dir_bits, radius_bits)), n, k, rho.contiguous().data_ptr(),
        signs.contiguous().data_ptr(), dir_idx.contiguous().data_ptr(), codebook.contiguous().data_ptr(),
        w.data_ptr(), k, r_hat.data_ptr(), _ptr(q), _ptr(gmin), _ptr(gstep), _stream_handle(stream)),
        "sph_fake_quant_forward")
    if want_codes:
        return w, r_hat, {"q": q, "gmin": gmin, "gstep": gstep}
    return w, r_hat


def fake_quant_backward(dir_bits: int, radius_bits: int, rho, signs, dir_idx, codebook, r_hat, grad_w,
                        perm, offsets, workspace=None, stream=None):
    """(dL/drho fp32 [n][k/8], dL/dcodebook fp32 [2^D][8]) with the straight-through estimator."""
    import torch
    n, nv = rho.shape
    k = nv * 8
    dev = rho.device
    nb = ctypes.c_size_t(0)
    _check(load_library().sph_fake_quant_backward_workspace_bytes(dir_bits, ctypes.byref(nb)),
           "sph_fake_quant_backward_workspace_bytes")
    if workspace is None or workspace.numel() < nb.value:
        workspace = torch.empty(nb.value, dtype=torch.uint8, device=dev)
    grad_w = grad_w.contiguous()
    g_rho = torch.empty_like(rho)
    g_cb = torch.empty((1 << dir_bits, 8), dtype=torch.float32, device=dev)
    _check(load_library().sph_fake_quant_backward(
        ctypes.byref(make_format(dir_bits, radius_bits)), n, k, rho.contiguous().data_ptr(),
        signs.contiguous().data_ptr(), dir_idx.contiguous().data_ptr(), codebook.contiguous().data_ptr(),
        r_hat.contiguous().data_ptr(), grad_w.data_ptr(), grad_w.stride(0), perm.data_ptr(),
        offsets.data_ptr(), g_rho.data_ptr(), g_cb.data_ptr(), workspace.data_ptr(), workspace.numel(),
        _stream_handle(stream)), "sph_fake_quant_backward")
    return g_rho, g_cb
