"""Benchmark of the SPHQuant decode path on one MI355X.

A step is one decode forward through every linear layer of a backbone. The projections that
read the same activations are packed as one matrix, as decode engines do (q, k and v stacked
into one qkv matrix, gate and up into one gate_up matrix): per layer the launches are qkv, o,
gate_up and down, each as sph_gemv (batch 1) or sph_gemm_small (batch > 1) on its own packed
copy in HBM, so the weight stream is never served from the 256 MB Infinity Cache. The step is
captured once in a HIP graph and replayed. --unfused runs the seven projections separately.

Default workload: W2 (8 sign + 6 direction + 4 radius bits per 8-vector), 32B-class shapes
(q/o 5120x5120, k/v 1024x5120, gate/up 25600x5120, down 5120x25600), 64 layers, batch 1:
9.13 GB of packed weights per step.

Prints one JSON line: whole-step packed-weight GB/s (`value`), linear-layer tokens/s, the
roofline of the dominant kernel (the decode of the largest matrices: gate_up and down), and
the fp64 CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFS = 2500.0   # MI355X dense fp16 matrix peak
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_24875_amd", "csrc", "sph_kernels.hip")

# HBM bytes per launch of the dominant kernel from rocprofv3 FETCH_SIZE + WRITE_SIZE runs, each
# scaled by the reading of a plain device copy of known size (see profiles/). Keyed by the
# SHA-256 of the kernel source and compile flags the counters were taken with: any change to
# the kernels makes the entry stale and `traffic` is reported as null.
TRAFFIC = {
    "67117cf4e921a554fe05a4f18909f0c7791f3b968329480c31c31bb3ff178865": {
        "7168x5120-m1": 11924914, "5120x5120-m1": 8754308,
        "51200x5120-m1": 82695931, "5120x25600-m1": 41959939},
}

def kernel_source_hash() -> str:
    """SHA-256 of the kernel source followed by the compile flags (both decide the code)."""
    import hashlib
    from paper_2609_24875_amd import build as B
    h = hashlib.sha256()
    with open(KERNEL_SOURCE, "rb") as f:
        h.update(f.read())
    h.update(" ".join(B.HIPCC_FLAGS).encode())
    return h.hexdigest()


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3, help="workload id in synth.WORKLOADS")
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--fmt", default="", help="override the workload's format (e.g. W3)")
    ap.add_argument("--layers", type=int, default=0, help="override layer count (0: workload's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-read-ceiling", action="store_true",
                    help="skip the plain streaming-read ceiling measurement")
    ap.add_argument("--cpu-sample-seconds", type=float, default=15.0)
    ap.add_argument("--unfused", action="store_true", help="launch q, k, v, gate, up separately")
    ap.add_argument("--path", default="decode", choices=("decode", "encode", "train"),
                    help="decode: the default benchmark; encode: device encoder and k-means codebook; "
                         "train: pseudo-quantised weight rebuild and its straight-through backward")
    ap.add_argument("--shapes", default="",
                    help="time only these NxK shapes (comma-separated) at --batch, each rotated over "
                         ">= 512 MB of packed copies")
    ap.add_argument("--no-target-shapes", action="store_true",
                    help="skip the batch-1 W2 12288x4096 / 4096x12288 launches in the decode line")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (HBM counter calibration)")
    return ap.parse_args()


FUSED = (("qkv", ("q", "k", "v")), ("o", ("o",)), ("gate_up", ("gate", "up")), ("down", ("down",)))


def layer_shapes(wl, fused: bool):
    """((label, n, k), ...) of the launches of one layer."""
    if not fused:
        return tuple(wl.shapes)
    by = {label: (n, k) for label, n, k in wl.shapes}
    if not all(m in by for _, members in FUSED for m in members):
        return tuple(wl.shapes)
    out = []
    for label, members in FUSED:
        ks = {by[m][1] for m in members}
        assert len(ks) == 1
        out.append((label, sum(by[m][0] for m in members), ks.pop()))
    return tuple(out)


def make_layer0(wl, fmt, m, shapes):
    """Codes, codebooks and activations of layer 0's matrices (seeded, uniform codes)."""
    D, V = synth.FORMATS[fmt]
    dim = synth.fmt_dim(fmt)
    mats = []
    for mi, (label, n, k) in enumerate(shapes):
        g = synth.rng(wl_id(wl), 0, mi, synth.STREAM_CODES)
        codes = synth.uniform_codes(n, k, D, V, g, dim=dim)
        codes["gmin"], codes["gstep"] = synth.row_scale_group_params(n, k, V, g)
        cb = synth.random_codebook(D, synth.rng(wl_id(wl), 0, mi, synth.STREAM_CODEBOOK), dim=dim)
        x = synth.activations(m, k, synth.rng(wl_id(wl), 0, mi, synth.STREAM_X))
        mats.append((label, n, k, codes, cb, x))
    return mats


def wl_id(wl):
    for i, w in synth.WORKLOADS.items():
        if w is wl:
            return i
    return 99


def cpu_baseline(mats, budget_s, step_bytes_total, per_mat_bytes, layers):
    """Time the fp64 oracle (decode + dot) on whole matrices of the workload's layer shapes,
    cycling through the layer's matrices until the time budget is used; report packed-weight
    GB/s over the matrices it finished (each finished matrix counts its packed bytes)."""
    from oracle import sph as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = int(os.environ.get("OMP_NUM_THREADS") or os.cpu_count())
    done_bytes = 0
    done = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        (label, n, k, codes, cb, x), nbytes = mats[done % len(mats)], per_mat_bytes[done % len(mats)]
        O.gemm(codes, cb, x)
        done_bytes += nbytes
        done += 1
    dt = time.perf_counter() - t0
    gbs = done_bytes / dt / 1e9
    return {
        "value": round(gbs, 4),
        "unit": "GB/s",
        "cores": int(threads),
        "cpu": cpu_model(),
        "kind": "oracle",
        "sample": f"{done} matrix decodes cycling over one layer's shapes "
                  f"[{', '.join(f'{m[0]} {m[1]}x{m[2]}' for m in mats)}] of the {layers}-layer step, "
                  f"{done_bytes / 1e9:.2f} GB of packed weights in {dt:.1f} s; "
                  f"step-equivalent {step_bytes_total / gbs / 1e9:.1f} s",
    }


FP64_PEAK_TFS = 78.6   # MI355X fp64 vector peak


def cpu_model() -> str:
    """The host CPU's model name and logical CPU count (from /proc/cpuinfo where present)."""
    name = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return f"{name or 'unknown CPU'}, {os.cpu_count()} logical CPUs"


def read_ceiling(torch, dev, nbytes=2 << 30, reps=10):
    """Plain streaming-read bandwidth of this GPU (libsph_probe.so, a measurement probe outside
    the library): GB/s of one launch over a buffer far larger than the Infinity Cache, from HIP
    events on the probe's stream; the best of three access patterns (grid stride, contiguous
    8 KiB blocks per wave, one contiguous slice per workgroup) at two grid sizes, each pattern's
    best reported too. None if the probe is not built."""
    import ctypes
    from paper_2609_24875_amd import build as B
    if not os.path.exists(B.PROBE_OUT):
        return None
    lib = ctypes.CDLL(B.PROBE_OUT)
    lib.sph_probe_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_int,
                                          ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p]
    never = 0x9E3779B9   # every word is 1, so each thread's XOR fold is 0 or 1
    buf = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
    flag = torch.zeros(1, dtype=torch.int32, device=dev)
    st = torch.cuda.Stream()
    names = ("grid stride", "wave blocks of 8 KiB", "workgroup slices")
    per = {}
    for pattern, name in enumerate(names):
        for grid in (4096, 16384):
            with torch.cuda.stream(st):
                for _ in range(2):
                    lib.sph_probe_stream_read(buf.data_ptr(), nbytes, grid, pattern, flag.data_ptr(), never,
                                              st.cuda_stream)
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(st)
                for _ in range(reps):
                    if lib.sph_probe_stream_read(buf.data_ptr(), nbytes, grid, pattern, flag.data_ptr(), never,
                                                 st.cuda_stream) != 0:
                        return None
                e1.record(st)
            torch.cuda.synchronize()
            gbs = nbytes * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9
            per[name] = round(max(per.get(name, 0.0), gbs), 1)
    del buf, flag
    torch.cuda.empty_cache()
    best = max(per.values())
    return {"GB/s": best, "bytes": nbytes, "frac_of_peak": round(best / HBM_PEAK_GBS, 4),
            "kernel": "plain streaming read, 16-byte loads (libsph_probe.so), best of the access patterns",
            "patterns": per}


def encode_main(args):
    """Encoder benchmark: a step is sph_encode of one 12288x4096 fp32 matrix (the 8B-class
    gate/up shape) plus sph_kmeans_codebook on it with the paper's 65,536 samples and 20
    iterations. The dominant kernel is the Eq. 5 nearest-direction search inside the encoder:
    for small codebooks 2^D fp64 cosines of 8 terms (8 multiplies + 7 adds) per vector on the
    vector ALUs, for the 2^13-entry codebook two matrix-core passes of 16-deep fp16 products."""
    import torch

    import paper_2609_24875_amd as pkg

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    fmt = args.fmt or "W3"
    D, V = synth.FORMATS[fmt]
    n, k, ns, iters = 12288, 4096, 65536, 20
    w64 = synth.outlier_gaussian_weights(n, k, synth.rng(7, n, k, synth.STREAM_WEIGHTS))
    w32 = w64.astype(np.float32)
    cb = synth.random_codebook(D, synth.rng(7, synth.STREAM_CODEBOOK))
    wd = torch.from_numpy(w32).to(dev)
    cbd = torch.from_numpy(cb.view(np.int16)).to(dev)
    ud = torch.from_numpy(synth.rng(7, ns, synth.STREAM_CODES).random(ns)).to(dev)
    ws = torch.empty(pkg.kmeans_workspace_bytes(D, V, n, k, ns), dtype=torch.uint8, device=dev)

    def timed(fn, reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    enc = lambda: pkg.encode(D, V, wd, cbd)  # noqa: E731
    km = lambda: pkg.kmeans_codebook(D, V, wd, ud, cbd, iters, workspace=ws)  # noqa: E731
    for _ in range(args.warmup):
        enc()
        km()
    torch.cuda.synchronize()
    enc_ms = timed(enc, args.steps)
    km_ms = timed(km, max(1, args.steps // 4))
    nvec = n * k // 8
    # 2^13 entries: the search runs on the matrix cores (two passes of 16-deep fp16 products per
    # entry and vector, hi/lo split of the direction); smaller codebooks: fp64 cosines on the ALUs
    mfma = D == 13
    flops = nvec * (1 << D) * (2 * 16 * 2 if mfma else 15)
    peak = MFMA_F16_PEAK_TFS if mfma else FP64_PEAK_TFS
    out = {
        "metric": "device encoder: weights encoded per second (Eq. 3, 5-7) and k-means codebook time",
        "value": round(n * k / (enc_ms / 1e3) / 1e9, 3),
        "unit": "Gweights/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(enc_ms + km_ms, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64 (from fp32 weights)",
        "data": "synthetic: N(0, 0.02^2) weights with 0.1% Student-t outliers x20, random positive "
                "unit fp16 codebook, uniform draws",
        "config": {"workload": f"encode-{fmt}-{n}x{k}", "format": f"{fmt} (8 sign + {D} direction + "
                   f"{V} radius bits)", "kmeans_samples": ns, "kmeans_iters": iters,
                   "encode_ms": round(enc_ms, 4), "kmeans_ms": round(km_ms, 4)},
        "roofline": {"kernel": f"{'k_encode_mx' if mfma else 'k_encode'} {fmt} {n}x{k}",
                     "bound": "mfma" if mfma else "alu",
                     "achieved": round(flops / (enc_ms / 1e3) / 1e12, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(flops / (enc_ms / 1e3) / 1e12 / peak, 4),
                     "traffic": None, "flops_per_launch": flops},
    }
    if not args.no_cpu_baseline:
        from oracle import sph as O
        try:
            from threadpoolctl import threadpool_info
            threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        except Exception:
            threads = int(os.environ.get("OMP_NUM_THREADS") or os.cpu_count())
        rows, t0 = 0, time.perf_counter()
        step = 16 if D > 8 else 256
        while time.perf_counter() - t0 < args.cpu_sample_seconds and rows < n:
            O.encode(w32[rows:rows + step].astype(np.float64), cb, V)
            rows += step
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(rows * k / dt / 1e9, 6), "unit": "Gweights/s",
                               "cores": int(threads), "kind": "oracle",
                               "sample": f"oracle encode of the first {rows} of {n} rows in {dt:.1f} s"}
    print(json.dumps(out), flush=True)


def train_main(args):
    """Fine-tuning benchmark: a step rebuilds the pseudo-quantised weight of one 12288x4096 layer
    (angular codebook, softplus radius, group fake quantisation, w^ = r^ s (.) c_z) and runs its
    straight-through backward (radius and codebook gradients, then the angle-logit gradient).
    The dominant kernel is the weight rebuild, bound by HBM: per 8-D vector it reads rho (4 B),
    signs (1 B) and the direction index (2 B) and writes w^ (32 B) and r^ (4 B)."""
    import torch

    from paper_2609_24875_amd import sph as B

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    fmt = args.fmt or "W2"
    D, V = synth.FORMATS[fmt]
    n, k = 12288, 4096
    nv = k // 8
    g = np.random.default_rng(8)
    rho = (g.standard_normal((n, nv)) - 3.0).astype(np.float32)
    signs = g.integers(0, 256, (n, nv)).astype(np.uint8)
    z = g.integers(0, 1 << D, (n, nv)).astype(np.uint16)
    phi = (g.standard_normal((1 << D, 7))).astype(np.float32)
    gw = (g.standard_normal((n, k)) * 1e-3).astype(np.float32)
    perm, off = B.direction_groups(D, z)
    t = {key: torch.from_numpy(np.ascontiguousarray(v)).to(dev)
         for key, v in dict(rho=rho, signs=signs, z=z.view(np.int16), phi=phi, gw=gw, perm=perm, off=off).items()}
    c = B.angular_codebook(D, t["phi"])
    w, r_hat = B.fake_quant_forward(D, V, t["rho"], t["signs"], t["z"], c)
    ws = torch.empty(1 << 22, dtype=torch.uint8, device=dev)

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    for _ in range(args.warmup):
        B.fake_quant_forward(D, V, t["rho"], t["signs"], t["z"], c)
    fwd_ms = timed(lambda: B.fake_quant_forward(D, V, t["rho"], t["signs"], t["z"], c), args.steps)
    bwd_ms = timed(lambda: B.fake_quant_backward(D, V, t["rho"], t["signs"], t["z"], c, r_hat, t["gw"],
                                                 t["perm"], t["off"], workspace=ws), args.steps)
    ang_ms = timed(lambda: B.angular_codebook_backward(D, t["phi"], B.angular_codebook(D, t["phi"])), args.steps)
    nvec = n * nv
    fwd_bytes = nvec * (4 + 1 + 2 + 32 + 4)
    bwd_bytes = nvec * ((32 + 2 + 1 + 4 + 4) + (4 + 32 + 4 + 1))
    step_ms = fwd_ms + bwd_ms + ang_ms
    out = {
        "metric": "pseudo-quantised weight rebuild + straight-through backward: algorithmic GB/s",
        "value": round((fwd_bytes + bwd_bytes) / (step_ms / 1e3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(step_ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32 weights and gradients, f64 level decisions",
        "data": "synthetic: N(-3, 1) radius parameters, uniform signs and directions, N(0, 1) angle "
                "logits, N(0, 1e-6) weight gradients",
        "config": {"workload": f"finetune-{fmt}-{n}x{k}", "format": f"{fmt} (8 sign + {D} direction + {V} "
                   f"radius bits)", "forward_ms": round(fwd_ms, 4), "backward_ms": round(bwd_ms, 4),
                   "angular_fwd_bwd_ms": round(ang_ms, 4), "backward_bytes": bwd_bytes},
        "roofline": {"kernel": f"k_fq_forward {fmt} {n}x{k}", "bound": "hbm",
                     "achieved": round(fwd_bytes / (fwd_ms / 1e3) / 1e9, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(fwd_bytes / (fwd_ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None, "bytes_per_launch": fwd_bytes},
    }
    if not args.no_cpu_baseline:
        from oracle import sph as O
        try:
            from threadpoolctl import threadpool_info
            threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        except Exception:
            threads = int(os.environ.get("OMP_NUM_THREADS") or os.cpu_count())
        c64 = c.cpu().numpy().astype(np.float64)
        rows, t0 = 0, time.perf_counter()
        while time.perf_counter() - t0 < args.cpu_sample_seconds and rows < n:
            sl = slice(rows, rows + 256)
            O.fake_quant_weights(rho[sl].astype(np.float64), signs[sl], z[sl], c64, V)
            O.fake_quant_backward(rho[sl].astype(np.float64), signs[sl], z[sl], c64, gw[sl].astype(np.float64), V)
            rows += 256
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round((fwd_bytes + bwd_bytes) * rows / n / dt / 1e9, 4), "unit": "GB/s",
                               "cores": int(threads), "kind": "oracle",
                               "sample": f"oracle forward + backward of the first {rows} of {n} rows in {dt:.1f} s"}
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only (the kernels are single-GPU; sharding is design only); --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.path == "encode":
        return encode_main(args)
    if args.path == "train":
        return train_main(args)
    if args.shapes:
        return shapes_main(args)
    import torch

    import paper_2609_24875_amd as pkg

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    wl = synth.WORKLOADS[args.workload]
    fmt = args.fmt or wl.fmt
    D, V = synth.FORMATS[fmt]
    m = args.batch
    layers = args.layers or wl.layers
    shapes = layer_shapes(wl, not args.unfused)
    pkg.load_library()
    if args.copy_calib_mib:
        # one plain copy of known size, so that HBM byte counters can be scaled
        nb = args.copy_calib_mib << 20
        src = torch.ones(nb // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # ---- inputs: layer 0 generated and packed, then replicated per layer (distinct buffers)
    t_setup = time.perf_counter()
    mats = make_layer0(wl, fmt, m, shapes)
    packed = []
    for label, n, k, codes, cb, x in mats:
        w0 = pkg.pack(D, V, codes, cb, device=dev, vec_dim=synth.fmt_dim(fmt))
        copies = [w0] + [clone_weights(pkg, w0) for _ in range(layers - 1)]
        xd = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.float16)
        ys = [torch.empty((m, n), dtype=torch.float32, device=dev) for _ in range(layers)]
        packed.append((label, n, k, copies, xd, ys))
    step_bytes = sum(len(p[3]) * p[3][0].nbytes for p in packed)
    per_mat_bytes = [p[3][0].nbytes for p in packed]
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t_setup

    def run_step():
        for li in range(layers):
            for label, n, k, copies, xd, ys in packed:
                if m == 1:
                    pkg.gemv(copies[li], xd[0], out=ys[li][0])
                elif m <= 32:
                    pkg.gemm_small(copies[li], xd, out=ys[li])
                else:
                    pkg.gemm(copies[li], xd, out=ys[li])

    # first calls outside capture, on the capture streams: the split-tile workspaces are allocated
    # (zero-filled) per stream, and an allocation inside a capture would add a fill per launch
    stream = torch.cuda.Stream()
    s2 = torch.cuda.Stream()
    for st_ in (stream, s2):
        with torch.cuda.stream(st_):
            run_step()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=stream):
        run_step()
    torch.cuda.synchronize()

    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):             # replays, and the events, on one stream
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    gbs = step_bytes / (ms / 1e3) / 1e9

    # ---- dominant kernel: batch-m decode on the largest shapes, launched back to back over the
    # per-layer copies inside a graph; average launch duration from HIP events on its stream.
    big = [p for p in packed if p[1] * p[2] == max(q[1] * q[2] for q in packed)]
    dom_launches = []
    for label, n, k, copies, xd, ys in big:
        for li in range(layers):
            dom_launches.append((copies[li], xd, ys[li]))
    g2 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g2, stream=s2):
        for w, xd, y in dom_launches:
            if m == 1:
                pkg.gemv(w, xd[0], out=y[0])
            elif m <= 32:
                pkg.gemm_small(w, xd, out=y)
            else:
                pkg.gemm(w, xd, out=y)
    torch.cuda.synchronize()
    reps = max(3, args.steps // 2)
    d0 = torch.cuda.Event(enable_timing=True)
    d1 = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s2):
        for _ in range(2):
            g2.replay()
        torch.cuda.synchronize()
        d0.record(s2)
        for _ in range(reps):
            g2.replay()
        d1.record(s2)
    torch.cuda.synchronize()
    dom_us = d0.elapsed_time(d1) * 1e3 / (reps * len(dom_launches))
    dom_bytes = sum(w.nbytes for w, _, _ in dom_launches) / len(dom_launches)
    dom_gbs = dom_bytes / (dom_us * 1e-6) / 1e9
    dom_flops = 2.0 * m * big[0][1] * big[0][2]
    del g2

    # ---- every shape the same way: average launch over the per-layer copies (us per GEMV)
    per_shape = {}
    for label, n, k, copies, xd, ys in packed:
        gs = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gs, stream=s2):
            for li in range(layers):
                if m == 1:
                    pkg.gemv(copies[li], xd[0], out=ys[li][0])
                elif m <= 32:
                    pkg.gemm_small(copies[li], xd, out=ys[li])
                else:
                    pkg.gemm(copies[li], xd, out=ys[li])
        torch.cuda.synchronize()
        with torch.cuda.stream(s2):
            gs.replay()
            torch.cuda.synchronize()
            d0.record(s2)
            for _ in range(reps):
                gs.replay()
            d1.record(s2)
        torch.cuda.synchronize()
        us = d0.elapsed_time(d1) * 1e3 / (reps * layers)
        per_shape[f"{label} {n}x{k}"] = {"us": round(us, 3),
                                         "GB/s": round(copies[0].nbytes / (us * 1e-6) / 1e9, 1)}
        del gs
    # the batch-1 W2 shapes the HBM target is stated on, each over >= 512 MB of copies
    target = None
    if m == 1 and fmt == "W2" and not args.no_target_shapes:
        target = {f"{n}x{k}": time_shape(torch, pkg, dev, fmt, m, n, k, s2, reps=reps)
                  for n, k in TARGET_SHAPES}
    ceiling = read_ceiling(torch, dev) if not args.no_read_ceiling else None

    out = {
        "metric": "packed-weight GB/s & % HBM peak for W2/W3 sph_gemv; linear-layer tokens/s",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 activations, fp32 accumulation",
        "data": "synthetic: seeded uniform codes and per-row radius scales, random positive "
                "unit codebook, fp16 N(0,1) activations",
        "config": {
            "workload": f"{wl.name}-{fmt}-m{m}" if args.fmt else f"{wl.name}-m{m}",
            "format": f"{fmt} ({synth.fmt_dim(fmt)} sign + {D} direction + {V} radius bits per "
                      f"{synth.fmt_dim(fmt)}-vector)",
            "layers": layers,
            "shapes": [f"{label} {n}x{k}" for label, n, k, *_ in packed],
            "batch": m,
            "packed_bytes_per_step": step_bytes,
            "launches_per_step": layers * len(packed),
            "fused": "none" if args.unfused or shapes == tuple(wl.shapes) else "qkv, gate_up",
            "graph": True,
        },
        "tokens_per_s": round(m / (ms / 1e3), 2),
        "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "per_shape": per_shape,
        "target_shapes": target,
        "read_ceiling": ceiling,
        "frac_read_ceiling": round(gbs / ceiling["GB/s"], 4) if ceiling else None,
        "roofline": ({
            "kernel": f"{kernel_label(fmt, m, big[0][1], big[0][2])} on {', '.join(f'{p[1]}x{p[2]}' for p in big)}",
            "bound": "hbm",
            "achieved": round(dom_gbs, 2),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(dom_gbs / HBM_PEAK_GBS, 4),
            "traffic": TRAFFIC.get(kernel_source_hash(), {}).get(f"{big[0][1]}x{big[0][2]}-m{m}"),
            "avg_launch_us": round(dom_us, 3),
            "bytes_per_launch": int(dom_bytes),
            "frac_read_ceiling": round(dom_gbs / ceiling["GB/s"], 4) if ceiling else None,
        } if m <= 32 else {
            # batches above 32: a dense contraction on the matrix cores, 2 m n k flop per launch
            "kernel": f"{kernel_label(fmt, m, big[0][1], big[0][2])} on {', '.join(f'{p[1]}x{p[2]}' for p in big)}",
            "bound": "mfma",
            "achieved": round(dom_flops / (dom_us * 1e-6) / 1e12, 2),
            "peak": MFMA_F16_PEAK_TFS,
            "unit": "TFLOP/s",
            "frac": round(dom_flops / (dom_us * 1e-6) / 1e12 / MFMA_F16_PEAK_TFS, 4),
            "traffic": None,
            "avg_launch_us": round(dom_us, 3),
            "flops_per_launch": int(dom_flops),
        }),
        "setup_s": round(setup_s, 1),
    }
    if not args.no_cpu_baseline:
        mats_cpu = [(label, n, k, codes, cb, x) for label, n, k, codes, cb, x in mats]
        out["cpu_baseline"] = cpu_baseline(mats_cpu, args.cpu_sample_seconds, step_bytes,
                                           per_mat_bytes, layers)
    print(json.dumps(out), flush=True)


def time_shape(torch, pkg, dev, fmt, m, n, k, stream, min_bytes=512 << 20, reps=10, seed=11):
    """Microseconds per launch of one n x k matrix at batch m: seeded uniform codes with per-row
    radius scales, packed once and copied until the copies hold at least `min_bytes` (so no
    launch is served from the 256 MB Infinity Cache), launched once per copy inside a HIP graph
    and timed with HIP events on the graph's stream."""
    D, V = synth.FORMATS[fmt]
    g = synth.rng(seed, n, k, synth.STREAM_CODES)
    codes = synth.uniform_codes(n, k, D, V, g)
    codes["gmin"], codes["gstep"] = synth.row_scale_group_params(n, k, V, g)
    cb = synth.random_codebook(D, synth.rng(seed, n, k, synth.STREAM_CODEBOOK))
    x = synth.activations(m, k, synth.rng(seed, n, k, synth.STREAM_X))
    w0 = pkg.pack(D, V, codes, cb, device=dev)
    ncopy = max(16, -(-min_bytes // w0.nbytes))
    copies = [w0] + [clone_weights(pkg, w0) for _ in range(ncopy - 1)]
    xd = torch.from_numpy(x.view(np.int16)).to(dev).view(torch.float16)
    y = torch.empty((m, n), dtype=torch.float32, device=dev)

    def launch(w):
        if m == 1:
            pkg.gemv(w, xd[0], out=y[0])
        elif m <= 32:
            pkg.gemm_small(w, xd, out=y)
        else:
            pkg.gemm(w, xd, out=y)

    with torch.cuda.stream(stream):
        for w in copies:
            launch(w)                        # first calls (workspaces) outside capture
    torch.cuda.synchronize()
    gs = torch.cuda.CUDAGraph()
    with torch.cuda.graph(gs, stream=stream):
        for w in copies:
            launch(w)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        gs.replay()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            gs.replay()
        e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * ncopy)
    nbytes = w0.nbytes
    del gs, copies
    torch.cuda.empty_cache()
    return {"us": round(us, 3), "GB/s": round(nbytes / (us * 1e-6) / 1e9, 1),
            "frac_hbm_peak": round(nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "bytes_per_launch": int(nbytes), "copies": ncopy, "launches_timed": reps * ncopy}


# The batch-1 W2 shapes the HBM target is stated on (the 8B-class gate/up and down matrices).
TARGET_SHAPES = ((12288, 4096), (4096, 12288))


def shapes_main(args):
    """Per-launch timing of the shapes named by --shapes (NxK,...) at --batch, each rotated over
    at least 512 MB of packed copies; one JSON line."""
    import torch

    import paper_2609_24875_amd as pkg

    if not torch.cuda.is_available():
        raise RuntimeError("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    pkg.load_library()
    fmt = args.fmt or "W2"
    st = torch.cuda.Stream()
    res = {}
    for spec in args.shapes.split(","):
        n, k = (int(v) for v in spec.lower().split("x"))
        res[f"{n}x{k}"] = time_shape(torch, pkg, dev, fmt, args.batch, n, k, st, reps=args.steps)
        print(f"# {fmt} m={args.batch} {n}x{k}: {res[f'{n}x{k}']}", file=sys.stderr, flush=True)
    print(json.dumps({"metric": "us per launch", "fmt": fmt, "batch": args.batch, "per_shape": res}),
          flush=True)


def kernel_label(fmt, m, n=0, k=0):
    """The decode kernel variant the library picks for this format, batch and n x k matrix
    (batches 9..16 on matrices of 120 * 2^20 weights or more run on the prefill kernel)."""
    if fmt in synth.FORMAT_DIM:
        return f"k_gemm_rowvec<{fmt},MB={min(32, 1 << (m - 1).bit_length()) if m > 1 else 1}> (one wave per row)"
    if m == 1:
        return f"k_gemm_valu<{fmt},M=1> (vector ALU)"
    if m == 2 and synth.FORMATS[fmt][0] < 13:
        return f"k_gemm_valu<{fmt},M=2> (vector ALU)"
    if m <= 8:
        return f"k_gemm_valu<{fmt},M={4 if m <= 4 else 8}> (4x4x4 MFMA blocks)"
    if m <= 16 and n * k < 120 << 20:
        return f"k_gemm_valu<{fmt},M=16> (16x16x32 MFMA tiles)"
    return f"k_gemm_prefill<{fmt}> (16x16x32 MFMA, LDS-staged activations)"


def clone_weights(pkg, w):
    """A second packed copy in its own device buffer (same layout, new base pointer)."""
    buf = w.buffer.clone()
    d = type(w.desc).from_buffer_copy(w.desc)
    d.d_base = buf.data_ptr()
    return pkg.SphWeights(d, buf, w.n, w.k, w.dir_bits, w.radius_bits, vec_dim=w.vec_dim)


if __name__ == "__main__":
    main()
