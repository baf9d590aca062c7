"""sph_gemm_small_noalloc (through the C ABI) against sph_gemm_small on the same inputs: bitwise
equal results on two calls in a row, the second with a smaller input, and the oracle's bar; a call
that would need more than the library's scratch array is refused."""
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


def _case(fmt, n, k, m, seed):
    D, V = synth.FORMATS[fmt]
    g = synth.rng(seed, n, k, synth.STREAM_CODES)
    codes = synth.uniform_codes(n, k, D, V, g)
    codes["gmin"], codes["gstep"] = synth.varied_group_params(n, k, V, g)
    cb = synth.random_codebook(D, synth.rng(seed, synth.STREAM_CODEBOOK))
    w = pkg.pack(D, V, codes, cb, device=DEV)
    x = synth.activations(m, k, synth.rng(seed, m, synth.STREAM_X))
    xd = torch.from_numpy(x.view(np.int16)).to(DEV).view(torch.float16)
    return w, codes, cb, x, xd


# (format, n, k, m): each pair is run in this order, the second call on a smaller input, and every
# call needs the scratch array. The first pair hands split tiles over through it across two
# workgroups (rows of 25600 weights at batch 1 and 2), the second across three and more (few tiles
# of long rows at batch 16 and 9, on the 2^13-entry codebook), the third uses it for the K-split
# partial outputs of the prefill kernel.
PAIRS = [
    (("W2", 5120, 25600, 1), ("W2", 1024, 25600, 2)),
    (("W3", 1024, 12288, 16), ("W3", 512, 8192, 9)),
    (("W2", 4096, 12288, 24), ("W2", 1024, 2048, 17)),
]


@pytest.mark.parametrize("first,second", PAIRS)
def test_noalloc_matches_workspace_call(first, second):
    for i, (fmt, n, k, m) in enumerate((first, second)):
        w, codes, cb, x, xd = _case(fmt, n, k, m, 40 + i)
        assert 0 < pkg.workspace_bytes(w, m) <= pkg.sph.NOALLOC_SCRATCH_BYTES
        y_ref = pkg.gemm_small(w, xd).cpu().numpy()
        out = torch.full((m, n), float("nan"), dtype=torch.float32, device=DEV)
        y = pkg.gemm_small_noalloc(w, xd, out).cpu().numpy()
        assert np.array_equal(y, y_ref), (fmt, n, k, m)
        rows = np.unique(np.concatenate([[0, n - 1], np.random.default_rng(n).integers(0, n, 64)]))
        assert O.rel_err(y[:, rows], O.gemm_rows(codes, cb, x, rows)) <= 2e-3
        # the scratch array is left zero-filled: a repeat gives the same bits
        y2 = pkg.gemm_small_noalloc(w, xd, torch.empty_like(out)).cpu().numpy()
        assert np.array_equal(y2, y_ref)


def test_noalloc_refuses_workspace_beyond_scratch():
    # 172160 x 3584 (a vocabulary-sized projection) at batch 8: 10760 tiles over wave ranges that
    # cross workgroups, two workspace parts of 128 values per tile, over the scratch array
    w, codes, cb, x, xd = _case("W2", 172160, 3584, 8, 45)
    assert pkg.workspace_bytes(w, 8) > pkg.sph.NOALLOC_SCRATCH_BYTES
    out = torch.empty((8, 172160), dtype=torch.float32, device=DEV)
    with pytest.raises(pkg.SphError) as e:
        pkg.gemm_small_noalloc(w, xd, out)
    assert e.value.status == 6
