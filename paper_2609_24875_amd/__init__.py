"""SPHQuant decode path for MI355X (gfx950): C-ABI library libsph.so and its Python binding."""
from .sph import (EXPORTS, FORMATS, LIB_PATH, SphError, SphLibraryMissing, SphWeights,  # noqa: F401
                  codes_to_host, encode, format_supported, gemm, gemm_small, gemm_small_noalloc, gemv,
                  kmeans_codebook, kmeans_workspace_bytes, load_library, pack, packed_bytes, status_str,
                  unpack, workspace_bytes)
