/*
 * sph.h -- C ABI of the SPHQuant decode path on MI355X (gfx950).
 *
 * SPHQuant (spherical weight-only quantisation) stores every 8-element weight vector w of a
 * matrix row, cut along the input dimension, as
 *   - 8 sign bits s            (Sec. 3.1, Eq. 3: s = sign(w), kept exactly),
 *   - a D-bit direction index z into a codebook of 2^D non-negative unit 8-D directions c_k
 *                              (Sec. 3.1, Eq. 5; K_dir = 7B - 8 bits for target width B),
 *   - a V-bit radius level q, dequantised per group of 128 weights (16 vectors) of one row as
 *     r^ = min_G + q * step_G  (Sec. 3.1, Eq. 7; "group minima and scales", App. A),
 * and rebuilds it as w^ = r^ * s (.) c_z (Eq. 4). The library's hot path multiplies the rebuilt
 * matrix with fp16 activations and accumulates in fp32 (Sec. 3.4 and App. D: fused decode in
 * registers, no dequantised weights ever written to memory).
 *
 * Conventions shared by every entry point:
 *  - W is n x k (n = d_out rows, k = d_in columns). k must be a multiple of 128 with
 *    128 <= k <= 2^20, 1 <= n <= 2^24, and ceil(n/16) * k/8 < 2^31.
 *  - Logical codes are row-major: signs/dir/q are [n][k/8], group params are [n][k/128].
 *    Sign bit j of a vector belongs to element 8v+j (least significant bit first); a set bit
 *    means the element is negative.
 *  - fp16 values (group params, codebook, activations) are passed as IEEE binary16 bit patterns.
 *  - The caller owns every buffer. The library never allocates device memory; it allocates
 *    host staging memory inside sph_pack_weights and sph_unpack only, and frees it on return.
 *  - Device pointers must be device-accessible HIP allocations of the current device, 16-byte
 *    aligned. Compute calls are asynchronous on the given stream; argument errors are detected
 *    on the host before any HIP call and reported through sph_status. Nothing throws or aborts
 *    across this ABI.
 */
#ifndef SPH_H
#define SPH_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPH_OK = 0,
  SPH_ERR_NULL = 1,               /* a required pointer is NULL                                 */
  SPH_ERR_SHAPE = 2,              /* n < 1, k not a positive multiple of 128, m out of range,   */
                                  /* leading dimension too small, or misaligned pointer         */
  SPH_ERR_UNSUPPORTED_FORMAT = 3, /* (vec_dim, dir_bits, radius_bits, group_size) not built in  */
  SPH_ERR_CODE_RANGE = 4,         /* a direction index >= 2^D or a radius level >= 2^V          */
  SPH_ERR_BAD_VALUE = 5,          /* non-finite or negative codebook entry, non-finite offset,  */
                                  /* non-finite or negative step                                */
  SPH_ERR_BUFFER_TOO_SMALL = 6,   /* device buffer smaller than sph_packed_bytes                */
  SPH_ERR_HIP = 7,                /* a HIP runtime call or kernel launch failed                 */
  SPH_ERR_BAD_DESCRIPTOR = 8      /* the sph_weights descriptor is not one this library filled  */
} sph_status;

typedef enum { SPH_F16 = 0, SPH_F32 = 1 } sph_dtype;

/* The representation (Sec. 3.1-3.2). Built-in (dir_bits, radius_bits) pairs, all with vec_dim 8
 * and group_size 128:
 *   (6, 4)  W2: 8 sign + 6 direction + 4 radius bits, the packed W2 format of Sec. 3.4 / App. D
 *   (13, 3) W3: K_dir = 7*3 - 8 = 13 with 3 radius bits (3.00 bits/weight payload, App. B)
 *   (4, 4)  16-bit vectors: 8 sign + 4 direction + 4 radius bits
 *   (6, 2)  16-bit vectors: 8 sign + 6 direction + 2 radius bits (2.00 bits/weight payload)
 *   (8, 8)  24-bit vectors: 8 sign + 8 direction + 8 radius bits
 *   (13, 4) W3 with 4 radius bits (3.125 bits/weight payload, the W3 row of Tab. 1)
 *   (6, 3), (7, 2), (8, 2)  further splits of the W2 budget from the bit-allocation study of
 *           Tab. 4 (8 sign bits + D direction + V radius bits)                                 */
typedef struct {
  int32_t vec_dim;      /* must be 8   */
  int32_t dir_bits;     /* D           */
  int32_t radius_bits;  /* V           */
  int32_t group_size;   /* must be 128 */
} sph_format;

/* A packed matrix on the device. Filled by sph_pack_weights; a plain host-side value that may be
 * copied. Points into the caller-owned device buffer; off[] and layout_version are private. */
typedef struct {
  sph_format fmt;
  int64_t n, k;
  void* d_base;
  size_t bytes;
  uint64_t off[8];
  uint32_t layout_version;
  uint32_t magic;
} sph_weights;

/* Bytes of device memory sph_pack_weights needs for an n x k matrix in format *fmt. The figure
 * covers the packed codes (rows padded to a multiple of 16), the fp16 group parameters, the
 * codebook and the lookup tables derived from it. */
sph_status sph_packed_bytes(const sph_format* fmt, int64_t n, int64_t k, size_t* bytes);

/* Validate the logical codes of an n x k matrix (Sec. 3.1, Eq. 3-7), pack them into the library's
 * device layout and copy them into d_buf (d_buf_bytes >= sph_packed_bytes). Inputs are host
 * arrays: signs uint8[n][k/8], dir_idx uint16[n][k/8] (< 2^D), radius_code uint8[n][k/8]
 * (< 2^V), group_min / group_step uint16[n][k/128] (fp16 bits: min finite, step finite and
 * >= 0), codebook uint16[2^D][8] (fp16 bits, finite and >= 0). Synchronous: returns after the
 * copy on `stream` has completed, so the host arrays may be freed. On success *out describes
 * the packed matrix. */
sph_status sph_pack_weights(const sph_format* fmt, int64_t n, int64_t k, const uint8_t* signs,
                            const uint16_t* dir_idx, const uint8_t* radius_code,
                            const uint16_t* group_min, const uint16_t* group_step,
                            const uint16_t* codebook, void* d_buf, size_t d_buf_bytes,
                            void* stream, sph_weights* out);

/* y = W^ x for one fp16 activation vector (batch 1): the fused dequantise-and-multiply GEMV of
 * Sec. 3.4 / App. D. d_x: device fp16[k]; d_y: device [n] of y_dtype (fp32 accumulation, then
 * rounded to fp16 when y_dtype is SPH_F16). d_ws/ws_bytes: device workspace of at least
 * sph_workspace_bytes(w, 1) bytes (see there; may be NULL when that is 0). The split-K sums are
 * combined in a fixed order, so repeated calls give bitwise identical results.
 * Asynchronous on `stream`. */
sph_status sph_gemv(const sph_weights* w, const void* d_x, void* d_y, sph_dtype y_dtype,
                    void* d_ws, size_t ws_bytes, void* stream);

/* Y = X W^T for 1 <= m <= 32 activation rows: d_x is device fp16[m][ldx] (ldx >= k), d_y is
 * device [m][ldy] of y_dtype (ldy >= n). Batches up to 8 run on the vector ALUs with exact fp16
 * products and fp32 accumulation; batches 9..32 round each decoded weight once to fp16 and run
 * on the matrix cores (MFMA) with fp32 accumulation. Asynchronous on `stream`. */
sph_status sph_gemm_small(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y,
                          int64_t ldy, sph_dtype y_dtype, void* d_ws, size_t ws_bytes,
                          void* stream);

/* Device workspace needed by sph_gemv (m = 1) or sph_gemm_small for this matrix and batch on
 * the current device (0 when the call needs none; d_ws may then be NULL). The workspace holds
 * split-K partial sums and one arrival counter per 16-row tile: it must be 256-byte aligned and
 * zero-filled before its first use, every call leaves it zero-filled again, and calls that may
 * run concurrently must not share one. */
sph_status sph_workspace_bytes(const sph_weights* w, int64_t m, size_t* bytes);

/* Read the packed matrix back as logical codes, on the device, with the same bit extraction the
 * compute kernels use: d_signs uint8[n][k/8], d_dir_idx uint16[n][k/8], d_radius_code
 * uint8[n][k/8] are caller-owned device arrays. For the table-lookup formats the sign bits and
 * the direction are recovered from the two lookup indices each row uses; a mismatch between the
 * direction seen through the low and the high table is reported by setting the direction to
 * 0xFFFF. Asynchronous on `stream`. Intended for bit-exactness tests. */
sph_status sph_unpack(const sph_weights* w, uint8_t* d_signs, uint16_t* d_dir_idx,
                      uint8_t* d_radius_code, void* stream);

/* Spherical quantisation of a dense matrix on the device (Sec. 3.1: Eq. 3 decomposition into signs,
 * radius and unit direction, Eq. 5 nearest direction by cosine, Eq. 6 least-squares radius
 * <|w|, c_z>, Eq. 7 per-group offset min_G, step (max_G - min_G)/(2^V - 1) and level
 * q = clip(round((r~ - min_G)/step_G), 0, 2^V - 1) with the offset and step as stored in fp16).
 * d_w: device fp32[n][ldw] (ldw >= k, ldw % 4 == 0, 16-byte aligned); d_codebook: device
 * fp16 bits [2^D][8]. Outputs are caller-owned device arrays in the layout sph_pack_weights reads:
 * d_signs uint8[n][k/8], d_dir_idx uint16[n][k/8], d_radius_code uint8[n][k/8],
 * d_group_min / d_group_step fp16 bits [n][k/128]. Arithmetic is fp64. Decisions: a coordinate is
 * negative when w < 0 (so -0 is positive); among equal cosines the lowest index wins; a radius of
 * zero divides by 1e-12 instead; rounding is to nearest, ties to even, for the level and for the
 * fp16 offset and step; a zero step gives level 0. The codebook is not validated here (a
 * non-finite or negative entry gives unspecified codes; sph_pack_weights rejects it later), and
 * non-finite weights give unspecified codes. Offsets or steps beyond the fp16 range become
 * infinite, which sph_pack_weights rejects. Asynchronous on `stream`; the result does not depend
 * on the launch or on earlier calls. */
sph_status sph_encode(const sph_format* fmt, int64_t n, int64_t k, const float* d_w, int64_t ldw,
                      const uint16_t* d_codebook, uint8_t* d_signs, uint16_t* d_dir_idx,
                      uint8_t* d_radius_code, uint16_t* d_group_min, uint16_t* d_group_step,
                      void* stream);

/* Device workspace needed by sph_kmeans_codebook for an n x k matrix and n_samples samples
 * (1 <= n_samples <= 2^24): 8 bytes per 8-D vector of the matrix (running sum of squared radii),
 * 76 bytes per sample (direction, assignment, objective part), 12 bytes per sample and codebook
 * split of the assignment (splits x samples stays below about 2^20 + n_samples), 64 bytes per
 * codebook entry (the fp64 centre), and 192 bytes per codebook entry and sample chunk for the
 * fixed-point centre sums (about 128 / ceil(2^D / 512) chunks, fewer when samples are few),
 * plus alignment. */
sph_status sph_kmeans_workspace_bytes(const sph_format* fmt, int64_t n, int64_t k, int64_t n_samples,
                                      size_t* bytes);

/* Radius-weighted spherical k-means codebook of a matrix (Sec. 3.1; Sec. 4.1 uses 65,536 samples
 * and 20 iterations). The matrix's 8-D vectors are decomposed as in sph_encode; sample j draws the
 * first vector (in row-major order) whose running sum of r^2 exceeds d_u[j] * (total r^2), so
 * vectors are drawn with replacement with probability r^2 / sum r^2; d_u is device fp64[n_samples]
 * of uniforms in [0, 1), drawn by the caller. Starting from the centres d_init (device fp16 bits
 * [2^D][8]), each of `iters` iterations assigns every sampled unit direction to its nearest centre
 * by cosine (lowest index among equals) and moves each centre to the normalised sum of its
 * directions; a centre without directions stays. d_codebook (device fp16 bits [2^D][8]) receives
 * the final centres rounded to nearest fp16. d_objective (device fp64[iters + 1], or NULL) receives
 * the summed cosine of each iteration's assignment and, last, of the final centres.
 * d_sample_idx (device int64[n_samples], or NULL) receives the drawn vector indices (row * k/8 +
 * vector). d_ws: workspace of sph_kmeans_workspace_bytes, 256-byte aligned, no initial contents;
 * concurrent calls must not share one. iters is 0..10000. fp64 arithmetic; every sum runs in a
 * fixed order, so repeated calls give bitwise identical results. Asynchronous on `stream`. */
sph_status sph_kmeans_codebook(const sph_format* fmt, int64_t n, int64_t k, const float* d_w, int64_t ldw,
                               const double* d_u, int64_t n_samples, int32_t iters,
                               const uint16_t* d_init, uint16_t* d_codebook, double* d_objective,
                               int64_t* d_sample_idx, void* d_ws, size_t ws_bytes, void* stream);

/* Whether (dir_bits, radius_bits) is one of the built-in formats: 1 yes, 0 no. */
int sph_format_supported(const sph_format* fmt);

/* Static, human-readable name of a status code. */
const char* sph_status_str(sph_status s);

#ifdef __cplusplus
}
#endif

#endif /* SPH_H */
