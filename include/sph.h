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
 *  - Logical codes are row-major: signs/dir/q are [n][k/8] (k/vec_dim for the 4-D and 16-D
 *    formats), group params are [n][k/128]. Sign bit j of a vector belongs to element 8v+j
 *    (least significant bit first); a set bit means the element is negative.
 *  - fp16 values (group params, codebook, activations) are passed as IEEE binary16 bit patterns.
 *  - The caller owns every buffer. The library never allocates device memory; it allocates
 *    host staging memory inside sph_pack_weights only, and frees it on return.
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
  SPH_ERR_BAD_VALUE = 5,          /* codebook entry non-finite, negative or above 2; offset     */
                                  /* non-finite; step non-finite or negative                    */
  SPH_ERR_BUFFER_TOO_SMALL = 6,   /* device buffer smaller than sph_packed_bytes                */
  SPH_ERR_HIP = 7,                /* a HIP runtime call or kernel launch failed                 */
  SPH_ERR_BAD_DESCRIPTOR = 8      /* the sph_weights descriptor is not one this library filled  */
} sph_status;

typedef enum { SPH_F16 = 0, SPH_F32 = 1 } sph_dtype;

/* The representation (Sec. 3.1-3.2). Built-in (dir_bits, radius_bits) pairs with vec_dim 8 and
 * group_size 128:
 *   (6, 4)  W2: 8 sign + 6 direction + 4 radius bits, the packed W2 format of Sec. 3.4 / App. D
 *   (13, 3) W3: K_dir = 7*3 - 8 = 13 with 3 radius bits (3.00 bits/weight payload, App. B)
 *   (4, 4)  16-bit vectors: 8 sign + 4 direction + 4 radius bits
 *   (6, 2)  16-bit vectors: 8 sign + 6 direction + 2 radius bits (2.00 bits/weight payload)
 *   (8, 8)  24-bit vectors: 8 sign + 8 direction + 8 radius bits
 *   (13, 4) W3 with 4 radius bits (3.125 bits/weight payload, the W3 row of Tab. 1)
 *   (6, 3), (7, 2), (8, 2)  further splits of the W2 budget from the bit-allocation study of
 *           Tab. 4 (8 sign bits + D direction + V radius bits)
 * and the other vector sizes of Tab. 7 (group_size 128): vec_dim 4 with (2, 3) (4 sign + 2 direction
 * + 3 radius bits) and vec_dim 16 with (14, 6) (16 sign + 14 direction + 6 radius bits); for vec_dim
 * 16 the sign array holds one uint16 per vector.                                               */
typedef struct {
  int32_t vec_dim;      /* 8, or 4 / 16 with the pairs above */
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
 * >= 0), codebook uint16[2^D][vec_dim] (fp16 bits, in [0, 2]: coordinates of non-negative unit
 * directions, Sec. 3.1, with room for rounding). Synchronous: returns after the
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
 * device [m][ldy] of y_dtype (ldy >= n). Every batch size forms exact products of fp16 numbers
 * and rounds only fp32 sums: batch 1, and batch 2 for formats with at most 8 direction bits, on the
 * vector ALUs (signed direction times activations, then times the fp32 radius); batches 3..8 on
 * 4x4x4 MFMA blocks, one vector per block, each block's sum times the fp32 radius; batches 9..32
 * on 16x16x32 MFMA tiles with Eq. 7 factored over each 128-weight group, offset * sum <t, x> +
 * step * sum q <t, x>, where t (the signed direction) and q * t (split exactly into two fp16
 * numbers) are the operands (9..16 inside the step plan; 17..32, and 9..16 on matrices of about
 * 10^8 weights or more, in the prefill kernel of sph_gemm with 16 or 32 activation rows staged in
 * LDS). Asynchronous on `stream`. */
sph_status sph_gemm_small(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y,
                          int64_t ldy, sph_dtype y_dtype, void* d_ws, size_t ws_bytes,
                          void* stream);

/* Y = X W^T for any batch 1 <= m <= 65536 (prefill and large batches): m <= 32 is sph_gemm_small;
 * larger batches run on the matrix cores (16x16x32 fp16 MFMA, fp32 accumulation) with the
 * factored exact-product arithmetic of sph_gemm_small's batches above 8, each weight's operands
 * rebuilt once per 64-row slice of X and per 128-column chunk of K. Same argument rules as
 * sph_gemm_small. When the
 * grid would not cover the chip, K is split and fp32 partial outputs go through the workspace
 * (sph_workspace_bytes(w, m); for m > 32 it needs no zero-fill) and are added in a fixed order,
 * so repeated calls give bitwise identical results. Asynchronous on `stream`. */
sph_status sph_gemm(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y, int64_t ldy,
                    sph_dtype y_dtype, void* d_ws, size_t ws_bytes, void* stream);

/* sph_gemm_small without a caller workspace, for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid allocation). Same arguments,
 * arithmetic, results (bitwise) and errors as sph_gemm_small, with d_ws/ws_bytes replaced by a
 * fixed array of SPH_NOALLOC_SCRATCH_BYTES in device memory that the library's code object holds
 * (one per GPU it runs on, kept until the process ends). A call whose sph_workspace_bytes exceeds
 * that size returns SPH_ERR_BUFFER_TOO_SMALL before any HIP call. The first call on a device looks
 * up the array's address and clears it with a kernel on `stream`; every call leaves it zero-filled
 * again. Every call on one GPU shares that GPU's array: calls that may overlap on one GPU (other
 * streams, other threads) race and must not be made. Allocates nothing, on the host or the device.
 * Asynchronous on `stream`. */
#define SPH_NOALLOC_SCRATCH_BYTES (16u << 20)
sph_status sph_gemm_small_noalloc(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y,
                                  int64_t ldy, sph_dtype y_dtype, void* stream);

/* Device workspace needed by sph_gemv (m = 1), sph_gemm_small or sph_gemm for this matrix and
 * batch (1 <= m <= 65536) on the current device (0 when the call needs none; d_ws may then be
 * NULL). For m <= 16 it holds the partial sums of 16-row tiles whose K range is split between
 * workgroups: 64-bit words (fp32 sum and a valid flag), one per value of a tile over two
 * workgroups, one per workgroup and value of a tile over more, and one 32-bit arrival counter per
 * tile; where the prefill kernel runs (m above 16, and 9..16 on large matrices: see
 * sph_gemm_small) it holds fp32 partial outputs of a K split. It must be 256-byte
 * aligned and zero-filled before its first use, and every call leaves it zero-filled again (above
 * m = 32 it needs no initial contents, but is still left zero-filled). Calls that may run
 * concurrently must not share one. No call waits for another workgroup to make progress, so calls
 * on other streams may occupy any part of the GPU meanwhile. */
sph_status sph_workspace_bytes(const sph_weights* w, int64_t m, size_t* bytes);

/* Read the packed matrix back as logical codes, on the device, with the same bit extraction the
 * compute kernels use: d_signs uint8[n][k/vec_dim] (uint16 for vec_dim 16), d_dir_idx
 * uint16[n][k/vec_dim], d_radius_code uint8[n][k/vec_dim] are caller-owned DEVICE arrays, written
 * asynchronously on `stream`; the caller copies them to the host and synchronizes. (A host-array,
 * synchronous form would need device staging memory, and the library never allocates device
 * memory; the Python binding does the copy.) For the table-lookup formats the sign bits and the
 * direction are recovered from the two lookup indices each row uses; a mismatch between the
 * direction seen through the low and the high table is reported by setting the direction to
 * 0xFFFF. Intended for bit-exactness tests. */
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

/* ---- Fine-tuning side (Sec. 3.3; App. A steps 6-10). fp32 device arrays unless stated. ---- */

/* Angular codebook (Sec. 3.3, Eq. 9-10): for each of the 2^D entries, seven angle logits phi
 * (d_phi fp32[2^D][7]) give theta_j = eps + (pi/2 - 2 eps) sigmoid(phi_j) and the positive unit
 * direction c_1 = cos t_1, c_i = (prod_{j<i} sin t_j) cos t_i (2 <= i <= 7), c_8 = prod_j sin t_j,
 * written to d_codebook fp32[2^D][8]. 1 <= dir_bits <= 13, 0 <= eps < 0.25. Asynchronous. */
sph_status sph_angular_codebook(int32_t dir_bits, const float* d_phi, float eps, float* d_codebook, void* stream);

/* Gradient of a loss through sph_angular_codebook: d_grad_codebook fp32[2^D][8] (dL/dc) gives
 * d_grad_phi fp32[2^D][7] (dL/dphi), from the closed-form derivatives of Eq. 9 and Eq. 10. */
sph_status sph_angular_codebook_backward(int32_t dir_bits, const float* d_phi, float eps,
                                         const float* d_grad_codebook, float* d_grad_phi, void* stream);

/* Inverse of Eq. 9-10 (initialises the angle logits from a codebook, App. A step 7):
 * theta_i = atan2(||c_{i+1..8}||, c_i), t = (theta - eps)/(pi/2 - 2 eps) clamped to
 * [1e-6, 1 - 1e-6], phi = log t - log(1 - t). d_codebook fp32[2^D][8] of non-negative unit
 * directions; d_phi fp32[2^D][7]. */
sph_status sph_angular_logits(int32_t dir_bits, const float* d_codebook, float eps, float* d_phi, void* stream);

/* Host-only, synchronous: the vectors grouped by direction index, for the codebook gradient
 * of sph_fake_quant_backward. dir_idx: host uint16[count] (< 2^D); perm: host int32[count]
 * receives the vector indices sorted by direction, stably (ascending index within a
 * direction); offsets: host int64[2^D + 1], direction z owns perm[offsets[z] .. offsets[z+1]).
 * 1 <= count < 2^31. SPH_ERR_CODE_RANGE for an index >= 2^D. */
sph_status sph_direction_groups(int32_t dir_bits, int64_t count, const uint16_t* dir_idx, int32_t* perm,
                                int64_t* offsets);

/* Radius parameters from a dense matrix (App. A steps 6-7): rho_i = log(exp(r~_i) - 1), the
 * inverse of softplus, of Eq. 6's radius r~_i = <|w_i|, c_{z_i}> floored at 1e-6. d_w fp32[n][ldw]
 * (ldw >= k, ldw % 4 == 0, 16-byte aligned), d_dir_idx uint16[n][k/8], d_codebook fp32[2^D][8]
 * (16-byte aligned), d_rho fp32[n][k/8]. */
sph_status sph_fake_quant_init_rho(const sph_format* fmt, int64_t n, int64_t k, const float* d_w, int64_t ldw,
                                   const uint16_t* d_dir_idx, const float* d_codebook, float* d_rho, void* stream);

/* The pseudo-quantised weight of a linear module (Sec. 3.3; App. A step 8): r = softplus(rho),
 * group-wise V-bit fake quantisation with Eq. 7's offset min_G and step (max_G - min_G)/(2^V - 1),
 * both rounded to fp16 as the finalised codes store them, q = clip(round((r - min_G)/step_G),
 * 0, 2^V - 1) half to even (0 for a zero step), r^ = min_G + q step_G, and w^_i = r^_i s_i (.)
 * c_{z_i} written to d_w_hat fp32[n][ldw] (ldw >= k, ldw % 4 == 0, 16-byte aligned). The radius,
 * offset, step and level are computed in fp64. d_rho fp32[n][k/8]; d_signs, d_dir_idx as in
 * sph_pack_weights; d_codebook fp32[2^D][8] (e.g. from sph_angular_codebook), not validated.
 * Optional outputs (NULL to skip): d_r_hat fp32[n][k/8] (needed by the backward), and together
 * d_radius_code uint8[n][k/8], d_group_min, d_group_step fp16 bits [n][k/128] -- the finalised
 * codes of App. A step 10. Asynchronous; results do not depend on the launch. */
sph_status sph_fake_quant_forward(const sph_format* fmt, int64_t n, int64_t k, const float* d_rho,
                                  const uint8_t* d_signs, const uint16_t* d_dir_idx, const float* d_codebook,
                                  float* d_w_hat, int64_t ldw, float* d_r_hat, uint8_t* d_radius_code,
                                  uint16_t* d_group_min, uint16_t* d_group_step, void* stream);

/* Device workspace of sph_fake_quant_backward for a 2^D-entry codebook (needs no zero-fill). */
sph_status sph_fake_quant_backward_workspace_bytes(int32_t dir_bits, size_t* bytes);

/* Gradients through sph_fake_quant_forward with the straight-through estimator (the rounding of
 * the radius is taken as the identity): given d_grad_w fp32[n][ldg] (dL/dW^; ldg >= k,
 * ldg % 4 == 0, 16-byte aligned), writes d_grad_rho fp32[n][k/8] with
 * dL/drho_i = sigmoid(rho_i) sum_j dL/dw^_ij s_ij c_{z_i,j}, and d_grad_codebook fp32[2^D][8]
 * with dL/dc_z = sum over vectors i of direction z of r^_i s_i (.) dL/dw^_i. d_r_hat is the
 * forward's r^; d_perm int32[n*k/8] and d_offsets int64[2^D + 1] are device copies of
 * sph_direction_groups for the same d_dir_idx (not validated). Sums run in a fixed order without
 * atomics, so repeated calls give bitwise identical results. d_ws: sph_fake_quant_backward_
 * workspace_bytes bytes, 16-byte aligned. Asynchronous. */
sph_status sph_fake_quant_backward(const sph_format* fmt, int64_t n, int64_t k, const float* d_rho,
                                   const uint8_t* d_signs, const uint16_t* d_dir_idx, const float* d_codebook,
                                   const float* d_r_hat, const float* d_grad_w, int64_t ldg, const int32_t* d_perm,
                                   const int64_t* d_offsets, float* d_grad_rho, float* d_grad_codebook, void* d_ws,
                                   size_t ws_bytes, void* stream);

/* Whether (dir_bits, radius_bits) is one of the built-in formats: 1 yes, 0 no. */
int sph_format_supported(const sph_format* fmt);

/* Static, human-readable name of a status code. */
const char* sph_status_str(sph_status s);

#ifdef __cplusplus
}
#endif

#endif /* SPH_H */
