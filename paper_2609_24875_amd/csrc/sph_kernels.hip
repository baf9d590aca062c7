// SPHQuant decode-and-multiply on gfx950 (MI355X): kernels and the C ABI of include/sph.h.
//
// The computation is the fused dequantise-and-multiply of Sec. 3.4 / App. D: every 8-D weight
// vector is rebuilt in registers as r^ * s (.) c_z (Eq. 4) with r^ = min_G + q * step_G (Eq. 7)
// and multiplied with fp16 activations, accumulating in fp32; nothing dequantised is written to
// memory. The mapping to the hardware is this library's own:
//  - device layout: 16-row tiles, one "record" per (tile, vector position) (sph_layout.h);
//  - vector-ALU path (batch 1): a lane owns one vector position of a tile and decodes its 16
//    rows (or, with two lanes per position, 8 of them) from 16-byte loads; signs are folded into two nibble-indexed lookup tables in LDS, so
//    the signed direction costs two 8-byte LDS reads and no sign arithmetic; products use
//    v_dot2_f32_f16 (exact fp16 products, fp32 sums); waves walk balanced ranges of
//    (tile, K-chunk) steps and split tiles are added in a fixed order, so results are bitwise
//    reproducible. Batch 2 runs the same way with two rows of products (except with the 2^13
//    codebook); batches up to 8 decode the same records, 4 lanes per vector position, into
//    4x4x4 MFMA blocks;
//  - matrix-core tile path (batch 9..16): each lane decodes one (row, vector) into exact fp16
//    A operands of v_mfma_f32_16x16x32_f16 (Eq. 7 factored over a group), activations form the
//    B operand;
//  - prefill (batch above 16, and 9..16 on large matrices): workgroups rebuild their tiles once
//    per K-chunk and multiply them with activations staged in LDS on the same 16x16x32 MFMA;
//  - 4-D and 16-D vectors: row-planar kernels, one wave per output row.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <type_traits>
#include <cstring>
#include <vector>

#include "sph_host.h"
#include "sph_layout.h"

typedef _Float16 f16;
typedef f16 f16x2 __attribute__((ext_vector_type(2)));
typedef f16 f16x4 __attribute__((ext_vector_type(4)));
typedef f16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct KArgs {
  const uint32_t* A;
  const uint32_t* B;
  const uint32_t* P;
  const uint16_t* C;  // codebook kind with 4 radius bits: bit 3 of q, one 16-bit word per record
  const uint4* T;
  const uint16_t* CB;  // the codebook as packed (read from memory by the 16-D kernel)
  uint32_t t_bytes;   // bytes of lookup tables staged into LDS
  const uint16_t* x;
  int64_t ldx;
  void* y;
  int64_t ldy;
  int y_f16;
  int n, nt, nv, ng, m;
  // vector-ALU work plan: ts = nt * nc steps in tile-major order, cut into contiguous wave ranges
  // of wl steps (the last one of a workgroup or of the launch possibly shorter, later waves
  // empty): across the whole launch (wg_tiles = 0), or inside each workgroup's wgs = wg_tiles * nc
  // steps of whole tiles
  int nc;             // steps (chunks of vector positions) per tile
  int nwg;            // workgroups
  int wg_tiles;       // tiles per workgroup, or 0 for ranges across workgroups
  int wl, wgs;        // steps per wave range and per workgroup (wg_tiles > 0)
  uint32_t wl_m, wgs_m;   // multipliers and shifts for division by wl and wgs (see udiv_by)
  int wl_k, wgs_k;
  int wpb;            // waves per workgroup
  int pmax;           // slot parts per tile
  int ts;
  uint64_t* ws_slot;  // [nt][pmax][M][16] tagged partial sums of split tiles, zero between calls
  uint32_t* ws_cnt;   // [nt] arrivals at each split tile, zero between calls
  // prefill path (batch > 32): K split into ks ranges; with ks > 1 each range writes fp32 partial
  // outputs [ks][m][nt * 16] to ws_part and a second kernel adds them in range order
  int ks;
  float* ws_part;
};

// ------------------------------------------------------------------------------------------
// Field extraction, shared by every kernel (so sph_unpack checks exactly what compute uses).
// ------------------------------------------------------------------------------------------

// Nibble kinds: the low/high table indices and the radius level of the row whose 16-bit (or,
// for W2, 14-bit) field sits in dword `d`. `odd` selects the second row of a dword; `qx` is the
// out-of-dword radius level (W2 odd rows) or the q byte word (NIB16Q8).
template <int KIND, int D>
__device__ __forceinline__ void decode_nib(uint32_t d, bool odd, uint32_t qx, uint32_t& lo,
                                           uint32_t& hi, uint32_t& q) {
  constexpr uint32_t IM = (1u << (D + 4)) - 1;
  if constexpr (KIND == SPH_KIND_W2) {
    constexpr int W = 8 + D;                   // field width
    constexpr uint32_t FM = (1u << W) - 1u;
    const uint32_t f = odd ? ((d >> W) & FM) : (d & FM);
    lo = f & IM;
    hi = f >> 4;
    q = odd ? qx : (d >> (2 * W));
  } else {
    const uint32_t f = odd ? (d >> 16) : (d & 0xFFFFu);
    lo = f & IM;
    hi = (f >> 4) & IM;
    if constexpr (KIND == SPH_KIND_NIB16) q = f >> (8 + D);
    else q = qx;
  }
}

// Codebook kind (D = 13): sign byte, direction index and level.
__device__ __forceinline__ void decode_cb13(uint32_t sdw, int sbyte, uint32_t zdw, bool odd,
                                            uint32_t& s, uint32_t& z, uint32_t& q) {
  s = (sdw >> (8 * sbyte)) & 0xFFu;
  const uint32_t f = odd ? (zdw >> 16) : (zdw & 0xFFFFu);
  z = f & 0x1FFFu;
  q = f >> 13;
}

// The signed direction s (.) c_z of one vector as 4 half2 words, looked up in LDS.
template <int KIND, int D>
__device__ __forceinline__ uint4 signed_dir_nib(const unsigned char* lds, uint32_t lo, uint32_t hi) {
  constexpr uint32_t THI = 16u << D;          // entries of T_lo
  const uint2 a = ((const uint2*)lds)[lo];
  const uint2 b = ((const uint2*)lds)[THI + hi];
  return make_uint4(a.x, a.y, b.x, b.y);
}

__device__ __forceinline__ uint4 signed_dir_cb13(const unsigned char* lds, uint32_t mask_off, uint32_t s,
                                                 uint32_t z) {
  const uint4 c = ((const uint4*)lds)[z];
  const uint2* mask = (const uint2*)(lds + mask_off);
  const uint2 ml = mask[s & 15u];
  const uint2 mh = mask[s >> 4];
  return make_uint4(c.x ^ ml.x, c.y ^ ml.y, c.z ^ mh.x, c.w ^ mh.y);
}

__device__ __forceinline__ float f16lo(uint32_t u) { return (float)__builtin_bit_cast(f16, (uint16_t)(u & 0xFFFFu)); }
__device__ __forceinline__ float f16hi(uint32_t u) { return (float)__builtin_bit_cast(f16, (uint16_t)(u >> 16)); }
__device__ __forceinline__ f16x2 as_h2(uint32_t u) { return __builtin_bit_cast(f16x2, u); }

// q * t for the 8 fp16 values of a signed direction t and a level q < 2^8, split exactly into two
// fp16 words, hi = fp16(q * t) and lo = q * t - hi. The product has at most 11 + 8 significant bits
// and is a multiple of t's unit in the last place, so the rounding residual is at most 2^7 such
// units and fits an fp16 significand exactly; the fused multiply-add returns it without rounding.
// |q * t| <= 255 * 2 because the packer admits codebook entries of at most 2, so nothing overflows.
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ void qt_split(uint4 t, uint32_t q, uint4& hi, uint4& lo) {
  const f16 qh = (f16)(float)q;
  const f16x2 qq = {qh, qh};
  const f16x2 h0 = as_h2(t.x) * qq, h1 = as_h2(t.y) * qq, h2 = as_h2(t.z) * qq, h3 = as_h2(t.w) * qq;
  const f16x2 l0 = __builtin_elementwise_fma(as_h2(t.x), qq, -h0);
  const f16x2 l1 = __builtin_elementwise_fma(as_h2(t.y), qq, -h1);
  const f16x2 l2 = __builtin_elementwise_fma(as_h2(t.z), qq, -h2);
  const f16x2 l3 = __builtin_elementwise_fma(as_h2(t.w), qq, -h3);
  hi = make_uint4(__builtin_bit_cast(uint32_t, h0), __builtin_bit_cast(uint32_t, h1), __builtin_bit_cast(uint32_t, h2),
                  __builtin_bit_cast(uint32_t, h3));
  lo = make_uint4(__builtin_bit_cast(uint32_t, l0), __builtin_bit_cast(uint32_t, l1), __builtin_bit_cast(uint32_t, l2),
                  __builtin_bit_cast(uint32_t, l3));
}

// Value of lane E of this lane's quad (lanes 4i..4i+3), by a DPP quad permutation.
template <int E>
__device__ __forceinline__ float quad_bcast(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), E * 0x55, 0xF, 0xF, false));
}

__device__ __forceinline__ float dot8(uint4 t, const uint32_t (&x)[4]) {
  float p = __builtin_amdgcn_fdot2(as_h2(t.x), as_h2(x[0]), 0.0f, false);
  p = __builtin_amdgcn_fdot2(as_h2(t.y), as_h2(x[1]), p, false);
  p = __builtin_amdgcn_fdot2(as_h2(t.z), as_h2(x[2]), p, false);
  return __builtin_amdgcn_fdot2(as_h2(t.w), as_h2(x[3]), p, false);
}

template <int N>
__device__ __forceinline__ void load_dw(uint32_t (&d)[N], const uint32_t* p) {
  if constexpr (N == 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint4 u = *(const uint4*)(p + 4 * i);
      d[4 * i] = u.x; d[4 * i + 1] = u.y; d[4 * i + 2] = u.z; d[4 * i + 3] = u.w;
    }
  } else if constexpr (N == 8) {
    const uint4 u = *(const uint4*)p, w = *(const uint4*)(p + 4);
    d[0] = u.x; d[1] = u.y; d[2] = u.z; d[3] = u.w; d[4] = w.x; d[5] = w.y; d[6] = w.z; d[7] = w.w;
  } else if constexpr (N == 4) {
    const uint4 u = *(const uint4*)p;
    d[0] = u.x; d[1] = u.y; d[2] = u.z; d[3] = u.w;
  } else if constexpr (N == 2) {
    const uint2 u = *(const uint2*)p;
    d[0] = u.x; d[1] = u.y;
  } else if constexpr (N == 1) {
    d[0] = *p;
  }
}

__device__ __forceinline__ void store_y(const KArgs& a, int b, int row, float v) {
  if (a.y_f16) ((f16*)a.y)[(int64_t)b * a.ldy + row] = (f16)v;
  else ((float*)a.y)[(int64_t)b * a.ldy + row] = v;
}

// ------------------------------------------------------------------------------------------
// Vector-ALU kernel: batch M (1, 2, 4 or 8), RPL rows of a record per lane.
//
// The work is ts = nt * nc steps: step (t, c) is chunk c (64/H consecutive vector positions, one
// per lane group) of tile t (16 rows). The steps, in tile-major order, are cut into contiguous
// ranges of equal length (to one step), one per wave, in the manner of stream-K. A tile that
// lies wholly inside a range is stored straight to y. A tile cut by range boundaries has parts
// in consecutive waves: each later part is handed over through tagged workspace slots, and the
// wave holding chunk 0 (whose range ends inside the tile) adds the parts in chunk order and
// stores y. Later parts sit at the start of their waves' ranges, so they are normally written
// long before that wave reaches its end; the order of the sum is fixed, so results do not depend
// on scheduling.
// ------------------------------------------------------------------------------------------
// Waves per workgroup of the vector-ALU kernel, and workgroups resident per CU.
constexpr int VALU_WPB = 16;
constexpr int VALU_WG_PER_CU = 1;
constexpr int VALU_THREADS = 64 * VALU_WPB;
// Rows per batch of table lookups, and whether lookup batches are pinned in pipelined order by
// scheduling barriers: in the 4x4x4-block mode (batch 3..8) the pinned order is 1-2% faster; the
// vector-ALU mode (batch 1, 2) is left to the compiler's schedule, which took the 32B-class
// batch-1 step from 3.09-3.11 to 3.04-3.05 ms (two runs each, one box).
constexpr int VALU_RB = 4;
template <bool MX>
constexpr bool VALU_PIPE_BARRIERS = MX;

template <int KIND>
constexpr bool IS_CB = KIND == SPH_KIND_CB13 || KIND == SPH_KIND_CB13Q4;

template <int KIND, int D>
struct Tables {
  static constexpr uint32_t bytes = IS_CB<KIND> ? ((16u << D) + 128u) : (256u << D);
};

// The tile variant (batch 9..16) passes each step's activations through a per-wave LDS buffer
// of 16 batch rows x 16 vector positions, rows padded to XT_ROW bytes so that the operand-order
// reads hit distinct banks: its global loads then read 4 rows x 256 contiguous bytes each instead
// of 16 rows x 64 bytes (operand order), half the cache lines per load, which is what bounds that
// variant. Done for the kinds with at most 7 direction bits: the 2^13-codebook kinds have no LDS
// left beside their table, and the 8-bit-direction kinds would exceed 128 registers with it;
// those read x in operand order.
constexpr int XT_ROW = 16 * 16 + 16;
constexpr int XT_WAVE = 16 * XT_ROW;   // bytes per wave
__host__ __device__ constexpr bool xt_staged(int kind, int mode) {
  return mode == 2 && (kind == SPH_KIND_W2 || kind == SPH_KIND_NIB16);
}

// Whether the split-tile slots and counters of one workgroup's waves fit in LDS next to the lookup
// table and the parameter (modes 0, 1) or activation (mode 2) staging. Host and device.
__host__ __device__ constexpr bool lds_handover_fits(int kind, int D, int M, int mode) {
  return ((kind == SPH_KIND_CB13 || kind == SPH_KIND_CB13Q4) ? ((16u << D) + 128u) : (256u << D)) +
             (16u * M * 16u * 4u + 17u * 4u) +
             (mode == 2 ? (xt_staged(kind, mode) ? 16u * (uint32_t)XT_WAVE : 0u) : 16u * 256u) <=
         160u * 1024u;
}

// MX selects the matrix-core variant (batch 2..16): the lane's rows are rebuilt as in the vector
// variant, scaled to fp16 and multiplied by 4x4x4 MFMA blocks, one block per vector position.
template <int KIND, int M, int RPL, bool MX = false>
struct Rec {
  static constexpr int ADW = IS_CB<KIND> ? RPL / 4 : RPL / 2;
  static constexpr int BDW = (KIND == SPH_KIND_NIB16Q8) ? RPL / 4 : IS_CB<KIND> ? RPL / 2 : 1;
  static constexpr int NX = MX ? M / 4 : M;
  uint32_t ra[ADW];
  uint32_t rb[BDW];
  uint32_t rc;         // stream C word of the record (codebook kind with 4 radius bits)
  uint32_t pw;         // one group-parameter word of the chunk, staged through LDS at compute time
  uint32_t xv[NX][4];  // vector variant: x[b] at this lane's position for every batch row b;
                       // MX: x[4g + lane % 4] at this lane's position for each group g of 4 rows
  bool pok;            // pw belongs to a group inside the row; else the group's radii are taken as 0
};

// Loads of one step. Branch-free, and no loaded value is ever selected or copied before use, so
// that the compiler can count outstanding loads across the software pipeline. Vector positions
// past the end of the row (whole groups, since k is a multiple of 128) read a valid record and
// contribute nothing because their group parameters are taken as zero. The chunk's group
// parameters (VPC/16 groups x 16 rows = VPC words, contiguous) are spread one word per lane.
template <int KIND, int M, int RPL, bool MX = false>
__device__ __forceinline__ void load_rec(Rec<KIND, M, RPL, MX>& R, const KArgs& a, int t, int c, int h, int vloc,
                                         int lane) {
  constexpr int H = 16 / RPL, VPC = 64 / H;
  constexpr int ADW_REC = IS_CB<KIND> ? 4 : 8;
  constexpr int BDW_REC = (KIND == SPH_KIND_W2 || KIND == SPH_KIND_NIB16Q2) ? 1 : (KIND == SPH_KIND_NIB16Q8) ? 4 : 8;
  constexpr int ADW = Rec<KIND, M, RPL, MX>::ADW, BDW = Rec<KIND, M, RPL, MX>::BDW;
  const int v = min(c * VPC + vloc, a.nv - 1);
  const int64_t rec = (int64_t)t * a.nv + v;
  load_dw<ADW>(R.ra, a.A + rec * ADW_REC + h * ADW);
  if constexpr (KIND == SPH_KIND_W2 || KIND == SPH_KIND_NIB16Q2) R.rb[0] = a.B[rec];
  else if constexpr (KIND != SPH_KIND_NIB16) load_dw<BDW>(R.rb, a.B + rec * BDW_REC + h * BDW);
  if constexpr (KIND == SPH_KIND_CB13Q4) R.rc = a.C[rec];
  else R.rc = 0;
  // parameter word `lane` of the chunk: group c*VPC/16 + lane/16, row lane%16 (clamped to the row)
  const int pg0 = c * (VPC / 16) + (lane & (VPC - 1)) / 16;
  const int pg = min(pg0, a.ng - 1);
  R.pw = a.P[((int64_t)t * a.ng + pg) * 16 + (lane & 15)];
  R.pok = pg0 < a.ng;
  if constexpr (MX) {
    // batch rows past m feed MFMA columns that are never stored; they read row m - 1
#pragma unroll
    for (int g = 0; g < Rec<KIND, M, RPL, MX>::NX; ++g) {
      const int bb = min(4 * g + (lane & 3), a.m - 1);
      load_dw<4>(R.xv[g], (const uint32_t*)(a.x + (int64_t)bb * a.ldx + 8 * (int64_t)v));
    }
  } else {
#pragma unroll
    for (int b = 0; b < M; ++b) {
      const int bb = (M == 1 || b < a.m) ? b : 0;
      load_dw<4>(R.xv[b], (const uint32_t*)(a.x + (int64_t)bb * a.ldx + 8 * (int64_t)v));
    }
  }
}

// Table lookups of the rows [r0, r0 + RB) of a record: field extraction and the LDS reads.
template <int KIND, int D, int M, int RPL, int RB, bool MX = false>
__device__ __forceinline__ void lookup_rows(const Rec<KIND, M, RPL, MX>& R, int r0, uint32_t qodd, const unsigned char* lds,
                                            uint32_t mask_off, uint4 (&tt)[RB], float (&qf)[RB]) {
#pragma unroll
  for (int i = 0; i < RB; ++i) {
    const int r = r0 + i;
    uint32_t q;
    if constexpr (IS_CB<KIND>) {
      uint32_t s, z;
      decode_cb13(R.ra[r / 4], r % 4, R.rb[r / 2], r & 1, s, z, q);
      if constexpr (KIND == SPH_KIND_CB13Q4) q |= ((qodd >> r) & 1u) << 3;
      tt[i] = signed_dir_cb13(lds, mask_off, s, z);
    } else {
      uint32_t lo, hi, qx = 0;
      if constexpr (KIND == SPH_KIND_W2) qx = (qodd >> (4 * (r / 2))) & 15u;
      if constexpr (KIND == SPH_KIND_NIB16Q2) qx = (qodd >> (2 * r)) & 3u;
      if constexpr (KIND == SPH_KIND_NIB16Q8) qx = (R.rb[r / 4] >> (8 * (r % 4))) & 0xFFu;
      decode_nib<KIND, D>(R.ra[r / 2], r & 1, qx, lo, hi, q);
      tt[i] = signed_dir_nib<KIND, D>(lds, lo, hi);
    }
    qf[i] = (float)q;
  }
}

// The rows of a record in batches of RB, software-pipelined: the lookups of batch j+1 are issued
// before the arithmetic of batch j, and scheduling barriers keep the compiler from interleaving
// them back (left alone, it keeps only a few LDS reads in flight per wave, far fewer than the
// LDS latency under bank conflicts needs).
template <int KIND, int D, int M, int RPL, bool MX = false>
__device__ __forceinline__ void compute_rec(const Rec<KIND, M, RPL, MX>& R, float (&acc)[M][RPL],
                                            const unsigned char* lds, uint32_t mask_off, uint32_t* pstage,
                                            int lane, int h, int vloc) {
  constexpr int RB = RPL < VALU_RB ? RPL : VALU_RB;
  constexpr int NB = RPL / RB;
  // group parameters: stage the chunk's words in this wave's LDS slot, read back this lane's rows
  pstage[lane] = R.pok ? R.pw : 0u;
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  uint32_t pp[RPL];
  const uint32_t* src = pstage + (vloc >> 4) * 16 + h * RPL;
#pragma unroll
  for (int i = 0; i < RPL; i += 4) {
    const uint4 u = *(const uint4*)(src + i);
    pp[i] = u.x; pp[i + 1] = u.y; pp[i + 2] = u.z; pp[i + 3] = u.w;
  }
  // radius bits kept outside the lane's A words, shifted to its first row
  uint32_t qodd = 0;
  if constexpr (KIND == SPH_KIND_W2) qodd = R.rb[0] >> (4 * (h * RPL / 2));
  if constexpr (KIND == SPH_KIND_NIB16Q2) qodd = R.rb[0] >> (2 * h * RPL);
  if constexpr (KIND == SPH_KIND_CB13Q4) qodd = R.rc >> (h * RPL);
  uint4 tt[2][RB];
  float qf[2][RB];
  lookup_rows<KIND, D, M, RPL, RB, MX>(R, 0, qodd, lds, mask_off, tt[0], qf[0]);
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    if (j + 1 < NB) lookup_rows<KIND, D, M, RPL, RB, MX>(R, (j + 1) * RB, qodd, lds, mask_off, tt[(j + 1) & 1], qf[(j + 1) & 1]);
    if constexpr (VALU_PIPE_BARRIERS<MX>) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int r = j * RB + i;
      const float rh = fmaf(qf[j & 1][i], f16hi(pp[r]), f16lo(pp[r]));
      if constexpr (MX) {
        // Exact products, as in the vector-ALU path: block v of the MFMA is this lane's vector
        // position, its row lane % 4 the quad lane's row 4 * (lane % 4) + r (rebuilt there as the
        // signed direction t, exact in fp16) and its column lane % 4 batch row 4g + lane % 4. So
        // lane (v, j) receives D[e] = <t, x> of row 4e + r and batch row 4g + j: fp16 products
        // summed in fp32 over the vector's 8 elements. Each is scaled in fp32 by that row's radius,
        // which lane e of the quad computed, and added to acc[4g + r][e].
        const uint4 t = tt[j & 1][i];
        const float re[4] = {quad_bcast<0>(rh), quad_bcast<1>(rh), quad_bcast<2>(rh), quad_bcast<3>(rh)};
        const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int g = 0; g < M / 4; ++g) {
          f32x4 d = __builtin_amdgcn_mfma_f32_4x4x4f16(__builtin_bit_cast(f16x4, make_uint2(t.x, t.y)),
                                                        __builtin_bit_cast(f16x4, make_uint2(R.xv[g][0], R.xv[g][1])), z, 0,
                                                        0, 0);
          d = __builtin_amdgcn_mfma_f32_4x4x4f16(__builtin_bit_cast(f16x4, make_uint2(t.z, t.w)),
                                                  __builtin_bit_cast(f16x4, make_uint2(R.xv[g][2], R.xv[g][3])), d, 0, 0, 0);
#pragma unroll
          for (int e = 0; e < 4; ++e) acc[4 * g + r][e] = fmaf(re[e], d[e], acc[4 * g + r][e]);
        }
      } else {
#pragma unroll
        for (int b = 0; b < M; ++b) acc[b][r] = fmaf(rh, dot8(tt[j & 1][i], R.xv[b]), acc[b][r]);
      }
    }
    if constexpr (VALU_PIPE_BARRIERS<MX>) __builtin_amdgcn_sched_barrier(0);
  }
}

// Tile variant (batch 9..16): lane (r, j) = (lane % 16, lane / 16) rebuilds row r of the vector
// positions 4i + j (i = 0..3) of a 16-position chunk, which is exactly the A operand of
// v_mfma_f32_16x16x32_f16 (16 rows x 4 positions); the B operand is x for batch rows
// 16nb + lane % 16 at the same positions. A chunk is one radius group, so Eq. 7 factors over it:
// sum_v r^_v <t_v, x_v> = offset * sum_v <t_v, x_v> + step * sum_v q_v <t_v, x_v>. The MFMA forms
// both sums with exact fp16 operands -- the signed directions t, and q * t split exactly into two
// fp16 words -- so every product is exact and only fp32 sums round; each lane then ends a step
// with both sums for (batch 16nb + lane % 16, rows 4 * (lane / 16) + e) and folds them into its
// accumulators with those rows' offset and step. No lane reduction is needed. One record dword
// (and one aux dword) per position and lane: 128 contiguous bytes per load over the wave.
template <int KIND, int NB>
struct RecT {
  uint32_t ra[4];
  uint32_t rb[4];
  uint32_t rc[4];         // stream C words (codebook kind with 4 radius bits)
  uint4 pw;               // (offset, step) of rows 4 * (lane / 16) + e of the chunk's group
  uint32_t xv[NB * 4][4]; // x[16nb + lane % 16] at position 4i + j, index nb * 4 + i; staged
                          // through LDS (NB = 1): x[4i + lane / 16] at position lane % 16
  bool pok;
};

template <int KIND, int NB>
__device__ __forceinline__ void load_rec_t(RecT<KIND, NB>& R, const KArgs& a, int t, int c, int lane) {
  constexpr bool B1 = KIND == SPH_KIND_W2 || KIND == SPH_KIND_NIB16Q2;   // one B dword per record
  constexpr int ADW_REC = IS_CB<KIND> ? 4 : 8;
  constexpr int BDW_REC = B1 ? 1 : (KIND == SPH_KIND_NIB16Q8) ? 4 : 8;
  const int r = lane & 15, j = lane >> 4;
  // the dword holding row r in each stream
  const int adw = IS_CB<KIND> ? r / 4 : r / 2;
  const int bdw = B1 ? 0 : (KIND == SPH_KIND_NIB16Q8) ? r / 4 : r / 2;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int v = min(c * 16 + 4 * i + j, a.nv - 1);
    const int64_t rec = (int64_t)t * a.nv + v;
    R.ra[i] = a.A[rec * ADW_REC + adw];
    if constexpr (KIND != SPH_KIND_NIB16) R.rb[i] = a.B[rec * BDW_REC + bdw];
    else R.rb[i] = 0;
    if constexpr (KIND == SPH_KIND_CB13Q4) R.rc[i] = a.C[rec];
    else R.rc[i] = 0;
  }
  // one 128-weight group per chunk: (offset, step) of the rows this lane's sums belong to
  const int pg = min(c, a.ng - 1);
  R.pw = *(const uint4*)(a.P + ((int64_t)t * a.ng + pg) * 16 + 4 * j);
  R.pok = c < a.ng;
  if constexpr (xt_staged(KIND, 2)) {
    static_assert(NB == 1, "the staged activations cover 16 batch rows");
    const int v = min(c * 16 + r, a.nv - 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int bb = min(4 * i + j, a.m - 1);   // columns past the batch are never stored
      load_dw<4>(R.xv[i], (const uint32_t*)(a.x + (int64_t)bb * a.ldx + 8 * (int64_t)v));
    }
  } else {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int bb = min(16 * nb + r, a.m - 1);   // columns past the batch are never stored
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = min(c * 16 + 4 * i + j, a.nv - 1);
        load_dw<4>(R.xv[nb * 4 + i], (const uint32_t*)(a.x + (int64_t)bb * a.ldx + 8 * (int64_t)v));
      }
    }
  }
}

template <int KIND, int D, int NB>
__device__ __forceinline__ void compute_rec_t(const RecT<KIND, NB>& R, float (&acc)[NB][4], const unsigned char* lds,
                                              uint32_t mask_off, unsigned char* xs, int lane) {
  const int r = lane & 15;
  if constexpr (xt_staged(KIND, 2)) {
    // row-order words into the wave's buffer; read back in operand order below (the LDS performs
    // a wave's operations in issue order, so the reads see these writes, and the next step's
    // writes come after this step's reads)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      *(uint4*)(xs + (4 * i + (lane >> 4)) * XT_ROW + r * 16) = make_uint4(R.xv[i][0], R.xv[i][1], R.xv[i][2], R.xv[i][3]);
  }
  uint4 tt[4];
  uint32_t q[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if constexpr (IS_CB<KIND>) {
      uint32_t sg, z;
      decode_cb13(R.ra[i], r % 4, R.rb[i], r & 1, sg, z, q[i]);
      if constexpr (KIND == SPH_KIND_CB13Q4) q[i] |= ((R.rc[i] >> r) & 1u) << 3;
      tt[i] = signed_dir_cb13(lds, mask_off, sg, z);
    } else {
      uint32_t l, hh, qx = 0;
      if constexpr (KIND == SPH_KIND_W2) qx = (R.rb[i] >> (4 * (r / 2))) & 15u;
      if constexpr (KIND == SPH_KIND_NIB16Q2) qx = (R.rb[i] >> (2 * r)) & 3u;
      if constexpr (KIND == SPH_KIND_NIB16Q8) qx = (R.rb[i] >> (8 * (r % 4))) & 0xFFu;
      decode_nib<KIND, D>(R.ra[i], r & 1, qx, l, hh, q[i]);
      tt[i] = signed_dir_nib<KIND, D>(lds, l, hh);
    }
  }
  // the staged activations are read only now (hoisted above the decode they would hold 16 more
  // registers through it, past the 128 of four waves per SIMD)
  if constexpr (xt_staged(KIND, 2)) __builtin_amdgcn_sched_barrier(0);
  f32x4 s0[NB], s1[NB];   // sum <t, x> and sum q <t, x> over the chunk
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) s0[nb] = s1[nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint4 hi, lo;
    qt_split(tt[i], q[i], hi, lo);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const uint32_t* xq = R.xv[nb * 4 + i];
      const f16x8 xb = xt_staged(KIND, 2)
                           ? *(const f16x8*)(xs + r * XT_ROW + (4 * i + (lane >> 4)) * 16)
                           : __builtin_bit_cast(f16x8, make_uint4(xq[0], xq[1], xq[2], xq[3]));
      s0[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, tt[i]), xb, s0[nb], 0, 0, 0);
      s1[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, hi), xb, s1[nb], 0, 0, 0);
      s1[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, lo), xb, s1[nb], 0, 0, 0);
    }
  }
  const uint4 pw = R.pok ? R.pw : make_uint4(0u, 0u, 0u, 0u);
  const uint32_t pe[4] = {pw.x, pw.y, pw.z, pw.w};
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[nb][e] = fmaf(f16hi(pe[e]), s1[nb][e], fmaf(f16lo(pe[e]), s0[nb][e], acc[nb][e]));
}

// Step dispatch over the three variants (MODE 0: vector ALU, 1: 4x4x4 blocks, 2: 16x16x32 tiles).
template <int KIND, int D, int M, int RPL, int MODE>
struct Step {
  static constexpr int AR = MODE == 2 ? M / 16 : M;       // accumulator rows per lane
  using R = typename std::conditional<MODE == 2, RecT<KIND, M / 16>, Rec<KIND, M, RPL, MODE == 1>>::type;
  static __device__ __forceinline__ void load(R& rec, const KArgs& a, int t, int c, int h, int vloc, int lane) {
    if constexpr (MODE == 2) load_rec_t<KIND, M / 16>(rec, a, t, c, lane);
    else load_rec<KIND, M, RPL, MODE == 1>(rec, a, t, c, h, vloc, lane);
  }
  static __device__ __forceinline__ void compute(const R& rec, float (&acc)[AR][RPL], const unsigned char* lds,
                                                 uint32_t mask_off, uint32_t* pstage, int lane, int h, int vloc) {
    if constexpr (MODE == 2) compute_rec_t<KIND, D, M / 16>(rec, acc, lds, mask_off, (unsigned char*)pstage, lane);
    else compute_rec<KIND, D, M, RPL, MODE == 1>(rec, acc, lds, mask_off, pstage, lane, h, vloc);
  }
};

// Exchange-and-add across lanes l and l^DIST (DIST = 32 or 16): lanes with bit DIST clear end
// with lo_keep[l] + lo_keep[l^DIST], the others with hi_keep[l] + hi_keep[l^DIST]. This is one
// gfx950 half-swap (v_permlane32_swap / v_permlane16_swap exchange the upper half of the first
// register with the lower half of the second, at 32- or 16-lane granularity) and an add, all on
// the vector ALU. The swap is written in assembly because this compiler version returns the
// first register twice from the builtin's result pair. The compiler cannot see hazards through
// the assembly, so it carries its own wait states: the leading s_nop 1 (two wait states) is what
// the compiler's hazard recognizer puts between a vector write of an operand and this
// instruction when it emits the builtin itself; it puts none after it, and the trailing s_nop is
// a margin of two cycles.
template <int DIST>
__device__ __forceinline__ float xchg_add(float lo_keep, float hi_keep, int lane) {
  (void)lane;
  float a = lo_keep, b = hi_keep;
  if constexpr (DIST == 32) asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
  else asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
  return a + b;
}

template <int CTRL>
__device__ __forceinline__ float dpp_add(float v) {
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

// Sum an item's accumulators over the lanes sharing h: a scatter over lane bits 5 and 4 with
// lane exchanges, then all-reductions inside 16-lane rows with DPP rotations. Afterwards every
// lane holds NVAL/4 totals, value i being flattened index i + (NVAL/2)*bit5 + (NVAL/4)*bit4.
template <int NVAL, int H>
__device__ __forceinline__ void wave_reduce(float (&v)[NVAL], int lane) {
  constexpr int N2 = NVAL / 2, N4 = NVAL / 4;
#pragma unroll
  for (int i = 0; i < N2; ++i) v[i] = xchg_add<32>(v[i], v[i + N2], lane);
#pragma unroll
  for (int i = 0; i < N4; ++i) v[i] = xchg_add<16>(v[i], v[i + N4], lane);
#pragma unroll
  for (int i = 0; i < N4; ++i) {
    float x = dpp_add<0x128>(v[i]);                      // row_ror:8
    x = dpp_add<0x124>(x);                                // row_ror:4
    if constexpr (H <= 2) x = dpp_add<0x122>(x);          // row_ror:2
    if constexpr (H <= 1) x = dpp_add<0x121>(x);          // row_ror:1
    v[i] = x;
  }
}

// floor(x / d) for 0 <= x < 2^31 and a launch-constant d, as (x * m) >> k with the host's
// m = ceil(2^k / d), k = 31 + ceil(log2 d): m fits in 32 bits and the product's excess over x / d
// stays below 1 / d, so the floor is exact. A multiply and a shift instead of an integer division
// sequence, which would cost the prologue a microsecond over the 16 waves of a CU.
__device__ __forceinline__ int udiv_by(int x, uint32_t m, int k) {
  return (int)(((uint64_t)(uint32_t)x * m) >> k);
}

// The wave (id = workgroup * VALU_WPB + wave in workgroup) whose range holds step s.
__device__ __forceinline__ int wave_of_step(const KArgs& a, int s) {
  if (a.wg_tiles == 0) return __builtin_amdgcn_readfirstlane(udiv_by(s, a.wl_m, a.wl_k));
  const int b = udiv_by(s, a.wgs_m, a.wgs_k);
  return __builtin_amdgcn_readfirstlane(b * VALU_WPB + udiv_by(s - b * a.wgs, a.wl_m, a.wl_k));
}

// ------------------------------------------------------------------------------------------
// Split tiles. A tile whose steps fall into the ranges of several waves has one part per wave: part
// 0 (holding chunk 0) ends its wave's range, parts 1 .. np-1 start the ranges of the following
// waves. The parts are added in two levels, and no wave ever waits for another workgroup:
//
// 1. Inside a workgroup the tile's parts meet in LDS. Every part but the first one there (the
//    local leader) puts its lane-reduced sums in its wave's slot, counts its arrival on a counter
//    of the tile and moves on at once. The leader -- part 0, or the entering tile's part in the
//    workgroup's first wave, in either case the last part its wave computes -- waits for the
//    other local parts, which run on waves of its own workgroup and so are resident and wait for
//    nothing themselves, and adds them to its own sums in a fixed order.
// 2. A tile inside one workgroup is then stored. A tile over two workgroups meets in one 64-bit
//    workspace word per value: each workgroup swaps its sum, tagged valid in the high half, into
//    the word with a device-coherent atomic exchange. The lane that gets the other workgroup's sum
//    back adds the two (a sum of two terms, the same whichever comes first), stores y and zeroes
//    the word; the other lane has nothing left to do. A tile over three or more workgroups (only
//    when a wave range is much shorter than a tile) meets in per-workgroup slots and a counter:
//    the slots are written before a release fence and the count, and the workgroup that counts
//    last, after an acquire fence, adds the workgroup sums in workgroup order, stores y and zeroes
//    the slots and the counter.
//
// Each level adds in an order fixed by the plan, whichever part or workgroup arrives last, so
// results are bitwise reproducible, and the workspace is zero again after every call. Where the
// LDS has no room for the slots (the tile variant with the largest tables), every part goes to
// level 2 as a group of its own.
// ------------------------------------------------------------------------------------------
__device__ __forceinline__ uint64_t slot_word(float v) {
  return (uint64_t)__builtin_bit_cast(uint32_t, v) | (1ull << 32);
}

// LDS meeting place of the split tiles inside a workgroup: per wave a slot for its first part (the
// only part a wave can hand over to a leader: a part 0 leads its tile's local parts), and the
// arrival counter of the tile whose part 0 wave w holds (cnt[w]) and of the tile that enters from
// the previous workgroup (cnt[VALU_WPB]). Each slot and counter serves one tile per launch.
template <int M>
struct WgHo {
  float slot[VALU_WPB][M * 16];
  uint32_t cnt[VALU_WPB + 1];
};

// Slot index (batch row * 16 + tile row) of value i of this lane after the wave reduction: vector
// variant, value b * RPL + r is batch row b, tile row h * RPL + r; 4x4x4 blocks, value 16g + 4r + e
// is batch row 4g + h, tile row 4e + r (see compute_rec); tiles, value 4nb + e is batch row
// 16nb + lane % 16, tile row 4 * (lane / 16) + e (see compute_rec_t).
template <int M, int RPL, int MODE>
struct PartIdx {
  static constexpr int H = 16 / RPL;
  static constexpr int AR = MODE == 2 ? M / 16 : M;
  static constexpr int NVAL = AR * RPL, N4 = MODE == 2 ? NVAL : NVAL / 4;
  int idx[N4];
  bool writer;   // one writer lane per h in each 16-lane row; the tile variant's sums are per lane
  __device__ __forceinline__ explicit PartIdx(int lane) {
    const int h = lane % H;
    writer = MODE == 2 || (lane & 15) < H;
    const int base = MODE == 2 ? 0 : ((lane >> 5) & 1) * (NVAL / 2) + ((lane >> 4) & 1) * N4;
#pragma unroll
    for (int i = 0; i < N4; ++i) {
      const int f = base + i;
      if constexpr (MODE == 2) idx[i] = (16 * (f / 4) + (lane & 15)) * 16 + 4 * (lane >> 4) + f % 4;
      else if constexpr (MODE == 1) idx[i] = ((f / 16) * 4 + h) * 16 + 4 * (f % 4) + (f / 4) % 4;
      else idx[i] = (f / RPL) * 16 + h * RPL + f % RPL;
    }
  }
};

template <int M, int RPL, int MODE>
__device__ __forceinline__ void store_part(const KArgs& a, int t, const PartIdx<M, RPL, MODE>& I,
                                           const float (&v)[PartIdx<M, RPL, MODE>::N4], bool ok) {
  if (!I.writer) return;
#pragma unroll
  for (int i = 0; i < PartIdx<M, RPL, MODE>::N4; ++i) {
    const int b = I.idx[i] / 16, grow = t * 16 + I.idx[i] % 16;
    if (b < a.m && grow < a.n) store_y(a, b, grow, ok ? v[i] : __builtin_nanf(""));
  }
}


// Where a tile's parts lie, seen from wave g: waves gr .. gl hold them (np parts); this
// workgroup's are waves lw0 .. lw0+nl-1, counted on LDS counter ci; the tile spans ngrp groups
// (workgroups, or single parts without LDS meeting), this wave's being group gi. A wave can only
// hold a part of a split tile in the first and the last tile of its range, and it finds gr and gl
// for both at the start, while its first loads are in flight (they take integer divisions that
// would otherwise sit at the end of its work).
struct SplitGeo {
  int gr, np, p, lw0, nl, ci, ngrp, gi;
};

template <bool LDS_HO>
__device__ __forceinline__ SplitGeo split_geo(int gr, int gl, int g) {
  SplitGeo s;
  s.gr = gr;
  s.np = gl - s.gr + 1;
  s.p = g - s.gr;
  if constexpr (LDS_HO) {
    const int b0 = (g / VALU_WPB) * VALU_WPB;
    s.lw0 = max(s.gr, b0);
    s.nl = min(gl, b0 + VALU_WPB - 1) - s.lw0 + 1;
    s.ci = s.gr >= b0 ? s.gr - b0 : VALU_WPB;
    s.ngrp = gl / VALU_WPB - s.gr / VALU_WPB + 1;
    s.gi = g / VALU_WPB - s.gr / VALU_WPB;
  } else {
    s.lw0 = g;
    s.nl = 1;
    s.ci = 0;
    s.ngrp = s.np;
    s.gi = s.p;
  }
  return s;
}

// Level 2: the group sum `v` of tile t (see above). `xpre`: this lane's words of a tile over two
// workgroups as read before this wave's last step (zero if not read); a word that already holds
// the other workgroup's sum is used as it stands, without an exchange (that workgroup has
// finished with it).
template <int M, int RPL, int MODE>
__device__ __forceinline__ void group_done(const KArgs& a, int t, const SplitGeo& s,
                                           const float (&v)[PartIdx<M, RPL, MODE>::N4],
                                           const uint64_t (&xpre)[PartIdx<M, RPL, MODE>::N4], int lane) {
  using I = PartIdx<M, RPL, MODE>;
  constexpr int NIDX = M * 16;
  const I ix(lane);
  if (s.ngrp == 1) {
    store_part<M, RPL, MODE>(a, t, ix, v, true);
    return;
  }
  uint64_t* slots = a.ws_slot + (int64_t)t * a.pmax * NIDX;
  if (s.ngrp == 2) {
    if (!ix.writer) return;
    uint64_t o[I::N4];   // all exchanges in flight together
#pragma unroll
    for (int i = 0; i < I::N4; ++i)
      o[i] = (xpre[i] >> 32)
                 ? xpre[i]
                 : __hip_atomic_exchange(slots + ix.idx[i], slot_word(v[i]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
    for (int i = 0; i < I::N4; ++i)
      if (o[i] >> 32) {
        const int b = ix.idx[i] / 16, grow = t * 16 + ix.idx[i] % 16;
        if (b < a.m && grow < a.n) store_y(a, b, grow, __builtin_bit_cast(float, (uint32_t)o[i]) + v[i]);
        __hip_atomic_store(slots + ix.idx[i], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    return;
  }
  if (ix.writer)
#pragma unroll
    for (int i = 0; i < I::N4; ++i)
      __hip_atomic_store(slots + s.gi * NIDX + ix.idx[i], slot_word(v[i]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
  uint32_t old = 0;
  if (lane == 0) old = __hip_atomic_fetch_add(a.ws_cnt + t, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (__builtin_amdgcn_readfirstlane(old) + 1 != (uint32_t)s.ngrp) return;
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  float tot[I::N4];
#pragma unroll
  for (int i = 0; i < I::N4; ++i) tot[i] = 0.0f;
  if (ix.writer) {
    for (int q = 0; q < s.ngrp; ++q)
#pragma unroll
      for (int i = 0; i < I::N4; ++i) {
        const float x = q == s.gi ? v[i]
                                  : __builtin_bit_cast(float, (uint32_t)__hip_atomic_load(
                                                                  slots + q * NIDX + ix.idx[i], __ATOMIC_RELAXED,
                                                                  __HIP_MEMORY_SCOPE_AGENT));
        tot[i] = q == 0 ? x : tot[i] + x;
      }
    for (int q = 0; q < s.ngrp; ++q)
#pragma unroll
      for (int i = 0; i < I::N4; ++i)
        __hip_atomic_store(slots + q * NIDX + ix.idx[i], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  store_part<M, RPL, MODE>(a, t, ix, tot, true);
  if (lane == 0) __hip_atomic_store(a.ws_cnt + t, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The other local parts' slots (local parts 1 .. nl-1), spread over the lanes: lane l reads slot
// index l % NIDX (+ 64 k) of local parts 1 + j0 + l / NIDX + PPI * jj (jj < JB), so that one round
// trip covers up to 16 parts (4 for the 16-row batch) however many values a part has.
template <int M>
struct LocalRead {
  static constexpr int NIDX = M * 16;
  static constexpr int PPI = NIDX >= 64 ? 1 : 64 / NIDX;   // parts per read instruction
  static constexpr int IPP = NIDX <= 64 ? 1 : NIDX / 64;   // read instructions per part
  static constexpr int JB = (16 / IPP < 16 / PPI) ? 16 / IPP : 16 / PPI;
  static constexpr int LDIV = NIDX >= 64 ? 64 : NIDX;
  float v[JB][IPP];

  // local part read into v[jj] by this lane
  __device__ __forceinline__ static int part(int j0, int jj, int lane) { return 1 + j0 + lane / LDIV + PPI * jj; }

  __device__ __forceinline__ void read(const WgHo<M>* ho, const SplitGeo& s, int j0, int lane) {
#pragma unroll
    for (int jj = 0; jj < JB; ++jj) {
      const int w = s.lw0 + min(part(j0, jj, lane), s.nl - 1);
#pragma unroll
      for (int k = 0; k < IPP; ++k) v[jj][k] = ho->slot[w % VALU_WPB][lane % NIDX + 64 * k];
    }
    // taken as modified here, so that the reads are issued where they stand (next to the count
    // they go with) rather than moved into the branch that uses them
#pragma unroll
    for (int jj = 0; jj < JB; ++jj)
#pragma unroll
      for (int k = 0; k < IPP; ++k) asm volatile("" : "+v"(v[jj][k]));
  }
};

// Level 1, by the leader of tile t's local parts: wait until the other nl - 1 have counted their
// arrival, then add to its own sums `own` those of the others (each lane its parts in increasing
// order, then the lanes holding one slot index by a fixed exchange tree), and go on to level 2. The
// slots are read in the same round trip as the count that shows them all written: the LDS performs
// a wave's operations in issue order, so reads issued after the count see every slot counted in
// it. The wait cannot run out (the parts come from resident waves of this workgroup, none of which
// waits before handing its part over); a bound of about 100 ms on the real-time counter still
// keeps the wave from hanging, marking the sums invalid (NaN) if it were ever reached.
template <int M, int RPL, int MODE>
__device__ __forceinline__ void leader_collect(const KArgs& a, int t, const SplitGeo& s, const WgHo<M>* ho,
                                               const float (&own)[PartIdx<M, RPL, MODE>::N4],
                                               const uint64_t (&xpre)[PartIdx<M, RPL, MODE>::N4], int lane) {
  using I = PartIdx<M, RPL, MODE>;
  using L = LocalRead<M>;
  constexpr int NIDX = L::NIDX, PPI = L::PPI, IPP = L::IPP, JB = L::JB;
  L R;
  bool ok = true;
  const uint64_t deadline = __builtin_amdgcn_s_memrealtime() + 10000000ull;
  for (;;) {
    const uint32_t c = __hip_atomic_load(&ho->cnt[s.ci], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    asm volatile("" ::: "memory");
    R.read(ho, s, 0, lane);
    if (__builtin_amdgcn_readfirstlane(c) + 1 == (uint32_t)s.nl) break;
    if (__builtin_amdgcn_s_memrealtime() > deadline) {
      ok = false;
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  float ps[IPP];
#pragma unroll
  for (int k = 0; k < IPP; ++k) ps[k] = 0.0f;
  for (int j0 = 0; 1 + j0 < s.nl; j0 += PPI * JB) {
    if (j0 > 0) R.read(ho, s, j0, lane);
#pragma unroll
    for (int jj = 0; jj < JB; ++jj)
      if (L::part(j0, jj, lane) < s.nl)
#pragma unroll
        for (int k = 0; k < IPP; ++k) ps[k] += R.v[jj][k];
  }
  // lanes l and l ^ NIDX, ... hold the same slot index: add them, larger distances first
  if constexpr (NIDX <= 16) ps[0] += __shfl_xor(ps[0], 32);
  if constexpr (NIDX <= 16) ps[0] += __shfl_xor(ps[0], 16);
  if constexpr (NIDX == 32) ps[0] += __shfl_xor(ps[0], 32);
  const I ix(lane);
  float tot[I::N4];
#pragma unroll
  for (int i = 0; i < I::N4; ++i) {
    const int src = ix.idx[i] % 64, k = ix.idx[i] / 64;
    float other = 0.0f;
#pragma unroll
    for (int kk = 0; kk < IPP; ++kk) {
      const float u = __shfl(ps[kk], src);
      if (kk == k) other = u;
    }
    tot[i] = ok ? own[i] + other : __builtin_nanf("");
  }
  group_done<M, RPL, MODE>(a, t, s, tot, xpre, lane);
}

// A part whose tile work is left for after the step loop (a range's first part, emitted inside it):
// kind 1, a group of its own at level 2; kind 2, a local leader (not expected: a range's first
// part leads only when it is the workgroup's sole part of its tile). Its values wait in its
// wave's LDS slot (free: the part hands nothing over), or without LDS meeting in `v`.
template <int NV>
struct Pending {
  int t = -1, kind = 0;
  float v[NV];
};
template <int M, int RPL, int MODE, bool LDS_HO>
using PendingOf = Pending<LDS_HO ? 1 : PartIdx<M, RPL, MODE>::N4>;

// Finish the part [ca, cb) of tile t computed by wave g: reduce across lanes, then store y (whole
// tile) or hand the part over as described above. FINAL: the range's last part, after which the
// wave has no loads in flight; a range's first part emitted inside the loop leaves any work that
// could wait or make a round trip to after the loop (`pend`).
template <int M, int RPL, int MODE, bool LDS_HO, bool FINAL>
__device__ __forceinline__ void emit_part(const KArgs& a, float (&acc)[MODE == 2 ? M / 16 : M][RPL], int t, int ca,
                                          int cb, int g, int gr, int gl, int lane, WgHo<M>* ho,
                                          PendingOf<M, RPL, MODE, LDS_HO>& pend,
                                          const uint64_t (&xpre)[PartIdx<M, RPL, MODE>::N4]) {
  using I = PartIdx<M, RPL, MODE>;
  constexpr int H = 16 / RPL;
  float vals[I::NVAL];
#pragma unroll
  for (int b = 0; b < I::AR; ++b)
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
      vals[b * RPL + r] = acc[b][r];
      acc[b][r] = 0.0f;
    }
  if constexpr (MODE != 2) wave_reduce<I::NVAL, H>(vals, lane);
  const I ix(lane);
  float v4[I::N4];
#pragma unroll
  for (int i = 0; i < I::N4; ++i) v4[i] = vals[i];
  if (ca == 0 && cb == a.nc) {
    store_part<M, RPL, MODE>(a, t, ix, v4, true);
    return;
  }
  const SplitGeo s = split_geo<LDS_HO>(gr, gl, g);
  if (LDS_HO && s.nl > 1 && g != s.lw0) {
    // hand over to the local leader: slot, then count (in this order in the LDS; the compiler
    // barrier keeps them so), no wait
    float* mine = ho->slot[g % VALU_WPB];
    if (ix.writer)
#pragma unroll
      for (int i = 0; i < I::N4; ++i) mine[ix.idx[i]] = v4[i];
    asm volatile("" ::: "memory");
    if (lane == 0) __hip_atomic_fetch_add(&ho->cnt[s.ci], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    return;
  }
  if constexpr (FINAL) {
    if (LDS_HO && s.nl > 1) leader_collect<M, RPL, MODE>(a, t, s, ho, v4, xpre, lane);
    else group_done<M, RPL, MODE>(a, t, s, v4, xpre, lane);
  } else {
    pend.t = t;
    pend.kind = (LDS_HO && s.nl > 1) ? 2 : 1;
    if constexpr (LDS_HO) {
      if (ix.writer)
#pragma unroll
        for (int i = 0; i < I::N4; ++i) ho->slot[g % VALU_WPB][ix.idx[i]] = v4[i];
    } else {
#pragma unroll
      for (int i = 0; i < I::N4; ++i) pend.v[i] = v4[i];
    }
  }
}

// The work left by a range's first part (see Pending).
template <int M, int RPL, int MODE, bool LDS_HO>
__device__ __forceinline__ void follow_up(const KArgs& a, int g, int gr, int gl, int lane, const WgHo<M>* ho,
                                          const PendingOf<M, RPL, MODE, LDS_HO>& pend) {
  using I = PartIdx<M, RPL, MODE>;
  if (pend.t < 0) return;
  const SplitGeo s = split_geo<LDS_HO>(gr, gl, g);
  if constexpr (LDS_HO) {
    const I ix(lane);
    float v[I::N4];
#pragma unroll
    for (int i = 0; i < I::N4; ++i) v[i] = ix.writer ? ho->slot[g % VALU_WPB][ix.idx[i]] : 0.0f;
    const uint64_t none[I::N4] = {};
    if (pend.kind == 2) leader_collect<M, RPL, MODE>(a, pend.t, s, ho, v, none, lane);
    else group_done<M, RPL, MODE>(a, pend.t, s, v, none, lane);
  } else {
    const uint64_t none[I::N4] = {};
    group_done<M, RPL, MODE>(a, pend.t, s, pend.v, none, lane);
  }
}

// Lookup tables staged in two halves around the first record's loads: the table words are
// fetched first, the record loads are issued behind them, and the LDS stores wait only for the
// table words, so the first record's memory round trip overlaps the staging.
//
// With 8-bit directions the sign-folded tables (16 * 2^(D+1) entries of 8 bytes, 64 KiB) are
// expanded in the workgroup from the 2^D-entry codebook (16 bytes per entry), 16 times fewer
// bytes to fetch: every workgroup of a launch reads the same lines, so that fetch is bound by
// the L2 serving them (0.4 us per launch saved). For the smaller tables the expansion's extra
// work cost more than it saved, and they are copied as packed. Entry e < 16 * 2^D of T_lo is
// (z, s) = (e / 16, e % 16); entry e of T_hi is (s, z) = (e / 2^D, e % 2^D) after the first
// 16 * 2^D; both are the codebook's low (T_lo) or high (T_hi) four fp16 with the sign bits of s
// applied, as the packer lays them out.
template <int KIND, int D>
struct TableWords {
  static constexpr bool EXPAND = !IS_CB<KIND> && D >= 8;
  static constexpr int NLO = 16 << D;                       // entries of T_lo (and of T_hi)
  static constexpr int N16 = (int)((Tables<KIND, D>::bytes - (IS_CB<KIND> ? 128u : 0u)) / 16u);
  static constexpr int NITEM = EXPAND ? 2 * NLO : N16;     // 8-byte entries, or 16-byte words
  static constexpr int PER = (NITEM + VALU_THREADS - 1) / VALU_THREADS;
  typename std::conditional<EXPAND, uint2, uint4>::type w[PER];
};

template <int KIND, int D>
__device__ __forceinline__ void fetch_tables(TableWords<KIND, D>& tw, const KArgs& a) {
  using TW = TableWords<KIND, D>;
#pragma unroll
  for (int i = 0; i < TW::PER; ++i) {
    const int j = min((int)threadIdx.x + VALU_THREADS * i, TW::NITEM - 1);
    if constexpr (TW::EXPAND) {
      const bool hi = j >= TW::NLO;
      const int z = hi ? (j - TW::NLO) & ((1 << D) - 1) : j >> 4;
      tw.w[i] = ((const uint2*)a.CB)[2 * z + (hi ? 1 : 0)];
    } else {
      tw.w[i] = a.T[j];
    }
  }
}

template <int KIND, int D>
__device__ __forceinline__ void store_tables(unsigned char* lds, const TableWords<KIND, D>& tw, const KArgs& a) {
  using TW = TableWords<KIND, D>;
#pragma unroll
  for (int i = 0; i < TW::PER; ++i) {
    const int j = (int)threadIdx.x + VALU_THREADS * i;
    if (j < TW::NITEM) {
      if constexpr (TW::EXPAND) {
        const uint32_t sg = j >= TW::NLO ? (uint32_t)(j - TW::NLO) >> D : (uint32_t)j & 15u;
        uint2 v = tw.w[i];
        v.x ^= ((sg & 1u) << 15) | ((sg & 2u) << 30);
        v.y ^= ((sg & 4u) << 13) | ((sg & 8u) << 28);
        ((uint2*)lds)[j] = v;
      } else {
        ((uint4*)lds)[j] = tw.w[i];
      }
    }
  }
  if constexpr (IS_CB<KIND>) {
    // mask[s] flips the fp16 sign bit of element j (of 4) where bit j of the nibble s is set.
    if (threadIdx.x < 16) {
      const uint32_t s = threadIdx.x;
      uint2 m;
      m.x = ((s & 1u) << 15) | ((s & 2u) << 30);
      m.y = ((s & 4u) << 13) | ((s & 8u) << 28);
      *(uint2*)(lds + a.t_bytes + s * 8u) = m;
    }
  }
}

// The kernel: tables and the first record are fetched together, then each wave walks its range
// of steps through a ring of record buffers (see below). No wave ever waits for another one.
template <int KIND, int D, int M, int RPL, int MODE = 0>
__global__ void __launch_bounds__(VALU_THREADS)
__attribute__((amdgpu_waves_per_eu(VALU_WPB * VALU_WG_PER_CU / 4))) k_gemm_valu(KArgs a) {
  using S = Step<KIND, D, M, RPL, MODE>;
  // split-tile parts of waves of the same workgroup meet in LDS when it has room
  constexpr bool LDS_HO = lds_handover_fits(KIND, D, M, MODE);
  static_assert(VALU_WPB == 16, "lds_handover_fits assumes 16 waves per workgroup");
  static_assert(LDS_HO, "the LDS holds the tables and the split-tile hand-over slots");
  __shared__ __align__(16) unsigned char lds[Tables<KIND, D>::bytes];
  // per-wave staging: the group parameters (modes 0, 1) or the activations (mode 2, see XT_ROW)
  constexpr int PST = MODE == 2 ? (xt_staged(KIND, MODE) ? XT_WAVE / 4 : 0) : 64;   // dwords per wave
  __shared__ __align__(16) uint32_t pstage_all[PST > 0 ? VALU_WPB * PST : 1];
  __shared__ __align__(16) unsigned char ho_raw[LDS_HO ? sizeof(WgHo<M>) : 4];
  WgHo<M>* ho = (WgHo<M>*)ho_raw;
  constexpr int H = 16 / RPL;
  const int lane = threadIdx.x & 63;
  // wave-uniform by construction; readfirstlane keeps the schedule in SGPRs
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = (int)blockIdx.x * a.wpb + wave;
  // The range bounds are wave-uniform; readfirstlane keeps them (and every branch on them) scalar.
  const int r_lim = a.wg_tiles > 0 ? min(((int)blockIdx.x + 1) * a.wgs, a.ts) : a.ts;
  int s_begin = (a.wg_tiles > 0 ? (int)blockIdx.x * a.wgs + wave * a.wl : g * a.wl);
  int s_end = min(s_begin + a.wl, r_lim);
  const bool active = s_begin < r_lim;
  if (!active) {                             // an empty range (returns after the barrier)
    s_begin = 0;
    s_end = 1;
  }
  s_begin = __builtin_amdgcn_readfirstlane(s_begin);
  s_end = __builtin_amdgcn_readfirstlane(s_end);
  const int t0 = __builtin_amdgcn_readfirstlane(s_begin / a.nc);
  const int c0 = s_begin - t0 * a.nc;
  const int h = lane % H, vloc = lane / H;

  typename S::R r0, r1;
  TableWords<KIND, D> tw;
  fetch_tables<KIND, D>(tw, a);
  S::load(r0, a, t0, c0, h, vloc, lane);
  // the waves holding the first and the last step of the range's first and last tile (see SplitGeo)
  const int tl = __builtin_amdgcn_readfirstlane((s_end - 1) / a.nc);
  const int gr0 = wave_of_step(a, t0 * a.nc), gl0 = wave_of_step(a, t0 * a.nc + a.nc - 1);
  const int grl = wave_of_step(a, tl * a.nc), gll = wave_of_step(a, tl * a.nc + a.nc - 1);
  store_tables<KIND, D>(lds, tw, a);
  if constexpr (LDS_HO)
    if (threadIdx.x <= VALU_WPB) ho->cnt[threadIdx.x] = 0u;
  const uint32_t mask_off = a.t_bytes;
  __syncthreads();
  if (!active) return;                       // no barrier follows
  uint32_t* pstage = pstage_all + wave * PST;

  float acc[S::AR][RPL];
#pragma unroll
  for (int b = 0; b < S::AR; ++b)
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr) acc[b][rr] = 0.0f;

  // Two record buffers in ping-pong: the loads of step i+1 are in flight while step i is
  // computed. The loop runs over pairs of steps, one per buffer, with a single exit at the
  // bottom (an early exit would give the compiler a path back to the loop head with loads still
  // pending, and it would wait for them). The range's last step is peeled off: the tile parts
  // that end inside the loop are whole tiles or the range's first part, and the last part, which
  // may be part 0 of a split tile, is finished after it.
  const int nsteps = s_end - s_begin;
  const int npairs = (nsteps - 1) >> 1;
  PendingOf<M, RPL, MODE, LDS_HO> pend;
  using PI = PartIdx<M, RPL, MODE>;
  const uint64_t xnone[PI::N4] = {};         // no workspace words read ahead (parts inside the loop)
  int t = t0, c = c0;                        // position of step 2i
  for (int i = 0; i < npairs; ++i) {
    int t1 = t, c1 = c + 1;
    if (c1 == a.nc) {
      ++t1;
      c1 = 0;
    }
    S::load(r1, a, t1, c1, h, vloc, lane);
    S::compute(r0, acc, lds, mask_off, pstage, lane, h, vloc);
    if (c1 == 0) emit_part<M, RPL, MODE, LDS_HO, false>(a, acc, t, t == t0 ? c0 : 0, a.nc, g, gr0, gl0, lane, ho, pend, xnone);
    int t2 = t1, c2 = c1 + 1;
    if (c2 == a.nc) {
      ++t2;
      c2 = 0;
    }
    S::load(r0, a, t2, c2, h, vloc, lane);   // step 2i + 2 <= nsteps - 1 exists
    S::compute(r1, acc, lds, mask_off, pstage, lane, h, vloc);
    if (c2 == 0) emit_part<M, RPL, MODE, LDS_HO, false>(a, acc, t1, t1 == t0 ? c0 : 0, a.nc, g, gr0, gl0, lane, ho, pend, xnone);
    t = t2;
    c = c2;
  }
  // r0 holds step 2 * npairs; one or two steps remain, the last one being the range's last.
  int tf = t, cf = c;                        // position of the last step
  if (nsteps - 2 * npairs == 2) {
    cf = c + 1;
    if (cf == a.nc) {
      ++tf;
      cf = 0;
    }
    S::load(r1, a, tf, cf, h, vloc, lane);
    S::compute(r0, acc, lds, mask_off, pstage, lane, h, vloc);
    if (cf == 0) emit_part<M, RPL, MODE, LDS_HO, false>(a, acc, t, t == t0 ? c0 : 0, a.nc, g, gr0, gl0, lane, ho, pend, xnone);
  }
  const int caf = tf == t0 ? c0 : 0;
  // one instance of the step code for the last step: its records are moved into r0 when r1 holds
  // them (a reference chosen between the two buffers would put both in scratch memory)
  if (nsteps - 2 * npairs == 2) r0 = r1;
  // The final part's tile over two workgroups, finished from this wave (its only part in this
  // workgroup, or the local leader): read its workspace words now, so that their round trip
  // overlaps the last step; if the other workgroup has already left its sums there, this wave
  // finishes the tile without an exchange at the end.
  uint64_t xw[PI::N4] = {};
  if (!(caf == 0 && cf + 1 == a.nc)) {
    const SplitGeo sl = split_geo<LDS_HO>(grl, gll, g);
    if (sl.ngrp == 2 && (sl.nl == 1 || g == sl.lw0)) {
      const PI ix(lane);
      const uint64_t* words = a.ws_slot + (int64_t)tf * a.pmax * (M * 16);
#pragma unroll
      for (int i = 0; i < PI::N4; ++i)
        xw[i] = ix.writer ? __hip_atomic_load(words + ix.idx[i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0ull;
    }
  }
  S::compute(r0, acc, lds, mask_off, pstage, lane, h, vloc);
  emit_part<M, RPL, MODE, LDS_HO, true>(a, acc, tf, caf, cf + 1, g, grl, gll, lane, ho, pend, xw);
  follow_up<M, RPL, MODE, LDS_HO>(a, g, gr0, gl0, lane, ho, pend);
}

// ------------------------------------------------------------------------------------------
// Unpack: logical codes through the compute kernels' field extraction.
// ------------------------------------------------------------------------------------------
template <int KIND, int D>
__global__ void __launch_bounds__(256) k_unpack(KArgs a, uint8_t* signs, uint16_t* dir, uint8_t* qo) {
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)a.nt * a.nv * 16;
  if (idx >= total) return;
  const int r = (int)(idx & 15);
  const int64_t rec = idx >> 4;
  const int64_t t = rec / a.nv, v = rec % a.nv;
  const int64_t row = t * 16 + r;
  if (row >= a.n) return;
  uint32_t s, z, q;
  if constexpr (IS_CB<KIND>) {
    decode_cb13(a.A[rec * 4 + (r >> 2)], r & 3, a.B[rec * 8 + (r >> 1)], r & 1, s, z, q);
    if constexpr (KIND == SPH_KIND_CB13Q4) q |= ((uint32_t)(a.C[rec] >> r) & 1u) << 3;
  } else {
    const uint32_t d = a.A[rec * 8 + (r >> 1)];
    uint32_t qx = 0;
    if constexpr (KIND == SPH_KIND_W2) qx = (a.B[rec] >> (4 * (r >> 1))) & 15u;
    if constexpr (KIND == SPH_KIND_NIB16Q2) qx = (a.B[rec] >> (2 * r)) & 3u;
    if constexpr (KIND == SPH_KIND_NIB16Q8) qx = (a.B[rec * 4 + (r >> 2)] >> (8 * (r & 3))) & 0xFFu;
    uint32_t lo, hi;
    decode_nib<KIND, D>(d, r & 1, qx, lo, hi, q);
    const uint32_t zlo = lo >> 4, zhi = hi & ((1u << D) - 1u);
    s = (lo & 15u) | ((hi >> D) << 4);
    z = (zlo == zhi) ? zlo : 0xFFFFu;
  }
  const int64_t o = row * a.nv + v;
  signs[o] = (uint8_t)s;
  dir[o] = (uint16_t)z;
  qo[o] = (uint8_t)q;
}

// ------------------------------------------------------------------------------------------
// Prefill kernel (batch > 16, and 9..16 on large matrices): Y = X W^T on 16x16x32 MFMA tiles
// with the operands rebuilt once per workgroup and k-chunk.
//
// A workgroup of PF_WAVES waves owns PF_TPW 16-row tiles per wave and MC batch rows (one grid
// column per MC-row slice of X), and walks K in chunks of 128 (16 vector positions = one radius
// group). Per chunk the X slice [MC][128] is staged in LDS (rows padded by 16 bytes against bank
// conflicts); each lane rebuilds, for each of its tiles, row lane % 16 at positions 4i + lane / 16
// (i = 0..3) as exact fp16 operands -- the signed direction t and the two halves of q * t, in the
// operand layout of the batch 9..16 tile mode -- and every rebuilt operand meets all MC / 16
// column blocks of X, each X fragment serving both tiles. Eq. 7 factors over the chunk's group:
// the chunk adds offset * sum <t, x> + step * sum q <t, x> to each output. With ks > 1
// the grid's third dimension splits K and the partial outputs are added in range order by
// k_prefill_reduce. The order of every sum is fixed, so results are reproducible.
// ------------------------------------------------------------------------------------------
constexpr int PF_WAVES = 8;
constexpr int PF_TPW = 2;
constexpr int PF_KS_MAX = 16;   // K ranges of a split at most
constexpr int PF_THREADS = 64 * PF_WAVES;
constexpr int PF_XROW = 128 * 2 + 16;   // bytes per staged X row (128 fp16 + padding)
#define SPH_MAX_BATCH 65536

// Per-chunk staging of the prefill kernel: the X slice and, for the workgroup's PF_WAVES * PF_TPW
// tiles, their records of the chunk (streams A, B, C) and group parameters. Each lands in LDS with
// one barrier; the next chunk's is meanwhile loaded into registers, so the multiply phase reads
// LDS only.
template <int KIND, int MC>
struct PfStage {
  static constexpr int TILES = PF_WAVES * PF_TPW;
  static constexpr bool B1 = KIND == SPH_KIND_W2 || KIND == SPH_KIND_NIB16Q2;
  static constexpr int ADW = IS_CB<KIND> ? 4 : 8;                                 // dwords per record
  static constexpr int BDW = KIND == SPH_KIND_NIB16 ? 0 : B1 ? 1 : (KIND == SPH_KIND_NIB16Q8) ? 4 : 8;
  static constexpr int CH = KIND == SPH_KIND_CB13Q4 ? 1 : 0;                      // halves per record
  // 16-byte pieces per tile and chunk (16 records; 16 rows of parameters)
  static constexpr int A16 = 16 * ADW / 4, B16 = 16 * BDW / 4, C16 = 16 * CH * 2 / 16, P16 = 4;
  static constexpr int CODE16 = TILES * (A16 + B16 + C16 + P16);
  static constexpr int X16 = MC * 16;
  static constexpr int PER = (X16 + CODE16 + PF_THREADS - 1) / PF_THREADS;
  // byte offsets inside one stage buffer
  static constexpr uint32_t x_bytes = MC * PF_XROW;
  static constexpr uint32_t a_off = x_bytes, b_off = a_off + TILES * A16 * 16, c_off = b_off + TILES * B16 * 16,
                            p_off = c_off + TILES * C16 * 16, bytes = p_off + TILES * P16 * 16;
};

template <int KIND, int D, int MC>
struct PfLds {
  static constexpr int nbuf = IS_CB<KIND> ? 1 : 2;
  static constexpr uint32_t x_off = (Tables<KIND, D>::bytes + 15u) / 16u * 16u;
  static constexpr uint32_t bytes = x_off + nbuf * PfStage<KIND, MC>::bytes;
};

// One rebuilt MFMA operand of the prefill kernel: the signed direction t of row r at one position
// (exact in fp16) and q * t split exactly into two fp16 words (see qt_split).
struct PfOp {
  uint4 t, hi, lo;
};

template <int KIND, int D>
__device__ __forceinline__ PfOp pf_rebuild(const uint32_t ra, const uint32_t rb, const uint32_t rc,
                                           const unsigned char* lds, uint32_t mask_off, int r) {
  PfOp o;
  uint32_t q;
  if constexpr (IS_CB<KIND>) {
    uint32_t sg, z;
    decode_cb13(ra, r % 4, rb, r & 1, sg, z, q);
    if constexpr (KIND == SPH_KIND_CB13Q4) q |= ((rc >> r) & 1u) << 3;
    o.t = signed_dir_cb13(lds, mask_off, sg, z);
  } else {
    uint32_t l, hh, qx = 0;
    if constexpr (KIND == SPH_KIND_W2) qx = (rb >> (4 * (r / 2))) & 15u;
    if constexpr (KIND == SPH_KIND_NIB16Q2) qx = (rb >> (2 * r)) & 3u;
    if constexpr (KIND == SPH_KIND_NIB16Q8) qx = (rb >> (8 * (r % 4))) & 0xFFu;
    decode_nib<KIND, D>(ra, r & 1, qx, l, hh, q);
    o.t = signed_dir_nib<KIND, D>(lds, l, hh);
  }
  qt_split(o.t, q, o.hi, o.lo);
  return o;
}

// Load the PER 16-byte pieces of chunk c that this thread stages (X rows past the batch repeat
// the last row; tiles past the matrix repeat the last tile: neither is ever stored).
template <int KIND, int MC>
struct PfPre {
  uint4 v[PfStage<KIND, MC>::PER];
};

template <int KIND, int MC>
__device__ __forceinline__ void pf_fetch(PfPre<KIND, MC>& pr, const KArgs& a, int t0, int mc0, int c) {
  using S = PfStage<KIND, MC>;
#pragma unroll
  for (int p = 0; p < S::PER; ++p) {
    int q = (int)threadIdx.x + PF_THREADS * p;
    uint4 val = make_uint4(0, 0, 0, 0);
    // divisors of empty streams are never used; max(1, .) keeps them defined
    constexpr int a16 = S::A16 > 0 ? S::A16 : 1, b16 = S::B16 > 0 ? S::B16 : 1, c16 = S::C16 > 0 ? S::C16 : 1;
    if (q < S::X16) {
      const int b = min(mc0 + (q >> 4), a.m - 1);
      val = *(const uint4*)(a.x + (int64_t)b * a.ldx + (int64_t)c * 128 + (q & 15) * 8);
    } else if ((q -= S::X16) < S::TILES * S::A16) {
      const int64_t t = min(t0 + q / a16, a.nt - 1);
      val = ((const uint4*)(a.A + (t * a.nv + c * 16) * S::ADW))[q % a16];
    } else if ((q -= S::TILES * S::A16) < S::TILES * S::B16) {
      const int64_t t = min(t0 + q / b16, a.nt - 1);
      val = ((const uint4*)(a.B + (t * a.nv + c * 16) * S::BDW))[q % b16];
    } else if ((q -= S::TILES * S::B16) < S::TILES * S::C16) {
      const int64_t t = min(t0 + q / c16, a.nt - 1);
      val = ((const uint4*)(a.C + (t * a.nv + c * 16) * S::CH))[q % c16];
    } else if ((q -= S::TILES * S::C16) < S::TILES * S::P16) {
      const int64_t t = min(t0 + q / S::P16, a.nt - 1);
      val = ((const uint4*)(a.P + (t * a.ng + c) * 16))[q % S::P16];
    }
    pr.v[p] = val;
  }
}

template <int KIND, int MC>
__device__ __forceinline__ void pf_put(unsigned char* st, const PfPre<KIND, MC>& pr) {
  using S = PfStage<KIND, MC>;
#pragma unroll
  for (int p = 0; p < S::PER; ++p) {
    const int q = (int)threadIdx.x + PF_THREADS * p;
    if (q < S::X16)
      *(uint4*)(st + (q >> 4) * PF_XROW + (q & 15) * 16) = pr.v[p];
    else if (q < S::X16 + S::CODE16)
      *(uint4*)(st + S::a_off + (q - S::X16) * 16) = pr.v[p];
  }
}

template <int KIND, int D, int MC>
__global__ void __launch_bounds__(PF_THREADS) k_gemm_prefill(KArgs a) {
  constexpr int NB = MC / 16;
  using S = PfStage<KIND, MC>;
  using L = PfLds<KIND, D, MC>;
  __shared__ __align__(16) unsigned char lds[L::bytes];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r = lane & 15, j = lane >> 4;
  const int mc0 = blockIdx.y * MC;
  const int t0 = (int)blockIdx.x * S::TILES;
  const int nc = a.ng;
  const int c0 = (int)((int64_t)nc * blockIdx.z / a.ks), c1 = (int)((int64_t)nc * (blockIdx.z + 1) / a.ks);
  PfPre<KIND, MC> pre;
  pf_fetch<KIND, MC>(pre, a, t0, mc0, c0);
  {
    // the tables in batches of up to 8 loads per thread, each batch one round trip
    constexpr int n16 = (int)((Tables<KIND, D>::bytes - (IS_CB<KIND> ? 128u : 0u)) / 16u);
    constexpr int TPER = (n16 + PF_THREADS - 1) / PF_THREADS, TB = TPER < 8 ? TPER : 8;
#pragma unroll
    for (int p0 = 0; p0 < TPER; p0 += TB) {
      uint4 tv[TB];
#pragma unroll
      for (int p = 0; p < TB; ++p) tv[p] = a.T[min((int)threadIdx.x + PF_THREADS * (p0 + p), n16 - 1)];
#pragma unroll
      for (int p = 0; p < TB; ++p) {
        const int t = (int)threadIdx.x + PF_THREADS * (p0 + p);
        if (t < n16) ((uint4*)lds)[t] = tv[p];
      }
    }
    if constexpr (IS_CB<KIND>) {
      if (threadIdx.x < 16) {
        const uint32_t sm = threadIdx.x;
        uint2 mk;
        mk.x = ((sm & 1u) << 15) | ((sm & 2u) << 30);
        mk.y = ((sm & 4u) << 13) | ((sm & 8u) << 28);
        *(uint2*)(lds + a.t_bytes + sm * 8u) = mk;
      }
    }
  }
  f32x4 acc[PF_TPW][NB];
#pragma unroll
  for (int u = 0; u < PF_TPW; ++u)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[u][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  // the row's dword in streams A and B, as in the batch 9..16 tile mode
  const int adw = IS_CB<KIND> ? r / 4 : r / 2;
  const int bdw = S::B1 ? 0 : (KIND == SPH_KIND_NIB16Q8) ? r / 4 : r / 2;
  for (int c = c0; c < c1; ++c) {
    unsigned char* st = lds + L::x_off + (L::nbuf == 2 ? (c & 1) : 0) * S::bytes;
    // with one buffer, wait until every wave has finished reading the previous chunk
    if constexpr (L::nbuf == 1) __syncthreads();
    pf_put<KIND, MC>(st, pre);
    // chunk c (and, first time round, the tables) become visible; with two buffers this also
    // orders the reads of buffer (c & 1) at chunk c - 2 before this chunk's writes to it
    __syncthreads();
    pf_fetch<KIND, MC>(pre, a, t0, mc0, min(c + 1, c1 - 1));   // in flight during the multiply
    const uint32_t* sa = (const uint32_t*)(st + S::a_off);
    const uint32_t* sb = (const uint32_t*)(st + S::b_off);
    const uint16_t* sc = (const uint16_t*)(st + S::c_off);
    const uint32_t* sp = (const uint32_t*)(st + S::p_off);
    auto rebuild_i = [&](int i, PfOp (&w)[PF_TPW]) {
#pragma unroll
      for (int u = 0; u < PF_TPW; ++u) {
        const int lt = wave * PF_TPW + u, rec = lt * 16 + 4 * i + j;
        const uint32_t ra = sa[rec * S::ADW + adw];
        uint32_t rb = 0u;
        if constexpr (S::BDW > 0) rb = sb[rec * S::BDW + bdw];
        uint32_t rc = 0u;
        if constexpr (S::CH > 0) rc = sc[rec];
        w[u] = pf_rebuild<KIND, D>(ra, rb, rc, lds, a.t_bytes, r);
      }
    };
    // A chunk is one radius group, so Eq. 7 factors over it: per (row, batch row) the chunk adds
    // offset * sum <t, x> + step * sum q <t, x>, both sums formed by the MFMA from exact fp16
    // operands. The operands of position group i + 1 are rebuilt before the multiplies of group i,
    // so that their LDS round trips overlap the matrix-core work.
    f32x4 s0[PF_TPW][NB], s1[PF_TPW][NB];
#pragma unroll
    for (int u = 0; u < PF_TPW; ++u)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) s0[u][nb] = s1[u][nb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    PfOp wc[PF_TPW];
    rebuild_i(0, wc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      PfOp wn[PF_TPW];
      if (i + 1 < 4) rebuild_i(i + 1, wn);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const f16x8 xb = __builtin_bit_cast(f16x8, *(const uint4*)(st + (16 * nb + r) * PF_XROW + (4 * i + j) * 16));
#pragma unroll
        for (int u = 0; u < PF_TPW; ++u) {
          s0[u][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, wc[u].t), xb, s0[u][nb], 0, 0, 0);
          s1[u][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, wc[u].hi), xb, s1[u][nb], 0, 0, 0);
          s1[u][nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, wc[u].lo), xb, s1[u][nb], 0, 0, 0);
        }
      }
      if (i + 1 < 4)
#pragma unroll
        for (int u = 0; u < PF_TPW; ++u) wc[u] = wn[u];
    }
    // fold the chunk's sums in with the offset and step of rows 4 * (lane / 16) + e
#pragma unroll
    for (int u = 0; u < PF_TPW; ++u) {
      const uint4 pw = *(const uint4*)(sp + (wave * PF_TPW + u) * 16 + 4 * j);
      const uint32_t pe[4] = {pw.x, pw.y, pw.z, pw.w};
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          acc[u][nb][e] = fmaf(f16hi(pe[e]), s1[u][nb][e], fmaf(f16lo(pe[e]), s0[u][nb][e], acc[u][nb][e]));
    }
  }
  // D[row][col] of a 16x16 block: lane holds col lane % 16 (batch row) and rows 4 * (lane / 16) + e
#pragma unroll
  for (int u = 0; u < PF_TPW; ++u) {
    const int tile = t0 + wave * PF_TPW + u;
    if (tile >= a.nt) continue;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int b = mc0 + 16 * nb + r;
      if (b >= a.m) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = tile * 16 + 4 * j + e;
        if (a.ks > 1) {
          a.ws_part[((int64_t)blockIdx.z * a.m + b) * ((int64_t)a.nt * 16) + row] = acc[u][nb][e];
        } else if (row < a.n) {
          store_y(a, b, row, acc[u][nb][e]);
        }
      }
    }
  }
}

// y[b][row] = sum over the K ranges, in range order, of the prefill partials, which are cleared.
// Four consecutive rows per thread, so that every access to the partials is 16 bytes wide (the
// rows are padded to whole tiles, and a range's partials start on a 64-byte boundary). All of a
// thread's partials are read before any is cleared: read-add-clear per range made each read wait
// for the previous range's store (the compiler cannot tell the addresses apart), one memory round
// trip per range.
__global__ void __launch_bounds__(256) k_prefill_reduce(KArgs a) {
  const int64_t npad = (int64_t)a.nt * 16, nq = npad / 4;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)a.m * nq) return;
  const int b = (int)(t / nq), row = (int)(t % nq) * 4;
  f32x4* p0 = (f32x4*)(a.ws_part + (int64_t)b * npad + row);
  const int64_t zs = (int64_t)a.m * nq;   // f32x4 elements between consecutive ranges
  f32x4 v[PF_KS_MAX];   // the kernel runs only for ks >= 2
#pragma unroll
  for (int z = 0; z < PF_KS_MAX; ++z)
    if (z < 2 || z < a.ks) v[z] = p0[z * zs];
  f32x4 s = v[0];
#pragma unroll
  for (int z = 1; z < PF_KS_MAX; ++z)
    if (z < 2 || z < a.ks) s += v[z];
#pragma unroll
  for (int z = 0; z < PF_KS_MAX; ++z)
    if (z < 2 || z < a.ks) p0[z * zs] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};   // left zero-filled, as every call promises
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (row + e < a.n) store_y(a, b, row + e, s[e]);
}

// ------------------------------------------------------------------------------------------
// Row-planar kernels for 4-D and 16-D vectors (Tab. 7), batch 1..32.
//
// One wave per output row. Per step a lane covers 64 consecutive weights of the row (16 4-D or
// 4 16-D vectors, inside one 128-weight group), so a step covers 4096 weights; the row sum is a
// wave reduction. The 4-D signed directions come from a 64-entry sign-folded table in LDS; a 16-D
// codebook entry is read from memory (the 512 KiB codebook stays in L2) and its signs applied by
// XOR on the fp16 sign bits. Batch 1 forms exact fp16 products with fp32 sums and applies the
// radius in fp32, as the 8-D vector-ALU mode does; larger batches decode the lane's vectors once
// and reuse them for every activation row with the same exact-product arithmetic.
// ------------------------------------------------------------------------------------------
constexpr int RV_WAVES = 4;

template <int KIND>
__device__ __forceinline__ void rv_vector(const KArgs& a, const uint2* tab, const uint4 f, int u, uint32_t bw, int vin,
                                          float lo, float st, float& r, uint32_t (&t)[8]) {
  if constexpr (KIND == SPH_KIND_V4) {
    const uint32_t word = u < 4 ? f.x : u < 8 ? f.y : u < 12 ? f.z : f.w;
    const uint32_t byte = (word >> (8 * (u & 3))) & 0xFFu;
    const uint32_t q = (byte >> 6) | (((bw >> (vin + u)) & 1u) << 2);
    r = fmaf((float)q, st, lo);
    const uint2 e = tab[byte & 63u];
    t[0] = e.x;
    t[1] = e.y;
  } else {
    const uint32_t fw = u == 0 ? f.x : u == 1 ? f.y : u == 2 ? f.z : f.w;
    const uint32_t s = fw & 0xFFFFu, z = (fw >> 16) & 0x3FFFu;
    const uint32_t q = (fw >> 30) | (((bw >> (4 * (vin + u))) & 15u) << 2);
    r = fmaf((float)q, st, lo);
    const uint4* cz = (const uint4*)(a.CB + (int64_t)z * 16);
    const uint4 c0 = cz[0], c1 = cz[1];
    const uint32_t c[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
#pragma unroll
    for (int i = 0; i < 8; ++i) t[i] = c[i] ^ ((((s >> (2 * i)) & 1u) << 15) | (((s >> (2 * i + 1)) & 1u) << 31));
  }
}

template <int KIND, int MB>
__global__ void __launch_bounds__(64 * RV_WAVES) k_gemm_rowvec(KArgs a) {
  constexpr int VEC = KIND == SPH_KIND_V4 ? 4 : 16;
  constexpr int NVL = 64 / VEC;              // vectors per lane and step
  constexpr int TW = VEC / 2;                // fp16 pairs per vector
  __shared__ uint2 tab[KIND == SPH_KIND_V4 ? 64 : 1];
  if constexpr (KIND == SPH_KIND_V4) {
    if (threadIdx.x < 64) tab[threadIdx.x] = ((const uint2*)a.T)[threadIdx.x];
    __syncthreads();
  }
  const int lane = threadIdx.x & 63;
  const int row = (int)blockIdx.x * RV_WAVES + (int)(threadIdx.x >> 6);
  if (row >= a.n) return;   // after the only barrier
  const int64_t k = (int64_t)a.ng * 128;
  float acc[MB];
#pragma unroll
  for (int b = 0; b < MB; ++b) acc[b] = 0.0f;
  for (int64_t k0 = 0; k0 < k; k0 += 4096) {
    const int64_t kw = k0 + (int64_t)lane * 64;
    if (kw >= k) continue;
    const int g = (int)(kw >> 7);
    const uint32_t pw = a.P[(int64_t)row * a.ng + g];
    const uint32_t bw = a.B[(int64_t)row * a.ng + g];
    const float lo = f16lo(pw), st = f16hi(pw);
    const int vin = (int)((kw & 127) / VEC);
    uint4 f;
    if constexpr (KIND == SPH_KIND_V4)
      f = *(const uint4*)((const uint8_t*)a.A + (int64_t)row * a.nv + kw / 4);
    else
      f = *(const uint4*)(a.A + (int64_t)row * a.nv + kw / 16);
    if constexpr (MB == 1) {
      const uint32_t* xp = (const uint32_t*)(a.x + kw);
#pragma unroll
      for (int u = 0; u < NVL; ++u) {
        float r;
        uint32_t t[8];
        rv_vector<KIND>(a, tab, f, u, bw, vin, lo, st, r, t);
        float d = 0.0f;
#pragma unroll
        for (int i = 0; i < TW; ++i) d = __builtin_amdgcn_fdot2(as_h2(t[i]), as_h2(xp[u * TW + i]), d, false);
        acc[0] = fmaf(r, d, acc[0]);
      }
    } else {
      // the lane's vectors once (signed directions exact in fp16, radii in fp32), then per batch
      // row the exact-product dots of each vector, scaled by its radius in fp32
      float rr[NVL];
      uint32_t tw[NVL][TW];
#pragma unroll
      for (int u = 0; u < NVL; ++u) {
        uint32_t t[8];
        rv_vector<KIND>(a, tab, f, u, bw, vin, lo, st, rr[u], t);
#pragma unroll
        for (int i = 0; i < TW; ++i) tw[u][i] = t[i];
      }
#pragma unroll
      for (int b = 0; b < MB; ++b) {
        if (b < a.m) {
          const uint4* xp = (const uint4*)(a.x + (int64_t)b * a.ldx + kw);
          uint32_t xw[32];
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const uint4 xv = xp[i];
            xw[4 * i] = xv.x; xw[4 * i + 1] = xv.y; xw[4 * i + 2] = xv.z; xw[4 * i + 3] = xv.w;
          }
          float s = acc[b];
#pragma unroll
          for (int u = 0; u < NVL; ++u) {
            float d = 0.0f;
#pragma unroll
            for (int i = 0; i < TW; ++i) d = __builtin_amdgcn_fdot2(as_h2(tw[u][i]), as_h2(xw[u * TW + i]), d, false);
            s = fmaf(rr[u], d, s);
          }
          acc[b] = s;
        }
      }
    }
  }
#pragma unroll
  for (int b = 0; b < MB; ++b) {
    float v = acc[b];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0 && b < a.m) store_y(a, b, row, v);
  }
}

// Logical codes of the row-planar kinds: signs (a byte for 4-D, a uint16 for 16-D), direction
// index and level, one thread per vector.
template <int KIND>
__global__ void __launch_bounds__(256) k_unpack_rowvec(KArgs a, uint8_t* signs, uint16_t* dir, uint8_t* qo) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nvec = (int64_t)a.n * a.nv;
  if (i >= nvec) return;
  const int64_t row = i / a.nv, v = i - row * a.nv;
  constexpr int VPG = KIND == SPH_KIND_V4 ? 32 : 8;
  const uint32_t bw = a.B[row * a.ng + v / VPG];
  const int vin = (int)(v % VPG);
  if constexpr (KIND == SPH_KIND_V4) {
    const uint32_t byte = ((const uint8_t*)a.A)[i];
    signs[i] = (uint8_t)(byte & 15u);
    dir[i] = (uint16_t)((byte >> 4) & 3u);
    qo[i] = (uint8_t)((byte >> 6) | (((bw >> vin) & 1u) << 2));
  } else {
    const uint32_t fw = a.A[i];
    ((uint16_t*)signs)[i] = (uint16_t)(fw & 0xFFFFu);
    dir[i] = (uint16_t)((fw >> 16) & 0x3FFFu);
    qo[i] = (uint8_t)((fw >> 30) | (((bw >> (4 * vin)) & 15u) << 2));
  }
}

// ------------------------------------------------------------------------------------------
// Host dispatch
// ------------------------------------------------------------------------------------------
namespace {

struct Launch {
  const void* fn;
  int block;          // threads per workgroup
  int grid;
  int nc, wg_tiles, wl, wgs, pmax, ts;
  size_t ws_bytes;    // workspace the launch needs
  size_t cnt_off;     // offset of the split-tile arrival counters in it
};

KArgs make_args(const sph_weights* w) {
  KArgs a{};
  const int kind = sph_kind_of_fmt(w->fmt.vec_dim, w->fmt.dir_bits, w->fmt.radius_bits);
  const char* base = (const char*)w->d_base;
  a.A = (const uint32_t*)(base + w->off[SPH_OFF_A]);
  a.B = (const uint32_t*)(base + w->off[SPH_OFF_B]);
  a.P = (const uint32_t*)(base + w->off[SPH_OFF_PARAMS]);
  a.C = (const uint16_t*)(base + w->off[SPH_OFF_C]);
  a.T = (const uint4*)(base + w->off[SPH_OFF_TABLES]);
  a.CB = (const uint16_t*)(base + w->off[SPH_OFF_CODEBOOK]);
  a.t_bytes = (uint32_t)sph_table_bytes(kind, w->fmt.dir_bits);
  a.n = (int)w->n;
  a.nt = (int)((w->n + 15) / 16);
  a.nv = (int)(w->k / w->fmt.vec_dim);
  a.ng = (int)(w->k / 128);
  return a;
}

// Rows per lane of the batch-1 mode: 8, two lanes per vector position (twice the waves, each
// step half as long). The template also takes 16 (one lane per position), which is no longer
// instantiated: with fixed-length wave ranges and the two-level split-tile hand-over it was
// slower on every shape timed (W2 4096x12288 8.36 -> 7.67 us with 8 rows, 5120x25600 16.9 ->
// 15.7, 5120x5120 7.41 -> 7.04, 51200x5120 27.5 -> 27.0; the 32B-class step 3.46 -> 3.32 ms).
constexpr int B1_RPL = 8;

template <int KIND, int D>
const void* valu_fn(int M) {
  switch (M) {
    case 1:
      return (const void*)k_gemm_valu<KIND, D, 1, B1_RPL, 0>;
    case 2:
      if constexpr (!IS_CB<KIND>) return (const void*)k_gemm_valu<KIND, D, 2, 8, 0>;
      return nullptr;
    case 4: return (const void*)k_gemm_valu<KIND, D, 4, 4, 1>;
    case 8: return (const void*)k_gemm_valu<KIND, D, 8, 4, 1>;
  }
  return (const void*)k_gemm_valu<KIND, D, 16, 4, 2>;
}

const void* pick(int D, int V, int M) {
  switch (sph_kind_of(D, V)) {
    case SPH_KIND_W2: return D == 7 ? valu_fn<SPH_KIND_W2, 7>(M) : valu_fn<SPH_KIND_W2, 6>(M);
    case SPH_KIND_NIB16:
      if (D == 4) return valu_fn<SPH_KIND_NIB16, 4>(M);
      if (D == 5) return valu_fn<SPH_KIND_NIB16, 5>(M);
      return valu_fn<SPH_KIND_NIB16, 6>(M);
    case SPH_KIND_NIB16Q8: return valu_fn<SPH_KIND_NIB16Q8, 8>(M);
    case SPH_KIND_NIB16Q2: return valu_fn<SPH_KIND_NIB16Q2, 8>(M);
    case SPH_KIND_CB13: return valu_fn<SPH_KIND_CB13, 13>(M);
    case SPH_KIND_CB13Q4: return valu_fn<SPH_KIND_CB13Q4, 13>(M);
  }
  return nullptr;
}

template <int KIND, int D>
const void* prefill_fn_mc(int mc) {
  if (mc == 16) return (const void*)k_gemm_prefill<KIND, D, 16>;
  if (mc == 32) return (const void*)k_gemm_prefill<KIND, D, 32>;
  return (const void*)k_gemm_prefill<KIND, D, 64>;
}

// Batch rows per workgroup: 16 for batches 9..16, 32 for 17..32, else 64 (the two fp32 sums of
// the factored product double the accumulators, which 128 rows would not leave room for).
int prefill_mc(int, int, int64_t m) { return m <= 16 ? 16 : m <= 32 ? 32 : 64; }

// Batches 17..32 always, and 9..16 on large matrices, run on the prefill kernel, whose activations
// are staged in LDS once per workgroup and chunk and shared by its 16 row tiles; in the 16x16x32
// tile mode every wave reloads them. From about 1.2 * 10^8 weights the reloads cost more than
// the staging: at 16 batch rows 51200x5120 takes about 70 us in the tile mode and 63 us on the
// prefill kernel, 32768x4096 37 and 34 us, while 24576x4096 (29.5 against 31.8 us) and smaller
// matrices stay faster in the tile mode; at 9 batch rows the prefill kernel gains 6-13% from
// 1.25 * 10^8 (5120x25600).
bool small_on_prefill(const sph_weights* w, int64_t m) {
  if (m > 16) return true;
  if (m < 9) return false;
  return (int64_t)w->n * w->k >= 120ll << 20;
}

const void* prefill_fn(int D, int V, int mc) {
  switch (sph_kind_of(D, V)) {
    case SPH_KIND_W2: return D == 7 ? prefill_fn_mc<SPH_KIND_W2, 7>(mc) : prefill_fn_mc<SPH_KIND_W2, 6>(mc);
    case SPH_KIND_NIB16:
      if (D == 4) return prefill_fn_mc<SPH_KIND_NIB16, 4>(mc);
      if (D == 5) return prefill_fn_mc<SPH_KIND_NIB16, 5>(mc);
      return prefill_fn_mc<SPH_KIND_NIB16, 6>(mc);
    case SPH_KIND_NIB16Q8: return prefill_fn_mc<SPH_KIND_NIB16Q8, 8>(mc);
    case SPH_KIND_NIB16Q2: return prefill_fn_mc<SPH_KIND_NIB16Q2, 8>(mc);
    case SPH_KIND_CB13: return prefill_fn_mc<SPH_KIND_CB13, 13>(mc);
    case SPH_KIND_CB13Q4: return prefill_fn_mc<SPH_KIND_CB13Q4, 13>(mc);
  }
  return nullptr;
}

template <int KIND>
const void* rowvec_fn_k(int m) {
  if (m <= 1) return (const void*)k_gemm_rowvec<KIND, 1>;
  if (m <= 4) return (const void*)k_gemm_rowvec<KIND, 4>;
  if (m <= 8) return (const void*)k_gemm_rowvec<KIND, 8>;
  if (m <= 16) return (const void*)k_gemm_rowvec<KIND, 16>;
  return (const void*)k_gemm_rowvec<KIND, 32>;
}

const void* rowvec_fn(int kind, int m) {
  return kind == SPH_KIND_V4 ? rowvec_fn_k<SPH_KIND_V4>(m) : rowvec_fn_k<SPH_KIND_V16>(m);
}

int fmt_kind(const sph_weights* w) { return sph_kind_of_fmt(w->fmt.vec_dim, w->fmt.dir_bits, w->fmt.radius_bits); }

const void* unpack_fn(int D, int V) {
  switch (sph_kind_of(D, V)) {
    case SPH_KIND_W2: return D == 7 ? (const void*)k_unpack<SPH_KIND_W2, 7> : (const void*)k_unpack<SPH_KIND_W2, 6>;
    case SPH_KIND_NIB16:
      if (D == 4) return (const void*)k_unpack<SPH_KIND_NIB16, 4>;
      if (D == 5) return (const void*)k_unpack<SPH_KIND_NIB16, 5>;
      return (const void*)k_unpack<SPH_KIND_NIB16, 6>;
    case SPH_KIND_NIB16Q8: return (const void*)k_unpack<SPH_KIND_NIB16Q8, 8>;
    case SPH_KIND_NIB16Q2: return (const void*)k_unpack<SPH_KIND_NIB16Q2, 8>;
    case SPH_KIND_CB13: return (const void*)k_unpack<SPH_KIND_CB13, 13>;
    case SPH_KIND_CB13Q4: return (const void*)k_unpack<SPH_KIND_CB13Q4, 13>;
  }
  return nullptr;
}

std::atomic<int> g_num_cus{0};

int num_cus() {
  int c = g_num_cus.load();
  if (c == 0) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
      c = cus;
    else
      c = 256;
    g_num_cus.store(c);
  }
  return c;
}



// Prefill plan: workgroups of PF_WAVES * PF_TPW tiles by MC batch rows; K is split only while the
// split grid still fits in one round on the CUs (each split adds a pass over fp32 partial outputs).
struct PrefillPlan {
  int gx, gy, ks, mc;
  size_t ws_bytes;
};

PrefillPlan prefill_plan(const sph_weights* w, int64_t m) {
  PrefillPlan P{};
  const int64_t nt = (w->n + 15) / 16, ng = w->k / 128;
  const int mc = prefill_mc(w->fmt.dir_bits, w->fmt.radius_bits, m);
  P.gx = (int)((nt + PF_WAVES * PF_TPW - 1) / (PF_WAVES * PF_TPW));
  P.gy = (int)((m + mc - 1) / mc);
  P.mc = mc;
  const int64_t g = (int64_t)P.gx * P.gy, cus = num_cus();
  // K is split as far as the grid still fits in one round on the CUs (at most 16 ranges, each at
  // least one chunk): a small grid otherwise leaves CUs idle (4096x12288 at 32 batch rows ran on
  // half of them with splits limited to powers of two up to 8, 17-18% slower)
  P.ks = (int)std::max<int64_t>(1, std::min<int64_t>(std::min<int64_t>(cus / g, ng), PF_KS_MAX));
  P.ws_bytes = P.ks > 1 ? (size_t)P.ks * m * nt * 16 * sizeof(float) : 0;
  return P;
}

// m and k of udiv_by for a divisor 1 <= d < 2^31.
void div_magic(int d, uint32_t& m, int& k) {
  int l = 0;
  while ((1ll << l) < d) ++l;
  k = 31 + l;
  m = (uint32_t)(((1ull << k) + (uint64_t)d - 1) / (uint64_t)d);
}

// Work plan. Vector-ALU path: one 16-wave workgroup per CU, every wave a contiguous range of wl
// steps (the last ones shorter or empty). Matrix-core path: a workgroup per tile, its waves
// splitting K.
Launch plan(const sph_weights* w, int m) {
  Launch L{};
  const int64_t nv = w->k / 8, nt = (w->n + 15) / 16;
  const int kind = sph_kind_of(w->fmt.dir_bits, w->fmt.radius_bits);
  const int cus = num_cus();
  // batch 1: vector ALU; 2..8: 4x4x4 MFMA blocks on the same records (4 lanes per vector
  // position); 9..16: 16x16x32 MFMA tiles (lane = row x position group). Every variant forms
  // exact fp16 products. All share the step plan below (16 positions per step for the batched
  // variants, 64 or 32 for batch 1). Larger batches run on the prefill kernel.
  if (m <= 16) {
    // batch 2 on the vector ALUs as well (exact products), except for the codebook kinds, whose
    // two-row kernel would spill
    const int M = m <= 1 ? 1 : (m == 2 && !sph_is_codebook_kind(kind)) ? 2 : m <= 4 ? 4 : m <= 8 ? 8 : 16;
    const int H = M == 1 ? 16 / B1_RPL : M == 2 ? 2 : 4;
    const int vpc = 64 / H;
    const int wpb = VALU_WPB;
    const int64_t nc = (nv + vpc - 1) / vpc;
    const int64_t ts = nt * nc;
    const int64_t slots = (int64_t)cus * VALU_WG_PER_CU;
    // whole tiles per workgroup (no tile split across workgroups, parts meet in LDS) ...
    const int64_t T = (nt + slots - 1) / slots;
    const int64_t gA = (nt + T - 1) / T;
    const int64_t lA = (T * nc + wpb - 1) / wpb;
    // ... or ranges of lB steps across the waves of the grid (tiles split across workgroups meet
    // in the workspace), on at most ts / wpb workgroups
    const int64_t gB = std::max<int64_t>(1, std::min<int64_t>(slots, ts / wpb));
    const int64_t lB = (ts + gB * wpb - 1) / (gB * wpb);
    // whole tiles per workgroup need the parts inside a workgroup to meet in LDS; they are used
    // when their longest wave is no longer than the balanced plan's, whose split tiles cross
    // workgroups and meet through global memory (allowing them one more step, to save that round
    // trip, made the 32B-class step 1.5% slower: 51200x5120 27.4 against 26.7 us)
    const bool aligned = lA <= lB && lds_handover_fits(kind, w->fmt.dir_bits, M, M <= 2 ? 0 : M <= 8 ? 1 : 2);
    L.fn = pick(w->fmt.dir_bits, w->fmt.radius_bits, M);
    L.block = 64 * wpb;
    L.nc = (int)nc;
    L.ts = (int)ts;
    if (aligned) {
      L.grid = (int)gA;
      L.wg_tiles = (int)T;
      L.wgs = (int)(T * nc);
      L.wl = (int)lA;
      L.pmax = 0;
      L.ws_bytes = 0;
    } else {
      // the waves that get a step: ceil(ts / lB) <= gB * wpb
      L.grid = (int)(((ts + lB - 1) / lB + wpb - 1) / wpb);
      L.wg_tiles = 0;
      L.wl = (int)lB;
      // every range but the launch's last holds lB steps, so a tile meets at most nc / lB + 2
      L.pmax = (int)(nc / lB + 2);
      // tagged slots [nt][pmax][M][16], then one arrival counter per tile
      L.cnt_off = ((size_t)nt * L.pmax * M * 16 * 8 + 255) / 256 * 256;
      L.ws_bytes = L.cnt_off + ((size_t)nt * 4 + 255) / 256 * 256;
    }
  }
  return L;
}

// The prefill kernel (and its split-K reduction) for a validated call.
sph_status launch_prefill(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y, int64_t ldy,
                          sph_dtype y_dtype, void* d_ws, size_t ws_bytes, hipStream_t s) {
  const PrefillPlan P = prefill_plan(w, m);
  const void* fn = prefill_fn(w->fmt.dir_bits, w->fmt.radius_bits, P.mc);
  if (!fn) return SPH_ERR_UNSUPPORTED_FORMAT;
  if (P.ws_bytes > 0) {
    if (!d_ws) return SPH_ERR_NULL;
    if (ws_bytes < P.ws_bytes) return SPH_ERR_BUFFER_TOO_SMALL;
    if ((uintptr_t)d_ws % 256 != 0) return SPH_ERR_SHAPE;
  }
  KArgs a = make_args(w);
  a.x = (const uint16_t*)d_x;
  a.ldx = ldx;
  a.y = d_y;
  a.ldy = ldy;
  a.y_f16 = (y_dtype == SPH_F16);
  a.m = (int)m;
  a.ks = P.ks;
  a.ws_part = (float*)d_ws;
  void* kargs[] = {&a};
  if (hipLaunchKernel(fn, dim3(P.gx, P.gy, P.ks), dim3(PF_THREADS), kargs, 0, s) != hipSuccess) return SPH_ERR_HIP;
  if (hipGetLastError() != hipSuccess) return SPH_ERR_HIP;
  if (P.ks > 1) {
    const int64_t total = (int64_t)m * ((w->n + 15) / 16) * 4;   // four rows per thread
    if (hipLaunchKernel((const void*)k_prefill_reduce, dim3((unsigned)((total + 255) / 256)), dim3(256), kargs, 0, s) !=
        hipSuccess)
      return SPH_ERR_HIP;
    if (hipGetLastError() != hipSuccess) return SPH_ERR_HIP;
  }
  return SPH_OK;
}

bool valid_desc(const sph_weights* w) {
  if (!w || w->magic != SPH_MAGIC || w->layout_version != SPH_LAYOUT_VERSION || !w->d_base) return false;
  if (sph_host_check_format(&w->fmt) != SPH_OK || sph_host_check_shape(w->n, w->k) != SPH_OK) return false;
  uint64_t off[8], total = 0;
  if (sph_host_layout(&w->fmt, w->n, w->k, off, &total) != SPH_OK || total > w->bytes) return false;
  for (int i = 0; i < 8; ++i)
    if (off[i] != w->off[i]) return false;
  return true;
}

sph_status launch(const Launch& L, const KArgs& a, hipStream_t s) {
  KArgs args = a;
  void* kargs[] = {&args};
  if (hipLaunchKernel(L.fn, dim3(L.grid), dim3(L.block), kargs, 0, s) != hipSuccess) return SPH_ERR_HIP;
  if (hipGetLastError() != hipSuccess) return SPH_ERR_HIP;
  return SPH_OK;
}

// Argument checks of sph_gemm_small (host only, before any HIP call).
sph_status check_small_args(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, const void* d_y,
                            int64_t ldy, sph_dtype y_dtype) {
  if (!w || !d_x || !d_y) return SPH_ERR_NULL;
  if (!valid_desc(w)) return SPH_ERR_BAD_DESCRIPTOR;
  if (m < 1 || m > 32) return SPH_ERR_SHAPE;
  if (ldx < w->k || ldy < w->n || ldx % 8 != 0) return SPH_ERR_SHAPE;
  if (y_dtype != SPH_F16 && y_dtype != SPH_F32) return SPH_ERR_SHAPE;
  if ((uintptr_t)d_x % 16 != 0 || (uintptr_t)d_y % 4 != 0) return SPH_ERR_SHAPE;
  return SPH_OK;
}

}  // namespace

// ------------------------------------------------------------------------------------------
// Scratch memory of sph_gemm_small_noalloc: a fixed-size device array that takes the place of the
// caller's workspace, for callers that cannot allocate. The loader gives every GPU that runs the
// library its own copy, held until the process ends. Host code never passes the array's name to
// a kernel (on the host it is a stand-in, not a device address): the device address of this GPU's
// copy is looked up once per device and kept.
// ------------------------------------------------------------------------------------------
#define SPH_SCRATCH_BYTES ((size_t)SPH_NOALLOC_SCRATCH_BYTES)
static __device__ __align__(256) unsigned char scratch[SPH_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

__global__ void __launch_bounds__(256) k_zero16(uint4* p, size_t n16) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (size_t)gridDim.x * 256)
    p[i] = make_uint4(0u, 0u, 0u, 0u);
}

// The current device's copy of `scratch`: on the first call on a device, its address (with that
// device current) and one clearing pass on `s` (a kernel, not a memset, so that it may be
// captured into a graph); the calls that use it leave it zero-filled again.
sph_status scratch_of_current_device(hipStream_t s, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return SPH_ERR_HIP;
  void* p = g_scratch[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch[dev].load(std::memory_order_acquire);
    if (!p) {
      void* q = nullptr;
      if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return SPH_ERR_HIP;
      hipLaunchKernelGGL(k_zero16, dim3(1024), dim3(256), 0, s, (uint4*)q, SPH_SCRATCH_BYTES / 16);
      if (hipGetLastError() != hipSuccess) return SPH_ERR_HIP;
      g_scratch[dev].store(q, std::memory_order_release);
      p = q;
    }
  }
  *out = p;
  return SPH_OK;
}

}  // namespace

// ------------------------------------------------------------------------------------------
// C ABI
// ------------------------------------------------------------------------------------------
extern "C" {

const char* sph_status_str(sph_status s) {
  switch (s) {
    case SPH_OK: return "ok";
    case SPH_ERR_NULL: return "null pointer";
    case SPH_ERR_SHAPE: return "bad shape, leading dimension or alignment";
    case SPH_ERR_UNSUPPORTED_FORMAT: return "unsupported format";
    case SPH_ERR_CODE_RANGE: return "code out of range";
    case SPH_ERR_BAD_VALUE: return "bad value (non-finite or negative)";
    case SPH_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case SPH_ERR_HIP: return "HIP runtime error";
    case SPH_ERR_BAD_DESCRIPTOR: return "bad weights descriptor";
  }
  return "unknown status";
}

int sph_format_supported(const sph_format* fmt) { return sph_host_check_format(fmt) == SPH_OK ? 1 : 0; }

sph_status sph_packed_bytes(const sph_format* fmt, int64_t n, int64_t k, size_t* bytes) {
  if (!bytes) return SPH_ERR_NULL;
  uint64_t off[8], total = 0;
  const int st = sph_host_layout(fmt, n, k, off, &total);
  if (st) return (sph_status)st;
  *bytes = (size_t)total;
  return SPH_OK;
}

sph_status sph_pack_weights(const sph_format* fmt, int64_t n, int64_t k, const uint8_t* signs,
                            const uint16_t* dir_idx, const uint8_t* radius_code,
                            const uint16_t* group_min, const uint16_t* group_step,
                            const uint16_t* codebook, void* d_buf, size_t d_buf_bytes, void* stream,
                            sph_weights* out) {
  if (!fmt || !out || !d_buf) return SPH_ERR_NULL;
  uint64_t off[8], total = 0;
  int st = sph_host_layout(fmt, n, k, off, &total);
  if (st) return (sph_status)st;
  st = sph_host_check_codes(fmt, n, k, signs, dir_idx, radius_code, group_min, group_step, codebook);
  if (st) return (sph_status)st;
  if ((uintptr_t)d_buf % 16 != 0) return SPH_ERR_SHAPE;
  if (d_buf_bytes < total) return SPH_ERR_BUFFER_TOO_SMALL;
  std::vector<uint8_t> blob(total, 0);
  sph_host_pack(fmt, n, k, signs, dir_idx, radius_code, group_min, group_step, codebook, off, blob.data());
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(d_buf, blob.data(), total, hipMemcpyHostToDevice, s) != hipSuccess) return SPH_ERR_HIP;
  if (hipStreamSynchronize(s) != hipSuccess) return SPH_ERR_HIP;
  sph_weights w{};
  w.fmt = *fmt;
  w.n = n;
  w.k = k;
  w.d_base = d_buf;
  w.bytes = (size_t)total;
  for (int i = 0; i < 8; ++i) w.off[i] = off[i];
  w.layout_version = SPH_LAYOUT_VERSION;
  w.magic = SPH_MAGIC;
  *out = w;
  return SPH_OK;
}

sph_status sph_workspace_bytes(const sph_weights* w, int64_t m, size_t* bytes) {
  if (!w || !bytes) return SPH_ERR_NULL;
  if (!valid_desc(w)) return SPH_ERR_BAD_DESCRIPTOR;
  if (m < 1 || m > SPH_MAX_BATCH) return SPH_ERR_SHAPE;
  if (sph_is_rowvec_kind(fmt_kind(w))) {
    *bytes = 0;
    return SPH_OK;
  }
  *bytes = small_on_prefill(w, m) ? prefill_plan(w, m).ws_bytes : plan(w, (int)m).ws_bytes;
  return SPH_OK;
}

sph_status sph_gemm(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y, int64_t ldy,
                    sph_dtype y_dtype, void* d_ws, size_t ws_bytes, void* stream) {
  if (!w) return SPH_ERR_NULL;
  if (m >= 1 && m <= 32) return sph_gemm_small(w, d_x, m, ldx, d_y, ldy, y_dtype, d_ws, ws_bytes, stream);
  if (!d_x || !d_y) return SPH_ERR_NULL;
  if (!valid_desc(w)) return SPH_ERR_BAD_DESCRIPTOR;
  if (m < 1 || m > SPH_MAX_BATCH) return SPH_ERR_SHAPE;
  if (ldx < w->k || ldy < w->n || ldx % 8 != 0) return SPH_ERR_SHAPE;
  if (y_dtype != SPH_F16 && y_dtype != SPH_F32) return SPH_ERR_SHAPE;
  if ((uintptr_t)d_x % 16 != 0 || (uintptr_t)d_y % 4 != 0) return SPH_ERR_SHAPE;
  if (sph_is_rowvec_kind(fmt_kind(w))) {
    // the 4-D and 16-D formats run their batch kernel on slices of 32 activation rows
    const size_t esz = y_dtype == SPH_F16 ? 2 : 4;
    for (int64_t b0 = 0; b0 < m; b0 += 32) {
      const sph_status st = sph_gemm_small(w, (const uint16_t*)d_x + b0 * ldx, std::min<int64_t>(32, m - b0), ldx,
                                           (char*)d_y + b0 * ldy * esz, ldy, y_dtype, nullptr, 0, stream);
      if (st != SPH_OK) return st;
    }
    return SPH_OK;
  }
  return launch_prefill(w, d_x, m, ldx, d_y, ldy, y_dtype, d_ws, ws_bytes, (hipStream_t)stream);
}

sph_status sph_gemm_small(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y,
                          int64_t ldy, sph_dtype y_dtype, void* d_ws, size_t ws_bytes, void* stream) {
  const sph_status st = check_small_args(w, d_x, m, ldx, d_y, ldy, y_dtype);
  if (st != SPH_OK) return st;
  if (sph_is_rowvec_kind(fmt_kind(w))) {
    KArgs a = make_args(w);
    a.x = (const uint16_t*)d_x;
    a.ldx = ldx;
    a.y = d_y;
    a.ldy = ldy;
    a.y_f16 = (y_dtype == SPH_F16);
    a.m = (int)m;
    void* kargs[] = {&a};
    if (hipLaunchKernel(rowvec_fn(fmt_kind(w), (int)m), dim3((unsigned)((w->n + RV_WAVES - 1) / RV_WAVES)),
                        dim3(64 * RV_WAVES), kargs, 0, (hipStream_t)stream) != hipSuccess)
      return SPH_ERR_HIP;
    return hipGetLastError() == hipSuccess ? SPH_OK : SPH_ERR_HIP;
  }
  if (small_on_prefill(w, m)) return launch_prefill(w, d_x, m, ldx, d_y, ldy, y_dtype, d_ws, ws_bytes, (hipStream_t)stream);
  const Launch L = plan(w, (int)m);
  if (!L.fn) return SPH_ERR_UNSUPPORTED_FORMAT;
  if (L.ws_bytes > 0) {
    if (!d_ws) return SPH_ERR_NULL;
    if (ws_bytes < L.ws_bytes) return SPH_ERR_BUFFER_TOO_SMALL;
    if ((uintptr_t)d_ws % 256 != 0) return SPH_ERR_SHAPE;
  }
  KArgs a = make_args(w);
  a.nc = L.nc;
  a.wpb = L.block / 64;
  a.nwg = L.grid;
  a.wg_tiles = L.wg_tiles;
  a.wl = L.wl;
  a.wgs = L.wgs;
  div_magic(L.wl, a.wl_m, a.wl_k);
  div_magic(L.wgs > 0 ? L.wgs : 1, a.wgs_m, a.wgs_k);
  a.pmax = L.pmax;
  a.ts = L.ts;
  if (L.ws_bytes > 0) {
    a.ws_slot = (uint64_t*)d_ws;
    a.ws_cnt = (uint32_t*)((char*)d_ws + L.cnt_off);
  }
  a.x = (const uint16_t*)d_x;
  a.ldx = ldx;
  a.y = d_y;
  a.ldy = ldy;
  a.y_f16 = (y_dtype == SPH_F16);
  a.m = (int)m;
  return launch(L, a, (hipStream_t)stream);
}

sph_status sph_gemv(const sph_weights* w, const void* d_x, void* d_y, sph_dtype y_dtype, void* d_ws,
                    size_t ws_bytes, void* stream) {
  if (!w) return SPH_ERR_NULL;
  return sph_gemm_small(w, d_x, 1, w->k, d_y, w->n, y_dtype, d_ws, ws_bytes, stream);
}

sph_status sph_gemm_small_noalloc(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y,
                                  int64_t ldy, sph_dtype y_dtype, void* stream) {
  sph_status st = check_small_args(w, d_x, m, ldx, d_y, ldy, y_dtype);
  if (st != SPH_OK) return st;
  size_t need = 0;
  st = sph_workspace_bytes(w, m, &need);
  if (st != SPH_OK) return st;
  if (need > SPH_SCRATCH_BYTES) return SPH_ERR_BUFFER_TOO_SMALL;
  if (need == 0) return sph_gemm_small(w, d_x, m, ldx, d_y, ldy, y_dtype, nullptr, 0, stream);
  void* ws = nullptr;
  st = scratch_of_current_device((hipStream_t)stream, &ws);
  if (st != SPH_OK) return st;
  return sph_gemm_small(w, d_x, m, ldx, d_y, ldy, y_dtype, ws, need, stream);
}

sph_status sph_unpack(const sph_weights* w, uint8_t* d_signs, uint16_t* d_dir_idx, uint8_t* d_radius_code,
                      void* stream) {
  if (!w || !d_signs || !d_dir_idx || !d_radius_code) return SPH_ERR_NULL;
  if (!valid_desc(w)) return SPH_ERR_BAD_DESCRIPTOR;
  KArgs a = make_args(w);
  const int kind = fmt_kind(w);
  const void* fn = kind == SPH_KIND_V4    ? (const void*)k_unpack_rowvec<SPH_KIND_V4>
                   : kind == SPH_KIND_V16 ? (const void*)k_unpack_rowvec<SPH_KIND_V16>
                                          : unpack_fn(w->fmt.dir_bits, w->fmt.radius_bits);
  if (!fn) return SPH_ERR_UNSUPPORTED_FORMAT;
  if (kind == SPH_KIND_V16 && (uintptr_t)d_signs % 2) return SPH_ERR_SHAPE;
  const int64_t total = sph_is_rowvec_kind(kind) ? (int64_t)a.n * a.nv : (int64_t)a.nt * a.nv * 16;
  const int64_t grid = (total + 255) / 256;
  uint8_t* s = d_signs;
  uint16_t* d = d_dir_idx;
  uint8_t* q = d_radius_code;
  void* kargs[] = {&a, &s, &d, &q};
  if (hipLaunchKernel(fn, dim3((unsigned)grid), dim3(256), kargs, 0, (hipStream_t)stream) != hipSuccess)
    return SPH_ERR_HIP;
  if (hipGetLastError() != hipSuccess) return SPH_ERR_HIP;
  return SPH_OK;
}

}  // extern "C"
