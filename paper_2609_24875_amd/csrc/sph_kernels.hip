// SPHQuant decode-and-multiply on gfx950 (MI355X): kernels and the C ABI of include/sph.h.
//
// The computation is the fused dequantise-and-multiply of Sec. 3.4 / App. D: every 8-D weight
// vector is rebuilt in registers as r^ * s (.) c_z (Eq. 4) with r^ = min_G + q * step_G (Eq. 7)
// and multiplied with fp16 activations, accumulating in fp32; nothing dequantised is written to
// memory. The mapping to the hardware is this library's own:
//  - device layout: 16-row tiles, one "record" per (tile, vector position) (sph_layout.h);
//  - vector-ALU path (batch 1..8): a lane owns one vector position of a tile and decodes up to
//    16 rows of it from 16-byte loads; signs are folded into two nibble-indexed lookup tables in
//    LDS, so the signed direction costs two 8-byte LDS reads and no sign arithmetic; products
//    use v_dot2_f32_f16 (exact fp16 products, fp32 sums); the waves of a workgroup split K and
//    meet in LDS, so the reduction order is fixed and results are bitwise reproducible;
//  - matrix-core path (batch 9..32): each lane decodes one (row, vector) into the A operand of
//    v_mfma_f32_16x16x32_f16 (weights rounded once to fp16), activations form the B operand.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstring>
#include <mutex>
#include <vector>

#include "sph_host.h"
#include "sph_layout.h"

typedef _Float16 f16;
typedef f16 f16x2 __attribute__((ext_vector_type(2)));
typedef f16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

struct KArgs {
  const uint32_t* A;
  const uint32_t* B;
  const uint32_t* P;
  const uint4* T;
  uint32_t t_bytes;   // bytes of lookup tables staged into LDS
  const uint16_t* x;
  int64_t ldx;
  void* y;
  int64_t ldy;
  int y_f16;
  int n, nt, nv, ng, m;
  int wpt;            // waves per tile
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
    const uint32_t f = odd ? ((d >> 14) & 0x3FFFu) : (d & 0x3FFFu);
    lo = f & IM;
    hi = f >> 4;
    q = odd ? qx : (d >> 28);
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
  constexpr uint32_t THI = (16u << D) * 8u;
  const uint2 a = *(const uint2*)(lds + lo * 8u);
  const uint2 b = *(const uint2*)(lds + THI + hi * 8u);
  return make_uint4(a.x, a.y, b.x, b.y);
}

__device__ __forceinline__ uint4 signed_dir_cb13(const unsigned char* lds, uint32_t mask_off, uint32_t s,
                                                 uint32_t z) {
  const uint4 c = *(const uint4*)(lds + z * 16u);
  const uint2 ml = *(const uint2*)(lds + mask_off + (s & 15u) * 8u);
  const uint2 mh = *(const uint2*)(lds + mask_off + (s >> 4) * 8u);
  return make_uint4(c.x ^ ml.x, c.y ^ ml.y, c.z ^ mh.x, c.w ^ mh.y);
}

__device__ __forceinline__ float f16lo(uint32_t u) { return (float)__builtin_bit_cast(f16, (uint16_t)(u & 0xFFFFu)); }
__device__ __forceinline__ float f16hi(uint32_t u) { return (float)__builtin_bit_cast(f16, (uint16_t)(u >> 16)); }
__device__ __forceinline__ f16x2 as_h2(uint32_t u) { return __builtin_bit_cast(f16x2, u); }

__device__ __forceinline__ float dot8(uint4 t, uint4 x) {
  float p = __builtin_amdgcn_fdot2(as_h2(t.x), as_h2(x.x), 0.0f, false);
  p = __builtin_amdgcn_fdot2(as_h2(t.y), as_h2(x.y), p, false);
  p = __builtin_amdgcn_fdot2(as_h2(t.z), as_h2(x.z), p, false);
  return __builtin_amdgcn_fdot2(as_h2(t.w), as_h2(x.w), p, false);
}

// Stage the lookup tables (and for the codebook kind the 16-entry sign-mask table, placed right
// after the codebook at LDS offset a.t_bytes) into LDS. Returns the first free LDS offset,
// rounded up to 16 bytes.
template <int KIND>
__device__ __forceinline__ uint32_t stage_tables(unsigned char* lds, const KArgs& a) {
  uint4* dst = (uint4*)lds;
  const uint32_t n16 = a.t_bytes / 16u;
  for (uint32_t i = threadIdx.x; i < n16; i += blockDim.x) dst[i] = a.T[i];
  uint32_t end = a.t_bytes;
  if constexpr (KIND == SPH_KIND_CB13) {
    // mask[s] flips the fp16 sign bit of element j (of 4) where bit j of the nibble s is set.
    if (threadIdx.x < 16) {
      const uint32_t s = threadIdx.x;
      uint2 m;
      m.x = ((s & 1u) << 15) | ((s & 2u) << 30);
      m.y = ((s & 4u) << 13) | ((s & 8u) << 28);
      *(uint2*)(lds + end + s * 8u) = m;
    }
    end += 128;
  }
  return (end + 15u) & ~15u;
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

// Reduce-scatter of CNT values across the lanes that differ in bits DMIN..32 of the lane id:
// after it, every lane holds CNT >> steps sums (flattened indices base .. base+CNT'-1) and the
// steps left once a single value remains are plain butterfly all-reductions.
template <int CNT, int DIST, int DMIN>
__device__ __forceinline__ void reduce_scatter(float* v, int lane, int& base) {
  if constexpr (DIST >= DMIN) {
    if constexpr (CNT > 1) {
      constexpr int HALF = CNT / 2;
      const bool bit = (lane & DIST) != 0;
#pragma unroll
      for (int i = 0; i < HALF; ++i) {
        const float send = bit ? v[i] : v[i + HALF];
        const float keep = bit ? v[i + HALF] : v[i];
        v[i] = keep + __shfl_xor(send, DIST);
      }
      if (bit) base += HALF;
      reduce_scatter<HALF, DIST / 2, DMIN>(v, lane, base);
    } else {
      v[0] += __shfl_xor(v[0], DIST);
      reduce_scatter<1, DIST / 2, DMIN>(v, lane, base);
    }
  }
}

__host__ __device__ constexpr int ilog2c(int x) { return x <= 1 ? 0 : 1 + ilog2c(x / 2); }

__device__ __forceinline__ void store_y(const KArgs& a, int b, int row, float v) {
  if (a.y_f16) ((f16*)a.y)[(int64_t)b * a.ldy + row] = (f16)v;
  else ((float*)a.y)[(int64_t)b * a.ldy + row] = v;
}

// ------------------------------------------------------------------------------------------
// Vector-ALU kernel: batch M (1, 2, 4 or 8), RPL rows of a record per lane.
// ------------------------------------------------------------------------------------------
template <int KIND, int D, int M, int RPL>
__global__ void __launch_bounds__(1024) k_gemm_valu(KArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  constexpr int H = 16 / RPL;                                          // lanes per record
  constexpr int ADW = (KIND == SPH_KIND_CB13) ? RPL / 4 : RPL / 2;     // A dwords per lane
  constexpr int BDW = (KIND == SPH_KIND_NIB16Q8) ? RPL / 4 : (KIND == SPH_KIND_CB13) ? RPL / 2 : 1;
  constexpr int ADW_REC = (KIND == SPH_KIND_CB13) ? 4 : 8;
  constexpr int BDW_REC = (KIND == SPH_KIND_W2) ? 1 : (KIND == SPH_KIND_NIB16Q8) ? 4 : 8;
  constexpr int NVAL = M * RPL;

  const uint32_t mask_off = a.t_bytes;
  const uint32_t red_off = stage_tables<KIND>(lds, a);
  float* red = (float*)(lds + red_off);
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, W = a.wpt;
  const int h = lane % H, vloc = lane / H;
  const int vstep = (64 / H) * W;

  for (int t = blockIdx.x; t < a.nt; t += gridDim.x) {
    float acc[M][RPL];
#pragma unroll
    for (int b = 0; b < M; ++b)
#pragma unroll
      for (int r = 0; r < RPL; ++r) acc[b][r] = 0.0f;

    for (int v = wave * (64 / H) + vloc; v < a.nv; v += vstep) {
      const int64_t rec = (int64_t)t * a.nv + v;
      uint32_t ra[ADW], rb[BDW];
      load_dw<ADW>(ra, a.A + rec * ADW_REC + h * ADW);
      if constexpr (KIND == SPH_KIND_W2) rb[0] = a.B[rec];
      else if constexpr (KIND != SPH_KIND_NIB16) load_dw<BDW>(rb, a.B + rec * BDW_REC + h * BDW);
      uint32_t pp[RPL];
      load_dw<RPL>(pp, a.P + ((int64_t)t * a.ng + (v >> 4)) * 16 + h * RPL);
      uint4 xv[M];
#pragma unroll
      for (int b = 0; b < M; ++b) {
        if (M == 1 || b < a.m) xv[b] = *(const uint4*)(a.x + (int64_t)b * a.ldx + 8 * (int64_t)v);
        else xv[b] = make_uint4(0, 0, 0, 0);
      }
      uint32_t qodd = 0;
      if constexpr (KIND == SPH_KIND_W2) qodd = rb[0] >> (4 * (h * RPL / 2));
#pragma unroll
      for (int r = 0; r < RPL; ++r) {
        uint4 tt;
        uint32_t q;
        if constexpr (KIND == SPH_KIND_CB13) {
          uint32_t s, z;
          decode_cb13(ra[r / 4], r % 4, rb[r / 2], r & 1, s, z, q);
          tt = signed_dir_cb13(lds, mask_off, s, z);
        } else {
          uint32_t lo, hi, qx = 0;
          if constexpr (KIND == SPH_KIND_W2) qx = (qodd >> (4 * (r / 2))) & 15u;
          if constexpr (KIND == SPH_KIND_NIB16Q8) qx = (rb[r / 4] >> (8 * (r % 4))) & 0xFFu;
          decode_nib<KIND, D>(ra[r / 2], r & 1, qx, lo, hi, q);
          tt = signed_dir_nib<KIND, D>(lds, lo, hi);
        }
        const float rh = fmaf((float)q, f16hi(pp[r]), f16lo(pp[r]));
#pragma unroll
        for (int b = 0; b < M; ++b) acc[b][r] = fmaf(rh, dot8(tt, xv[b]), acc[b][r]);
      }
    }

    // Wave reduction over the lanes that share h, then across waves in LDS (fixed order).
    float vals[NVAL];
#pragma unroll
    for (int b = 0; b < M; ++b)
#pragma unroll
      for (int r = 0; r < RPL; ++r) vals[b * RPL + r] = acc[b][r];
    int base = 0;
    reduce_scatter<NVAL, 32, H>(vals, lane, base);
    constexpr int STEPS = ilog2c(64 / H), LV = ilog2c(NVAL);
    constexpr int LEFT = (LV < STEPS) ? (NVAL >> LV) : (NVAL >> STEPS);
    bool writer = true;
    if constexpr (LV < STEPS) {
      // bits of the all-reduced distances (32 >> LV down to H) must be zero
      constexpr int hi_dist = 32 >> LV;
      constexpr int mask = (2 * hi_dist - 1) & ~(H - 1);
      writer = (lane & mask) == 0;
    }
    if (writer) {
#pragma unroll
      for (int i = 0; i < LEFT; ++i) {
        const int f = base + i;
        const int b = f / RPL, r = f % RPL;
        red[(wave * M + b) * 16 + h * RPL + r] = vals[i];
      }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < M * 16; i += blockDim.x) {
      const int b = i / 16, row = i % 16;
      float s = 0.0f;
      for (int w = 0; w < W; ++w) s += red[(w * M + b) * 16 + row];
      const int grow = t * 16 + row;
      if (b < a.m && grow < a.n) store_y(a, b, grow, s);
    }
    __syncthreads();
  }
}

// ------------------------------------------------------------------------------------------
// Matrix-core kernel: batch up to 16*NB; weights rounded once to fp16, fp32 accumulation.
// ------------------------------------------------------------------------------------------

// Decode row r of record `rec` and return its signed direction (4 half2) and radius level.
template <int KIND, int D>
__device__ __forceinline__ uint4 decode_row(const unsigned char* lds, uint32_t mask_off, const KArgs& a,
                                            int64_t rec, int r, uint32_t& q) {
  if constexpr (KIND == SPH_KIND_CB13) {
    const uint32_t sdw = a.A[rec * 4 + (r >> 2)];
    const uint32_t zdw = a.B[rec * 8 + (r >> 1)];
    uint32_t s, z;
    decode_cb13(sdw, r & 3, zdw, r & 1, s, z, q);
    return signed_dir_cb13(lds, mask_off, s, z);
  } else {
    const uint32_t d = a.A[rec * 8 + (r >> 1)];
    uint32_t qx = 0;
    if constexpr (KIND == SPH_KIND_W2) qx = (a.B[rec] >> (4 * (r >> 1))) & 15u;
    if constexpr (KIND == SPH_KIND_NIB16Q8) qx = (a.B[rec * 4 + (r >> 2)] >> (8 * (r & 3))) & 0xFFu;
    uint32_t lo, hi;
    decode_nib<KIND, D>(d, r & 1, qx, lo, hi, q);
    return signed_dir_nib<KIND, D>(lds, lo, hi);
  }
}

__device__ __forceinline__ uint32_t scale_pack(uint32_t t, float rh) {
  const f16 lo = (f16)(rh * f16lo(t));
  const f16 hi = (f16)(rh * f16hi(t));
  return (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
}

template <int KIND, int D, int NB>
__global__ void __launch_bounds__(1024) k_gemm_mfma(KArgs a) {
  extern __shared__ __align__(16) unsigned char lds[];
  const uint32_t mask_off = a.t_bytes;
  const uint32_t red_off = stage_tables<KIND>(lds, a);
  float* red = (float*)(lds + red_off);
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, W = a.wpt;
  const int r = lane & 15, j = lane >> 4;

  for (int t = blockIdx.x; t < a.nt; t += gridDim.x) {
    f32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};

    for (int vb = 4 * wave; vb < a.nv; vb += 4 * W) {
      const int v = vb + j;
      const int64_t rec = (int64_t)t * a.nv + v;
      uint32_t q;
      const uint4 tt = decode_row<KIND, D>(lds, mask_off, a, rec, r, q);
      const uint32_t pr = a.P[((int64_t)t * a.ng + (v >> 4)) * 16 + r];
      const float rh = fmaf((float)q, f16hi(pr), f16lo(pr));
      uint4 wq;
      wq.x = scale_pack(tt.x, rh);
      wq.y = scale_pack(tt.y, rh);
      wq.z = scale_pack(tt.z, rh);
      wq.w = scale_pack(tt.w, rh);
      const f16x8 wa = __builtin_bit_cast(f16x8, wq);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int b = nb * 16 + r;
        uint4 xq = make_uint4(0, 0, 0, 0);
        if (b < a.m) xq = *(const uint4*)(a.x + (int64_t)b * a.ldx + 8 * (int64_t)v);
        acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(wa, __builtin_bit_cast(f16x8, xq), acc[nb], 0, 0, 0);
      }
    }
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int e = 0; e < 4; ++e) red[((wave * NB + nb) * 64 + lane) * 4 + e] = acc[nb][e];
    __syncthreads();
    for (int i = threadIdx.x; i < NB * 256; i += blockDim.x) {
      const int nb = i / 256, l = (i / 4) % 64, e = i % 4;
      float s = 0.0f;
      for (int w = 0; w < W; ++w) s += red[((w * NB + nb) * 64 + l) * 4 + e];
      const int row = 4 * (l >> 4) + e, b = nb * 16 + (l & 15);
      const int grow = t * 16 + row;
      if (b < a.m && grow < a.n) store_y(a, b, grow, s);
    }
    __syncthreads();
  }
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
  if constexpr (KIND == SPH_KIND_CB13) {
    decode_cb13(a.A[rec * 4 + (r >> 2)], r & 3, a.B[rec * 8 + (r >> 1)], r & 1, s, z, q);
  } else {
    const uint32_t d = a.A[rec * 8 + (r >> 1)];
    uint32_t qx = 0;
    if constexpr (KIND == SPH_KIND_W2) qx = (a.B[rec] >> (4 * (r >> 1))) & 15u;
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
// Host dispatch
// ------------------------------------------------------------------------------------------
namespace {

struct Launch {
  const void* fn;
  int wpt;
  int grid;
  uint32_t lds;
};

KArgs make_args(const sph_weights* w) {
  KArgs a{};
  const int kind = sph_kind_of(w->fmt.dir_bits, w->fmt.radius_bits);
  const char* base = (const char*)w->d_base;
  a.A = (const uint32_t*)(base + w->off[SPH_OFF_A]);
  a.B = (const uint32_t*)(base + w->off[SPH_OFF_B]);
  a.P = (const uint32_t*)(base + w->off[SPH_OFF_PARAMS]);
  a.T = (const uint4*)(base + w->off[SPH_OFF_TABLES]);
  a.t_bytes = (uint32_t)sph_table_bytes(kind, w->fmt.dir_bits);
  a.n = (int)w->n;
  a.nt = (int)((w->n + 15) / 16);
  a.nv = (int)(w->k / 8);
  a.ng = (int)(w->k / 128);
  return a;
}

template <int KIND, int D>
const void* valu_fn(int M) {
  switch (M) {
    case 1: return (const void*)k_gemm_valu<KIND, D, 1, 16>;
    case 2: return (const void*)k_gemm_valu<KIND, D, 2, 16>;
    case 4: return (const void*)k_gemm_valu<KIND, D, 4, 8>;
    default: return (const void*)k_gemm_valu<KIND, D, 8, 4>;
  }
}

template <int KIND, int D>
const void* mfma_fn(int NB) {
  return NB == 1 ? (const void*)k_gemm_mfma<KIND, D, 1> : (const void*)k_gemm_mfma<KIND, D, 2>;
}

const void* pick(int D, int V, bool mfma, int sel) {
  const int kind = sph_kind_of(D, V);
  switch (kind) {
    case SPH_KIND_W2: return mfma ? mfma_fn<SPH_KIND_W2, 6>(sel) : valu_fn<SPH_KIND_W2, 6>(sel);
    case SPH_KIND_NIB16:
      if (D == 4) return mfma ? mfma_fn<SPH_KIND_NIB16, 4>(sel) : valu_fn<SPH_KIND_NIB16, 4>(sel);
      if (D == 5) return mfma ? mfma_fn<SPH_KIND_NIB16, 5>(sel) : valu_fn<SPH_KIND_NIB16, 5>(sel);
      return mfma ? mfma_fn<SPH_KIND_NIB16, 6>(sel) : valu_fn<SPH_KIND_NIB16, 6>(sel);
    case SPH_KIND_NIB16Q8: return mfma ? mfma_fn<SPH_KIND_NIB16Q8, 8>(sel) : valu_fn<SPH_KIND_NIB16Q8, 8>(sel);
    case SPH_KIND_CB13: return mfma ? mfma_fn<SPH_KIND_CB13, 13>(sel) : valu_fn<SPH_KIND_CB13, 13>(sel);
  }
  return nullptr;
}

const void* unpack_fn(int D, int V) {
  switch (sph_kind_of(D, V)) {
    case SPH_KIND_W2: return (const void*)k_unpack<SPH_KIND_W2, 6>;
    case SPH_KIND_NIB16:
      if (D == 4) return (const void*)k_unpack<SPH_KIND_NIB16, 4>;
      if (D == 5) return (const void*)k_unpack<SPH_KIND_NIB16, 5>;
      return (const void*)k_unpack<SPH_KIND_NIB16, 6>;
    case SPH_KIND_NIB16Q8: return (const void*)k_unpack<SPH_KIND_NIB16Q8, 8>;
    case SPH_KIND_CB13: return (const void*)k_unpack<SPH_KIND_CB13, 13>;
  }
  return nullptr;
}

int g_num_cus = 0;

int num_cus() {
  if (g_num_cus == 0) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
      g_num_cus = cus;
    else
      g_num_cus = 256;
  }
  return g_num_cus;
}

uint32_t lds_tables(const sph_weights* w) {
  const int kind = sph_kind_of(w->fmt.dir_bits, w->fmt.radius_bits);
  uint32_t b = (uint32_t)sph_table_bytes(kind, w->fmt.dir_bits);
  if (kind == SPH_KIND_CB13) b += 128;
  return (b + 15u) & ~15u;
}

// Waves per tile: enough vector positions per lane to amortise the reduction, at most 16.
Launch plan(const sph_weights* w, int m) {
  Launch L{};
  const int64_t nv = w->k / 8, nt = (w->n + 15) / 16;
  const bool mfma = m > 8;
  const int kind = sph_kind_of(w->fmt.dir_bits, w->fmt.radius_bits);
  int wpt;
  if (!mfma) {
    const int M = m <= 1 ? 1 : m <= 2 ? 2 : m <= 4 ? 4 : 8;
    const int H = M <= 2 ? 1 : M == 4 ? 2 : 4;
    const int64_t per_wave = (64 / H) * 4;      // ~4 records per lane
    wpt = (int)((nv + per_wave - 1) / per_wave);
    wpt = wpt < 1 ? 1 : wpt > 16 ? 16 : wpt;
    L.fn = pick(w->fmt.dir_bits, w->fmt.radius_bits, false, M);
    L.lds = lds_tables(w) + (uint32_t)(wpt * M * 16 * 4);
  } else {
    const int NB = m <= 16 ? 1 : 2;
    const int64_t per_wave = 4 * 8;             // 8 MFMA steps per wave
    wpt = (int)((nv + per_wave - 1) / per_wave);
    const int wmax = (kind == SPH_KIND_CB13) ? 8 : 16;
    wpt = wpt < 1 ? 1 : wpt > wmax ? wmax : wpt;
    L.fn = pick(w->fmt.dir_bits, w->fmt.radius_bits, true, NB);
    L.lds = lds_tables(w) + (uint32_t)(wpt * NB * 64 * 4 * 4);
  }
  L.wpt = wpt;
  const int64_t cap = (int64_t)num_cus() * 4;
  L.grid = (int)(nt < cap ? nt : cap);
  return L;
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

std::mutex g_attr_mu;
std::vector<const void*> g_attr_set;

// Kernels whose LDS exceeds the default 64 KiB get the gfx950 maximum, once per function.
bool allow_big_lds(const void* fn) {
  std::lock_guard<std::mutex> lk(g_attr_mu);
  for (const void* f : g_attr_set)
    if (f == fn) return true;
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024) != hipSuccess) return false;
  g_attr_set.push_back(fn);
  return true;
}

sph_status launch(const Launch& L, const KArgs& a, hipStream_t s) {
  if (L.lds > 160 * 1024) return SPH_ERR_HIP;
  if (L.lds > 64 * 1024 && !allow_big_lds(L.fn)) return SPH_ERR_HIP;
  KArgs args = a;
  void* kargs[] = {&args};
  if (hipLaunchKernel(L.fn, dim3(L.grid), dim3(64 * L.wpt), kargs, L.lds, s) != hipSuccess) return SPH_ERR_HIP;
  if (hipGetLastError() != hipSuccess) return SPH_ERR_HIP;
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
  if (m < 1 || m > 32) return SPH_ERR_SHAPE;
  *bytes = 0;
  return SPH_OK;
}

sph_status sph_gemm_small(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y,
                          int64_t ldy, sph_dtype y_dtype, void* d_ws, size_t ws_bytes, void* stream) {
  (void)d_ws;
  (void)ws_bytes;
  if (!w || !d_x || !d_y) return SPH_ERR_NULL;
  if (!valid_desc(w)) return SPH_ERR_BAD_DESCRIPTOR;
  if (m < 1 || m > 32) return SPH_ERR_SHAPE;
  if (ldx < w->k || ldy < w->n || ldx % 8 != 0) return SPH_ERR_SHAPE;
  if (y_dtype != SPH_F16 && y_dtype != SPH_F32) return SPH_ERR_SHAPE;
  if ((uintptr_t)d_x % 16 != 0 || (uintptr_t)d_y % 4 != 0) return SPH_ERR_SHAPE;
  const Launch L = plan(w, (int)m);
  if (!L.fn) return SPH_ERR_UNSUPPORTED_FORMAT;
  KArgs a = make_args(w);
  a.x = (const uint16_t*)d_x;
  a.ldx = ldx;
  a.y = d_y;
  a.ldy = ldy;
  a.y_f16 = (y_dtype == SPH_F16);
  a.m = (int)m;
  a.wpt = L.wpt;
  return launch(L, a, (hipStream_t)stream);
}

sph_status sph_gemv(const sph_weights* w, const void* d_x, void* d_y, sph_dtype y_dtype, void* d_ws,
                    size_t ws_bytes, void* stream) {
  if (!w) return SPH_ERR_NULL;
  return sph_gemm_small(w, d_x, 1, w->k, d_y, w->n, y_dtype, d_ws, ws_bytes, stream);
}

sph_status sph_unpack(const sph_weights* w, uint8_t* d_signs, uint16_t* d_dir_idx, uint8_t* d_radius_code,
                      void* stream) {
  if (!w || !d_signs || !d_dir_idx || !d_radius_code) return SPH_ERR_NULL;
  if (!valid_desc(w)) return SPH_ERR_BAD_DESCRIPTOR;
  KArgs a = make_args(w);
  const void* fn = unpack_fn(w->fmt.dir_bits, w->fmt.radius_bits);
  if (!fn) return SPH_ERR_UNSUPPORTED_FORMAT;
  const int64_t total = (int64_t)a.nt * a.nv * 16;
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
