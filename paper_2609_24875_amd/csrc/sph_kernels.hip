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
//    use v_dot2_f32_f16 (exact fp16 products, fp32 sums); persistent waves walk balanced
//    (tile, K-segment) items and split-K partial sums are added in a fixed order, so results
//    are bitwise reproducible;
//  - matrix-core path (batch 9..32): each lane decodes one (row, vector) into the A operand of
//    v_mfma_f32_16x16x32_f16 (weights rounded once to fp16), activations form the B operand.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>
#include <cstring>
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
  int wpt;            // waves per tile (matrix-core kernel)
  // vector-ALU work plan: items = nt * S, each `cps` chunks of one tile
  int nc, cps, S, items;
  int wpb, gw;        // waves per workgroup, waves in the grid
  uint64_t* ws_slot;  // [nt][S][M][16] tagged partial sums (S > 1), flags zero between calls
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

__device__ __forceinline__ void store_y(const KArgs& a, int b, int row, float v) {
  if (a.y_f16) ((f16*)a.y)[(int64_t)b * a.ldy + row] = (f16)v;
  else ((float*)a.y)[(int64_t)b * a.ldy + row] = v;
}

// ------------------------------------------------------------------------------------------
// Vector-ALU kernel: batch M (1, 2, 4 or 8), RPL rows of a record per lane.
//
// Persistent waves walk a balanced list of work items. An item is one tile (16 rows) and a
// segment of `cps` consecutive chunks of its vector positions; a chunk is 64/H positions, one
// per lane group. The next record's loads are issued before the current record is computed.
// An item's partial sums go straight to y when the tile has a single segment; otherwise they
// are written to tagged workspace slots, and the wave that ran the tile's first segment adds
// the segments in a fixed order once its own items are done, so results do not depend on
// scheduling and no wave ever waits while it still owes partial sums to others.
// ------------------------------------------------------------------------------------------
template <int KIND, int D>
struct Tables {
  static constexpr uint32_t bytes = (KIND == SPH_KIND_CB13) ? ((16u << D) + 128u) : (256u << D);
};

template <int KIND, int M, int RPL>
struct Rec {
  static constexpr int ADW = (KIND == SPH_KIND_CB13) ? RPL / 4 : RPL / 2;
  static constexpr int BDW = (KIND == SPH_KIND_NIB16Q8) ? RPL / 4 : (KIND == SPH_KIND_CB13) ? RPL / 2 : 1;
  uint32_t ra[ADW];
  uint32_t rb[BDW];
  uint32_t pw;        // one group-parameter word of the chunk, staged through LDS at compute time
  uint4 xv[M];
  bool ok;            // vector position inside the row; else x is taken as 0
};

// Loads of one step. Branch-free so that the compiler can count outstanding loads across the
// software pipeline: positions past the end of the row read a valid record and contribute
// through x = 0. The chunk's group parameters (VPC/16 groups x 16 rows = VPC words, contiguous)
// are spread one word per lane.
template <int KIND, int M, int RPL>
__device__ __forceinline__ void load_rec(Rec<KIND, M, RPL>& R, const KArgs& a, int t, int c, int h, int vloc,
                                         int lane) {
  constexpr int H = 16 / RPL, VPC = 64 / H;
  constexpr int ADW_REC = (KIND == SPH_KIND_CB13) ? 4 : 8;
  constexpr int BDW_REC = (KIND == SPH_KIND_W2) ? 1 : (KIND == SPH_KIND_NIB16Q8) ? 4 : 8;
  constexpr int ADW = Rec<KIND, M, RPL>::ADW, BDW = Rec<KIND, M, RPL>::BDW;
  const int v0 = c * VPC + vloc;
  const bool ok = v0 < a.nv;
  const int v = ok ? v0 : a.nv - 1;
  const int64_t rec = (int64_t)t * a.nv + v;
  load_dw<ADW>(R.ra, a.A + rec * ADW_REC + h * ADW);
  if constexpr (KIND == SPH_KIND_W2) R.rb[0] = a.B[rec];
  else if constexpr (KIND != SPH_KIND_NIB16) load_dw<BDW>(R.rb, a.B + rec * BDW_REC + h * BDW);
  // parameter word `lane` of the chunk: group c*VPC/16 + lane/16, row lane%16 (clamped to the row)
  const int pg = min(c * (VPC / 16) + (lane & (VPC - 1)) / 16, a.ng - 1);
  R.pw = a.P[((int64_t)t * a.ng + pg) * 16 + (lane & 15)];
#pragma unroll
  for (int b = 0; b < M; ++b) {
    const int bb = (M == 1 || b < a.m) ? b : 0;
    R.xv[b] = *(const uint4*)(a.x + (int64_t)bb * a.ldx + 8 * (int64_t)v);
  }
  R.ok = ok;
}

// Rows of the record in batches of RB: all table lookups of a batch are issued before any
// of its arithmetic, so one LDS round trip serves RB rows.
template <int KIND, int D, int M, int RPL>
__device__ __forceinline__ void compute_rec(const Rec<KIND, M, RPL>& R, float (&acc)[M][RPL],
                                            const unsigned char* lds, uint32_t mask_off, uint32_t* pstage,
                                            int lane, int h, int vloc, int m) {
  constexpr int RB = RPL < 4 ? RPL : 4;
  // group parameters: stage the chunk's words in this wave's LDS slot, read back this lane's rows
  pstage[lane] = R.pw;
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
  uint4 xv[M];
#pragma unroll
  for (int b = 0; b < M; ++b) {
    const bool use = R.ok && (M == 1 || b < m);
    xv[b] = use ? R.xv[b] : make_uint4(0, 0, 0, 0);
  }
  uint32_t qodd = 0;
  if constexpr (KIND == SPH_KIND_W2) qodd = R.rb[0] >> (4 * (h * RPL / 2));
#pragma unroll
  for (int r0 = 0; r0 < RPL; r0 += RB) {
    uint4 tt[RB];
    float qf[RB];
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int r = r0 + i;
      uint32_t q;
      if constexpr (KIND == SPH_KIND_CB13) {
        uint32_t s, z;
        decode_cb13(R.ra[r / 4], r % 4, R.rb[r / 2], r & 1, s, z, q);
        tt[i] = signed_dir_cb13(lds, mask_off, s, z);
      } else {
        uint32_t lo, hi, qx = 0;
        if constexpr (KIND == SPH_KIND_W2) qx = (qodd >> (4 * (r / 2))) & 15u;
        if constexpr (KIND == SPH_KIND_NIB16Q8) qx = (R.rb[r / 4] >> (8 * (r % 4))) & 0xFFu;
        decode_nib<KIND, D>(R.ra[r / 2], r & 1, qx, lo, hi, q);
        tt[i] = signed_dir_nib<KIND, D>(lds, lo, hi);
      }
      qf[i] = (float)q;
    }
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      const int r = r0 + i;
      const float rh = fmaf(qf[i], f16hi(pp[r]), f16lo(pp[r]));
#pragma unroll
      for (int b = 0; b < M; ++b) acc[b][r] = fmaf(rh, dot8(tt[i], xv[b]), acc[b][r]);
    }
  }
}

// Exchange-and-add across lanes l and l^DIST: lanes with bit DIST clear end with
// lo_keep[l] + lo_keep[l^DIST], the others with hi_keep[l] + hi_keep[l^DIST]. (The gfx950
// permlane-swap builtins would do this in one instruction, but this compiler version folds the
// sum of their two results into twice one of them, so they are not used.)
template <int DIST>
__device__ __forceinline__ float xchg_add(float lo_keep, float hi_keep, int lane) {
  const bool bit = (lane & DIST) != 0;
  const float send = bit ? lo_keep : hi_keep;
  const float keep = bit ? hi_keep : lo_keep;
  return keep + __shfl_xor(send, DIST);
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

// Split-K slots: one 64-bit word per (tile, segment, batch row, tile row) holding the fp32
// partial sum in the low half and a valid flag in the high half, written and read with
// device-coherent (agent-scope) atomics so that a single load sees value and flag together.
__device__ __forceinline__ void slot_store(uint64_t* p, float v) {
  __hip_atomic_store(p, (uint64_t)__builtin_bit_cast(uint32_t, v) | (1ull << 32), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}

// Emit a finished item: straight to y when its tile has a single segment, else as partial sums
// in the tile's slots (the tile's reducer adds them at the end of its own work).
template <int M, int RPL>
__device__ __forceinline__ void emit_item(const KArgs& a, float (&acc)[M][RPL], int t, int s, int lane, int h) {
  constexpr int H = 16 / RPL;
  constexpr int NVAL = M * RPL, N4 = NVAL / 4;
  float vals[NVAL];
#pragma unroll
  for (int b = 0; b < M; ++b)
#pragma unroll
    for (int r = 0; r < RPL; ++r) {
      vals[b * RPL + r] = acc[b][r];
      acc[b][r] = 0.0f;
    }
  wave_reduce<NVAL, H>(vals, lane);
  const int base = ((lane >> 5) & 1) * (NVAL / 2) + ((lane >> 4) & 1) * N4;
  if ((lane & 15) >= H) return;              // one writer lane per h in each 16-lane row
  if (a.S == 1) {
#pragma unroll
    for (int i = 0; i < N4; ++i) {
      const int f = base + i, b = f / RPL, row = h * RPL + f % RPL;
      const int grow = t * 16 + row;
      if (b < a.m && grow < a.n) store_y(a, b, grow, vals[i]);
    }
  } else {
    uint64_t* slot = a.ws_slot + ((int64_t)t * a.S + s) * (M * 16);
#pragma unroll
    for (int i = 0; i < N4; ++i) {
      const int f = base + i, b = f / RPL, row = h * RPL + f % RPL;
      slot_store(slot + b * 16 + row, vals[i]);
    }
  }
}

// Reducer of tile t: wait for every segment's slot to be valid (the segments are written by
// waves that never wait before finishing their own items), add the segments in order, clear the
// slots for the next call, write y. The wait is bounded by a deadline on the constant 100 MHz
// real-time counter (about 50 ms, thousands of times a whole launch); a wait that runs out (not
// expected) writes NaN rather than hanging.
template <int M>
__device__ __forceinline__ void reduce_tile(const KArgs& a, int t, int lane) {
  uint64_t* slots = a.ws_slot + (int64_t)t * a.S * (M * 16);
  const uint64_t deadline = __builtin_amdgcn_s_memrealtime() + 5000000ull;
  for (int j = lane; j < M * 16; j += 64) {
    float sum = 0.0f;
    bool ok = true;
    for (int sg = 0; sg < a.S; ++sg) {
      uint64_t* p = slots + sg * (M * 16) + j;
      uint64_t w = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      while ((w >> 32) == 0 && __builtin_amdgcn_s_memrealtime() < deadline) {
        __builtin_amdgcn_s_sleep(2);
        w = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      ok = ok && (w >> 32) != 0;
      sum += __builtin_bit_cast(float, (uint32_t)w);
      __hip_atomic_store(p, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    const int b = j / 16, grow = t * 16 + (j % 16);
    if (b < a.m && grow < a.n) store_y(a, b, grow, ok ? sum : __builtin_nanf(""));
  }
}

// A wave's position in its sequence of (item, chunk) steps; wave-uniform.
struct Pos {
  int item, t, s, c, cend;
  bool live;
};

__device__ __forceinline__ Pos first_pos(const KArgs& a, int item) {
  Pos p;
  item = __builtin_amdgcn_readfirstlane(item);
  p.item = item;
  p.live = item < a.items;
  p.t = item / a.S;
  p.s = item % a.S;
  p.c = p.s * a.cps;
  p.cend = min(a.nc, p.c + a.cps);
  return p;
}

__device__ __forceinline__ Pos next_pos(const KArgs& a, const Pos& p) {
  if (p.c + 1 < p.cend) {
    Pos q = p;
    q.c = p.c + 1;
    return q;
  }
  return first_pos(a, p.item + a.gw);
}

// Persistent waves walk balanced items (a tile and a run of chunks) in steps of one record.
// Two record buffers in ping-pong: the loads of step i+1 are in flight while step i is computed,
// and no register copy ever waits on loads still in flight; the step after the last one
// re-reads a valid record so that the loads stay unconditional. Emitting an item never waits
// on memory, so the pipeline runs through item boundaries; split tiles are reduced at the end.
template <int KIND, int D, int M, int RPL>
__global__ void __launch_bounds__(1024) k_gemm_valu(KArgs a) {
  __shared__ __align__(16) unsigned char lds[Tables<KIND, D>::bytes];
  __shared__ __align__(16) uint32_t pstage_all[16 * 64];
  __shared__ int red_list[16 * 32];
  constexpr int H = 16 / RPL;
  stage_tables<KIND>(lds, a);
  const uint32_t mask_off = a.t_bytes;
  __syncthreads();

  const int lane = threadIdx.x & 63;
  // wave-uniform by construction; readfirstlane keeps the schedule in SGPRs. Items are striped
  // over workgroups first so that every CU gets a share.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  Pos p0 = first_pos(a, wave * (int)gridDim.x + blockIdx.x);
  if (!p0.live) return;                        // no barrier follows
  uint32_t* pstage = pstage_all + wave * 64;
  int* reds = red_list + wave * 32;
  int nred = 0;
  const int h = lane % H, vloc = lane / H;

  float acc[M][RPL];
#pragma unroll
  for (int b = 0; b < M; ++b)
#pragma unroll
    for (int r = 0; r < RPL; ++r) acc[b][r] = 0.0f;

  Rec<KIND, M, RPL> r0, r1;
  load_rec<KIND, M, RPL>(r0, a, p0.t, p0.c, h, vloc, lane);
  while (true) {
    const Pos p1 = next_pos(a, p0);
    load_rec<KIND, M, RPL>(r1, a, p1.live ? p1.t : p0.t, p1.live ? p1.c : p0.c, h, vloc, lane);
    compute_rec<KIND, D, M, RPL>(r0, acc, lds, mask_off, pstage, lane, h, vloc, a.m);
    if (p0.c + 1 >= p0.cend) {
      emit_item<M, RPL>(a, acc, p0.t, p0.s, lane, h);
      if (a.S > 1 && p0.s == 0) {
        if (lane == 0) reds[nred] = p0.t;
        ++nred;
      }
    }
    if (!p1.live) break;
    const Pos p2 = next_pos(a, p1);
    load_rec<KIND, M, RPL>(r0, a, p2.live ? p2.t : p1.t, p2.live ? p2.c : p1.c, h, vloc, lane);
    compute_rec<KIND, D, M, RPL>(r1, acc, lds, mask_off, pstage, lane, h, vloc, a.m);
    if (p1.c + 1 >= p1.cend) {
      emit_item<M, RPL>(a, acc, p1.t, p1.s, lane, h);
      if (a.S > 1 && p1.s == 0) {
        if (lane == 0) reds[nred] = p1.t;
        ++nred;
      }
    }
    if (!p2.live) break;
    p0 = p2;
  }
  // The reducer role comes last, after this wave has produced all of its own partial sums.
  for (int i = 0; i < nred; ++i) reduce_tile<M>(a, __builtin_amdgcn_readfirstlane(reds[i]), lane);
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
  constexpr int WMAX = (KIND == SPH_KIND_CB13) ? 8 : 16;
  __shared__ __align__(16) unsigned char lds[Tables<KIND, D>::bytes + WMAX * NB * 1024];
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
  int block;          // threads per workgroup
  int grid;
  int wpt;            // matrix-core kernel: waves per tile
  int nc, cps, S, items;
  size_t ws_bytes;    // workspace the launch needs
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

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Work plan. Vector-ALU path: persistent waves filling every CU to the occupancy the kernel
// allows.
// The chunks-per-item count minimises the rounds of items times their length plus a fixed
// cost per item for its reduction.
Launch plan(const sph_weights* w, int m) {
  Launch L{};
  const int64_t nv = w->k / 8, nt = (w->n + 15) / 16;
  const int kind = sph_kind_of(w->fmt.dir_bits, w->fmt.radius_bits);
  const int cus = num_cus();
  if (m <= 8) {
    const int M = m <= 1 ? 1 : m <= 2 ? 2 : m <= 4 ? 4 : 8;
    const int H = M <= 2 ? 1 : M == 4 ? 2 : 4;
    const int vpc = 64 / H;
    const int wpb = 16;                         // one 16-wave workgroup per CU
    const int grid = cus;
    const int64_t gw = (int64_t)grid * wpb;
    const int64_t nc = (nv + vpc - 1) / vpc;
    // Cost of a plan: rounds of items times (record batches per item + a fixed cost per batch
    // and per item). Split plans (S > 1) pay an extra reduction at the end of the waves' work.
    int64_t best_cps = 1;
    double best = 1e300;
    for (int64_t cps = 1; cps <= nc; ++cps) {
      const int64_t S = (nc + cps - 1) / cps;
      const int64_t items = nt * S;
      const int64_t rounds = (items + gw - 1) / gw;
      if (S > 1 && rounds > 32) continue;       // reducer list bound per wave
      // steps of the busiest wave, plus a small cost per item (its reduction) and one for the
      // split reduction at the end of the waves' work
      const double cost = (double)rounds * ((double)cps + 0.5) + (S > 1 ? 2.0 : 0.0);
      if (cost < best - 1e-9) {
        best = cost;
        best_cps = cps;
      }
    }
    L.fn = pick(w->fmt.dir_bits, w->fmt.radius_bits, false, M);
    L.block = 64 * wpb;
    L.nc = (int)nc;
    L.cps = (int)best_cps;
    L.S = (int)((nc + best_cps - 1) / best_cps);
    L.items = (int)(nt * L.S);
    const int64_t need = (L.items + wpb - 1) / wpb;
    L.grid = (int)(need < grid ? need : grid);
    L.ws_bytes = L.S > 1 ? (size_t)nt * L.S * M * 16 * 8 : 0;
  } else {
    const int NB = m <= 16 ? 1 : 2;
    const int64_t per_wave = 4 * 8;             // 8 MFMA steps per wave
    int wpt = (int)((nv + per_wave - 1) / per_wave);
    const int wmax = (kind == SPH_KIND_CB13) ? 8 : 16;
    wpt = wpt < 1 ? 1 : wpt > wmax ? wmax : wpt;
    L.fn = pick(w->fmt.dir_bits, w->fmt.radius_bits, true, NB);
    L.wpt = wpt;
    L.block = 64 * wpt;
    const int64_t cap = (int64_t)cus * 4;
    L.grid = (int)(nt < cap ? nt : cap);
    L.ws_bytes = 0;
  }
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

sph_status launch(const Launch& L, const KArgs& a, hipStream_t s) {
  KArgs args = a;
  void* kargs[] = {&args};
  if (hipLaunchKernel(L.fn, dim3(L.grid), dim3(L.block), kargs, 0, s) != hipSuccess) return SPH_ERR_HIP;
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
  *bytes = plan(w, (int)m).ws_bytes;
  return SPH_OK;
}

sph_status sph_gemm_small(const sph_weights* w, const void* d_x, int64_t m, int64_t ldx, void* d_y,
                          int64_t ldy, sph_dtype y_dtype, void* d_ws, size_t ws_bytes, void* stream) {
  if (!w || !d_x || !d_y) return SPH_ERR_NULL;
  if (!valid_desc(w)) return SPH_ERR_BAD_DESCRIPTOR;
  if (m < 1 || m > 32) return SPH_ERR_SHAPE;
  if (ldx < w->k || ldy < w->n || ldx % 8 != 0) return SPH_ERR_SHAPE;
  if (y_dtype != SPH_F16 && y_dtype != SPH_F32) return SPH_ERR_SHAPE;
  if ((uintptr_t)d_x % 16 != 0 || (uintptr_t)d_y % 4 != 0) return SPH_ERR_SHAPE;
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
  a.gw = L.grid * (L.block / 64);
  a.cps = L.cps;
  a.S = L.S;
  a.items = L.items;
  if (L.ws_bytes > 0) a.ws_slot = (uint64_t*)d_ws;
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
