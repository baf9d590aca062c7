// Spherical encoder and codebook initialisation on the device (Sec. 3.1, Eq. 3 and 5-7;
// Sec. 4.1 for the k-means settings).
//
// All arithmetic is fp64 on the vector ALUs, from fp32 weights, so that each integer decision (a
// direction index, a radius level, a sampled vector) is taken in the same precision as in a plain
// fp64 implementation of the equations. Sums whose order fixes the bits of a stored value (the
// squared radius, the least-squares radius of Eq. 6, the norm of a k-means centre) use the
// pairwise order ((p0+p1)+(p2+p3))+((p4+p5)+(p6+p7)) with the products rounded first, never
// fused. Every reduction runs in a fixed order, so repeated calls give bitwise identical results.
//
// Work layout:
//   encoder      one thread per 8-D vector (four per thread), 16 neighbouring lanes form one
//                128-weight group; the codebook is staged in LDS as fp64 in 512-entry chunks and
//                read by broadcast.
//   k-means      squared radii and their running sum (three-pass scan), inverse-CDF sampling by
//                binary search, then per iteration: assignment (the centre range split over
//                workgroups, splits combined in ascending order), exact fixed-point centre sums
//                (integer LDS atomics per block, integer sums across blocks, so the order of
//                arrival does not matter), renormalisation.
#include <hip/hip_runtime.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "sph_fp.h"
#include "sph_host.h"
#include "sph_layout.h"

namespace {

constexpr double kEps = 1e-12;  // Eq. 3's guard against a zero radius
constexpr int kThreads = 256;
constexpr int kVpt = 4;          // vectors (or samples) per thread in the assignment kernels
constexpr int kChunk = 512;      // codebook entries per LDS pass: 32 KiB of fp64
constexpr int kScanItems = 8;    // vectors per thread in the radius scan
constexpr int kScanBlock = kThreads * kScanItems;
constexpr int kTargetBlocks = 1024;  // workgroups the k-means launches aim for (256 CUs)

// Pairwise sum of the eight rounded products a[j] * b[j].
__device__ __forceinline__ double dot8_pairwise(const double* a, const double* b) {
#pragma clang fp contract(off)
  double p[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) p[j] = a[j] * b[j];
  return ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
}

// Eq. 3 on one fp32 vector: magnitudes |w_j| (w_+), sign bits (set where w_j < 0) and the
// unit direction w_+ / max(||w||, eps). Returns the radius.
__device__ __forceinline__ double decompose(const float* __restrict__ w, int64_t ldw, int64_t nv, int64_t i,
                                            double a[8], double d[8], uint32_t& neg) {
#pragma clang fp contract(off)
  const int64_t row = i / nv, v = i - row * nv;
  const float4* p = reinterpret_cast<const float4*>(w + row * ldw + v * 8);
  const float4 x0 = p[0], x1 = p[1];
  const float f[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
  neg = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    neg |= (f[j] < 0.0f ? 1u : 0u) << j;
    a[j] = fabs((double)f[j]);
  }
  const double r = sqrt(dot8_pairwise(a, a));
  const double rr = r < kEps ? kEps : r;
#pragma unroll
  for (int j = 0; j < 8; ++j) d[j] = a[j] / rr;
  return r;
}

// Eq. 5 over entries [base, base + cnt) of a codebook held in LDS (fp64, 8 per entry): strict
// comparison in ascending index order keeps the lowest index among equal cosines.
__device__ __forceinline__ void argmax_chunk(const double* __restrict__ cl, int cnt, int base,
                                             const double (&d)[kVpt][8], double (&best)[kVpt],
                                             int (&bz)[kVpt]) {
  for (int e = 0; e < cnt; ++e) {
    const double2* ce2 = reinterpret_cast<const double2*>(cl + e * 8);
    const double2 c01 = ce2[0], c23 = ce2[1], c45 = ce2[2], c67 = ce2[3];
    const double c[8] = {c01.x, c01.y, c23.x, c23.y, c45.x, c45.y, c67.x, c67.y};
#pragma unroll
    for (int u = 0; u < kVpt; ++u) {
      double s = d[u][0] * c[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) s = fma(d[u][j], c[j], s);
      if (s > best[u]) {
        best[u] = s;
        bz[u] = base + e;
      }
    }
  }
}

// Stage entries [c0, c1) of the codebook chunk by chunk into LDS and run the argmax over them.
// The source is either the fp16 codebook or fp64 centres. Every thread of the block must call this.
template <typename T>
__device__ __forceinline__ void argmax_codebook(const T* __restrict__ src, int c0, int c1, double* cl,
                                                const double (&d)[kVpt][8], double (&best)[kVpt],
                                                int (&bz)[kVpt]) {
  for (int base = c0; base < c1; base += kChunk) {
    const int cnt = min(kChunk, c1 - base);
    __syncthreads();
    for (int t = threadIdx.x; t < cnt * 8; t += kThreads) {
      if constexpr (sizeof(T) == 2)
        cl[t] = h2d(src[(int64_t)base * 8 + t]);
      else
        cl[t] = src[(int64_t)base * 8 + t];
    }
    __syncthreads();
    argmax_chunk(cl, cnt, base, d, best, bz);
  }
}

// ------------------------------------------------------------------------------------ encoder

struct EncArgs {
  const float* w;
  int64_t ldw, nv, nvec;
  const uint16_t* cb;
  int ncb, vmax;
  uint8_t* signs;
  uint16_t* dir;
  uint8_t* q;
  uint16_t* gmin;
  uint16_t* gstep;
};

// Eq. 3, 5, 6 and 7 for kVpt * 256 consecutive vectors. Groups of 16 vectors never straddle a
// row (k is a multiple of 128) and start at multiples of 16 in the flat vector index, so each
// group is 16 aligned lanes of one wave, all inside or all outside [0, nvec).
__global__ __launch_bounds__(kThreads) void k_encode(EncArgs a) {
  __shared__ double cl[kChunk * 8];
  const int64_t blk = (int64_t)blockIdx.x * kThreads * kVpt;
  double d[kVpt][8], best[kVpt];
  int bz[kVpt];
#pragma unroll
  for (int u = 0; u < kVpt; ++u) {
    const int64_t i = blk + u * kThreads + threadIdx.x;
    best[u] = -INFINITY;
    bz[u] = 0;
    double av[8];
    uint32_t neg;
    if (i < a.nvec) {
      decompose(a.w, a.ldw, a.nv, i, av, d[u], neg);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) d[u][j] = 0.0;
    }
  }
  argmax_codebook(a.cb, 0, a.ncb, cl, d, best, bz);
#pragma unroll
  for (int u = 0; u < kVpt; ++u) {
    const int64_t i = blk + u * kThreads + threadIdx.x;
    // the magnitudes and signs are read again rather than kept live across the argmax
    double av[8] = {0, 0, 0, 0, 0, 0, 0, 0}, dd[8];
    uint32_t neg = 0;
    if (i < a.nvec) decompose(a.w, a.ldw, a.nv, i, av, dd, neg);
    double c[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) c[j] = h2d(a.cb[(int64_t)bz[u] * 8 + j]);
    const double rt = dot8_pairwise(av, c);  // Eq. 6
    double lo = rt, hi = rt;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      lo = fmin(lo, __shfl_xor(lo, o, 16));
      hi = fmax(hi, __shfl_xor(hi, o, 16));
    }
    const uint16_t lo16 = d2h(lo), st16 = d2h((hi - lo) / (double)a.vmax);
    const double lod = h2d(lo16), std_ = h2d(st16);
    int q = 0;
    if (std_ > 0.0) {
      const double t = rint((rt - lod) / std_);
      q = (int)fmin(fmax(t, 0.0), (double)a.vmax);
    }
    if (i < a.nvec) {
      a.signs[i] = (uint8_t)neg;
      a.dir[i] = (uint16_t)bz[u];
      a.q[i] = (uint8_t)q;
      if ((threadIdx.x & 15) == 0) {
        a.gmin[i >> 4] = lo16;
        a.gstep[i >> 4] = st16;
      }
    }
  }
}

// Matrix-core direction search for the 2^13-entry codebook (exact in fp16). A unit direction d is
// split as d_hi = fp16(d), d_lo = fp16(d - d_hi); with K = 16 = (c, c) . (d_hi, d_lo) one
// v_mfma_f32_16x16x16_f16 scores 16 entries against 16 vectors with exact products and fp32
// sums. |score - c.d| <= 2^-22 + 8 * 2^-24 (the split) + 16 * 2^-24 * 2 (fp32 sums) < delta =
// 3e-6 (the matrix cores keep fp16 subnormal inputs, which the split produces for coordinates
// below 2^-14). The fp64 argmax e* then has score >= s(e*) - delta >= best score - 2 delta:
// every entry within kMxSlack (> 2 delta, with margin) of the best score is a candidate. Pass 1 finds each vector's best score; pass 2 rescores, and evaluates the fp64
// cosine (the same FMA chain as the vector-ALU search, in ascending entry order) only for the
// candidates. The result equals the full fp64 scan's. Lane layout: vector j = lane % 16 of each 16-vector block
// (one radius group), entries 4 * (lane / 16) + e of each 16-entry block; the four lanes of a
// vector are combined at the end (larger cosine, then lower index).
constexpr int kMxWaves = 8;
constexpr int kMxNB = 4;                                   // 16-vector blocks per wave
constexpr int kMxVecPerWg = kMxWaves * kMxNB * 16;         // 512
constexpr int kMxMaxEntries = 8192;
constexpr float kMxSlack = 2e-5f;

typedef _Float16 h4v __attribute__((ext_vector_type(4)));
typedef float f4v __attribute__((ext_vector_type(4)));

// A operand of lane (j, qd) for entry block e0: coordinates 4 * (qd & 1) .. + 3 of entry e0 + j
// (k 8..15 repeat k 0..7), one 8-byte LDS read.
__device__ __forceinline__ h4v mx_a_operand(const uint4* cbl, int e0, int j, int qd) {
  return __builtin_bit_cast(h4v, ((const uint2*)cbl)[(e0 + j) * 2 + (qd & 1)]);
}

// Scores of non-negative vectors are compared through their bit patterns as signed integers:
// for non-negative floats the order is the same, and integer max needs no NaN canonicalisation.
__device__ __forceinline__ int fbits(float x) { return __builtin_bit_cast(int, x); }
__device__ __forceinline__ int max4bits(const f4v acc) {
  return max(max(fbits(acc[0]), fbits(acc[1])), max(fbits(acc[2]), fbits(acc[3])));
}

__global__ __launch_bounds__(64 * kMxWaves) void k_encode_mx(EncArgs a, int64_t nchunks) {
  __shared__ uint4 cbl[kMxMaxEntries];   // the fp16 codebook, 16 bytes per entry (2^13 entries)
  for (int t = threadIdx.x; t < kMxMaxEntries; t += 64 * kMxWaves) cbl[t] = ((const uint4*)a.cb)[t];
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j = lane & 15, qd = lane >> 4;
  for (int64_t ch = blockIdx.x; ch < nchunks; ch += gridDim.x) {
    const int64_t v0 = ch * kMxVecPerWg + (int64_t)wave * (kMxNB * 16);
    double d[kMxNB][8];
    h4v bop[kMxNB];
    bool ok[kMxNB];
#pragma unroll
    for (int nb = 0; nb < kMxNB; ++nb) {
      const int64_t i = v0 + nb * 16 + j;
      ok[nb] = i < a.nvec;
      double av[8];
      uint32_t neg;
      if (ok[nb]) {
        decompose(a.w, a.ldw, a.nv, i, av, d[nb], neg);
      } else {
#pragma unroll
        for (int t = 0; t < 8; ++t) d[nb][t] = 0.0;
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        // both halves pass through an empty asm so that the select stays a register select
        // (an indexed read would put d in scratch memory)
        double x0 = d[nb][t], x1 = d[nb][4 + t];
        asm volatile("" : "+v"(x0), "+v"(x1));
        const double x = (qd & 1) ? x1 : x0;
        const _Float16 hi = (_Float16)(float)x;
        bop[nb][t] = qd < 2 ? hi : (_Float16)(float)(x - (double)hi);
      }
    }
    // pass 1: the best matrix-core score of every vector (scores of the non-negative entries and
    // directions are >= 0 up to rounding; only a zero vector has its best at 0)
    int mx[kMxNB];
#pragma unroll
    for (int nb = 0; nb < kMxNB; ++nb) mx[nb] = INT_MIN;
#pragma unroll 4
    for (int e0 = 0; e0 < kMxMaxEntries; e0 += 16) {
      const h4v aop = mx_a_operand(cbl, e0, j, qd);
#pragma unroll
      for (int nb = 0; nb < kMxNB; ++nb) {
        const f4v acc = __builtin_amdgcn_mfma_f32_16x16x16f16(aop, bop[nb], f4v{0.0f, 0.0f, 0.0f, 0.0f}, 0, 0, 0);
        mx[nb] = max(mx[nb], max4bits(acc));
      }
    }
    int thr[kMxNB];
#pragma unroll
    for (int nb = 0; nb < kMxNB; ++nb) {
      int v = max(mx[nb], __shfl_xor(mx[nb], 16, 64));
      v = max(v, __shfl_xor(v, 32, 64));
      const float t = __builtin_bit_cast(float, v) - kMxSlack;
      // a threshold below 0 (a zero vector) takes every entry; vectors past the end take none
      thr[nb] = !ok[nb] ? INT_MAX : t < 0.0f ? INT_MIN : fbits(t);
    }
    // pass 2: fp64 cosines of the candidates, ascending entry order per lane
    double best[kMxNB];
    int bz[kMxNB];
#pragma unroll
    for (int nb = 0; nb < kMxNB; ++nb) {
      best[nb] = -INFINITY;
      bz[nb] = kMxMaxEntries;
    }
#pragma unroll 2
    for (int e0 = 0; e0 < kMxMaxEntries; e0 += 16) {
      const h4v aop = mx_a_operand(cbl, e0, j, qd);
#pragma unroll
      for (int nb = 0; nb < kMxNB; ++nb) {
        const f4v acc = __builtin_amdgcn_mfma_f32_16x16x16f16(aop, bop[nb], f4v{0.0f, 0.0f, 0.0f, 0.0f}, 0, 0, 0);
        if (max4bits(acc) >= thr[nb]) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (fbits(acc[e]) >= thr[nb]) {
              const int ent = e0 + 4 * qd + e;
              const uint4 ce = cbl[ent];
              const uint32_t cw[4] = {ce.x, ce.y, ce.z, ce.w};
              double c[8];
#pragma unroll
              for (int t = 0; t < 8; ++t) c[t] = h2d((uint16_t)(cw[t / 2] >> (16 * (t & 1))));
              double sc = d[nb][0] * c[0];
#pragma unroll
              for (int t = 1; t < 8; ++t) sc = fma(d[nb][t], c[t], sc);
              if (sc > best[nb]) {
                best[nb] = sc;
                bz[nb] = ent;
              }
            }
          }
        }
      }
    }
#pragma unroll
    for (int nb = 0; nb < kMxNB; ++nb) {
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const double ob = __shfl_xor(best[nb], o, 64);
        const int oz = __shfl_xor(bz[nb], o, 64);
        if (ob > best[nb] || (ob == best[nb] && oz < bz[nb])) {
          best[nb] = ob;
          bz[nb] = oz;
        }
      }
      if (bz[nb] >= a.ncb) bz[nb] = 0;   // no candidate (non-finite input): any valid index
    }
    // Eq. 6 and 7 as in k_encode; the four lanes of a vector agree, the first writes
#pragma unroll
    for (int nb = 0; nb < kMxNB; ++nb) {
      const int64_t i = v0 + nb * 16 + j;
      double av[8] = {0, 0, 0, 0, 0, 0, 0, 0}, dd[8];
      uint32_t neg = 0;
      if (ok[nb]) decompose(a.w, a.ldw, a.nv, i, av, dd, neg);
      double c[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) c[t] = h2d(a.cb[(int64_t)bz[nb] * 8 + t]);
      const double rt = dot8_pairwise(av, c);
      double lo = rt, hi = rt;
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        lo = fmin(lo, __shfl_xor(lo, o, 16));
        hi = fmax(hi, __shfl_xor(hi, o, 16));
      }
      const uint16_t lo16 = d2h(lo), st16 = d2h((hi - lo) / (double)a.vmax);
      const double lod = h2d(lo16), std_ = h2d(st16);
      int q = 0;
      if (std_ > 0.0) q = (int)fmin(fmax(rint((rt - lod) / std_), 0.0), (double)a.vmax);
      if (ok[nb] && qd == 0) {
        a.signs[i] = (uint8_t)neg;
        a.dir[i] = (uint16_t)bz[nb];
        a.q[i] = (uint8_t)q;
        if (j == 0) {
          a.gmin[i >> 4] = lo16;
          a.gstep[i >> 4] = st16;
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------------ k-means

// Block-wide exclusive prefix of one value per thread, in a fixed order; also returns the block
// total. `sh` holds kThreads doubles.
__device__ __forceinline__ double block_exclusive(double v, double* sh, double& total) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  double incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double t = __shfl_up(incl, o, 64);
    if (lane >= o) incl += t;
  }
  if (lane == 63) sh[wv] = incl;
  __syncthreads();
  double woff = 0.0;
  for (int k = 0; k < wv; ++k) woff += sh[k];
  double tot = 0.0;
  for (int k = 0; k < kThreads / 64; ++k) tot += sh[k];
  __syncthreads();
  total = tot;
  return woff + (incl - v);
}

// Squared radius r^2 of every vector (r from Eq. 3), stored in cdf[], and each block's total.
__global__ __launch_bounds__(kThreads) void k_r2(const float* __restrict__ w, int64_t ldw, int64_t nv,
                                                 int64_t nvec, double* __restrict__ cdf,
                                                 double* __restrict__ bsum) {
  __shared__ double sh[kThreads / 64];
  const int64_t i0 = (int64_t)blockIdx.x * kScanBlock + (int64_t)threadIdx.x * kScanItems;
  double s = 0.0;
  for (int j = 0; j < kScanItems; ++j) {
    const int64_t i = i0 + j;
    if (i >= nvec) break;
    double av[8], d[8];
    uint32_t neg;
    const double r = decompose(w, ldw, nv, i, av, d, neg);
    const double r2 = r * r;
    cdf[i] = r2;
    s += r2;
  }
  double total;
  block_exclusive(s, sh, total);
  if (threadIdx.x == 0) bsum[blockIdx.x] = total;
}

// Exclusive running sum of the nb block totals, in place, by one block.
__global__ __launch_bounds__(kThreads) void k_scan_blocks(double* __restrict__ bsum, int64_t nb) {
  __shared__ double sh[kThreads / 64];
  const int64_t per = (nb + kThreads - 1) / kThreads;
  const int64_t b0 = (int64_t)threadIdx.x * per, b1 = min(nb, b0 + per);
  double s = 0.0;
  for (int64_t b = b0; b < b1; ++b) s += bsum[b];
  double total;
  double run = block_exclusive(s, sh, total);
  for (int64_t b = b0; b < b1; ++b) {
    const double v = bsum[b];
    bsum[b] = run;
    run += v;
  }
}

// Running sum of r^2 in storage order: cdf[i] = sum of r^2 over vectors 0..i.
__global__ __launch_bounds__(kThreads) void k_scan_apply(double* __restrict__ cdf, const double* __restrict__ boff,
                                                         int64_t nvec) {
  __shared__ double sh[kThreads / 64];
  const int64_t i0 = (int64_t)blockIdx.x * kScanBlock + (int64_t)threadIdx.x * kScanItems;
  double v[kScanItems];
  double s = 0.0;
  for (int j = 0; j < kScanItems; ++j) {
    const int64_t i = i0 + j;
    v[j] = i < nvec ? cdf[i] : 0.0;
    s += v[j];
  }
  double total;
  const double off = boff[blockIdx.x] + block_exclusive(s, sh, total);
  double run = 0.0;
  for (int j = 0; j < kScanItems; ++j) {
    const int64_t i = i0 + j;
    run += v[j];
    if (i < nvec) cdf[i] = off + run;
  }
}

// Inverse-CDF draw (Sec. 3.1): sample j takes the first vector whose running r^2 exceeds
// u_j * total, clamped to the last vector; its unit direction goes to ds[j][0..8).
__global__ __launch_bounds__(kThreads) void k_sample(const float* __restrict__ w, int64_t ldw, int64_t nv,
                                                     int64_t nvec, const double* __restrict__ cdf,
                                                     const double* __restrict__ u, int64_t ns,
                                                     double* __restrict__ ds, int64_t* __restrict__ sidx) {
  const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (j >= ns) return;
  const double target = u[j] * cdf[nvec - 1];
  int64_t lo = 0, hi = nvec;
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (cdf[mid] > target)
      hi = mid;
    else
      lo = mid + 1;
  }
  const int64_t idx = lo < nvec ? lo : nvec - 1;
  if (sidx) sidx[j] = idx;
  double av[8], d[8];
  uint32_t neg;
  decompose(w, ldw, nv, idx, av, d, neg);
#pragma unroll
  for (int c = 0; c < 8; ++c) ds[j * 8 + c] = d[c];
}

__global__ __launch_bounds__(kThreads) void k_init_centres(const uint16_t* __restrict__ init, int64_t count,
                                                           double* __restrict__ cen) {
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (t < count) cen[t] = h2d(init[t]);
}

// Eq. 5 for every sample against centres [split * per, (split + 1) * per): the best cosine and its
// index per sample and split (blockIdx.y is the split).
__global__ __launch_bounds__(kThreads) void k_assign_split(const double* __restrict__ ds, int64_t ns,
                                                           const double* __restrict__ cen, int ncb, int per,
                                                           double* __restrict__ sbest, int32_t* __restrict__ sidx) {
  __shared__ double cl[kChunk * 8];
  const int64_t blk = (int64_t)blockIdx.x * kThreads * kVpt;
  const int c0 = blockIdx.y * per, c1 = min(ncb, c0 + per);
  double d[kVpt][8], best[kVpt];
  int bz[kVpt];
#pragma unroll
  for (int u = 0; u < kVpt; ++u) {
    const int64_t j = blk + u * kThreads + threadIdx.x;
    best[u] = -INFINITY;
    bz[u] = c0;
#pragma unroll
    for (int c = 0; c < 8; ++c) d[u][c] = j < ns ? ds[j * 8 + c] : 0.0;
  }
  argmax_codebook(cen, c0, c1, cl, d, best, bz);
#pragma unroll
  for (int u = 0; u < kVpt; ++u) {
    const int64_t j = blk + u * kThreads + threadIdx.x;
    if (j < ns) {
      sbest[blockIdx.y * ns + j] = best[u];
      sidx[blockIdx.y * ns + j] = bz[u];
    }
  }
}

// The splits combined in ascending order with a strict comparison (the same decision as one scan
// over all centres); z[j] gets the nearest centre and each block writes the sum of its samples'
// cosines to their centre (each summed in pairwise order, then in a fixed order over the block).
__global__ __launch_bounds__(kThreads) void k_assign_final(const double* __restrict__ ds, int64_t ns,
                                                           const double* __restrict__ cen, int nsplit,
                                                           const double* __restrict__ sbest,
                                                           const int32_t* __restrict__ sidx,
                                                           int32_t* __restrict__ z, double* __restrict__ opart) {
  __shared__ double sh[kThreads / 64];
  const int64_t j = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  double v = 0.0;
  if (j < ns) {
    double best = sbest[j];
    int bz = sidx[j];
    for (int t = 1; t < nsplit; ++t) {
      const double b = sbest[t * ns + j];
      if (b > best) {
        best = b;
        bz = sidx[t * ns + j];
      }
    }
    z[j] = bz;
    double d[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) d[c] = ds[j * 8 + c];
    v = dot8_pairwise(d, cen + (int64_t)bz * 8);
  }
  double total;
  block_exclusive(v, sh, total);
  if (threadIdx.x == 0) opart[blockIdx.x] = total;
}

// Objective of one assignment: the blocks' sums, lane-strided in block order and then combined
// by a fixed lane tree.
__global__ __launch_bounds__(64) void k_objective(const double* __restrict__ opart, int64_t nblk,
                                                  double* __restrict__ out) {
  double s = 0.0;
  for (int64_t b = threadIdx.x; b < nblk; b += 64) s += opart[b];
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  if (threadIdx.x == 0) *out = s;
}

// Centre sums by exact fixed-point accumulation. A direction component v in [0, 1 + 2^-52] is
// truncated to T = floor(v * 2^100) and added as three 40-bit limbs in 64-bit integers. Integer
// addition is associative, so the sums do not depend on the order in which samples are added,
// and 2^24 samples cannot overflow a limb. The sum is exact up to the 2^-100 truncation of each
// term. Block (r, p) adds the samples of chunk p whose centre lies in range r with LDS atomics
// and stores its limbs; one wave per centre then adds the chunks' limbs.
constexpr int kFixBits = 100;
constexpr int kLimbBits = 40;
constexpr uint64_t kLimbMask = (1ull << kLimbBits) - 1;
constexpr int kLimbs = 8 * 3;       // limbs per centre
constexpr int kAccRange = 512;      // centres per LDS accumulator: 96 KiB

__device__ __forceinline__ void to_limbs(double v, uint64_t& l0, uint64_t& l1, uint64_t& l2) {
  const uint64_t bits = __builtin_bit_cast(uint64_t, v);
  const int ex = (int)(bits >> 52);  // components are >= 0; 0 for zero and subnormals
  unsigned __int128 t = 0;
  if (ex != 0) {
    const uint64_t m = (bits & 0xFFFFFFFFFFFFFull) | 0x10000000000000ull;
    const int sh = ex - 1075 + kFixBits;  // v = m * 2^(ex - 1075)
    if (sh >= 0)
      t = (unsigned __int128)m << sh;
    else if (sh > -64)
      t = m >> -sh;
  }
  l0 = (uint64_t)t & kLimbMask;
  l1 = (uint64_t)(t >> kLimbBits) & kLimbMask;
  l2 = (uint64_t)(t >> (2 * kLimbBits));
}

__global__ __launch_bounds__(kThreads) void k_accumulate(const double* __restrict__ ds, int64_t ns,
                                                         const int32_t* __restrict__ z, int ncb, int64_t ch,
                                                         unsigned long long* __restrict__ part) {
  __shared__ unsigned long long la[kAccRange * kLimbs];
  const int c0 = blockIdx.x * kAccRange, c1 = min(ncb, c0 + kAccRange), nc = c1 - c0;
  const int p = blockIdx.y;
  for (int t = threadIdx.x; t < nc * kLimbs; t += kThreads) la[t] = 0;
  __syncthreads();
  const int64_t j0 = (int64_t)p * ch, j1 = min(ns, j0 + ch);
  for (int64_t j = j0 + threadIdx.x; j < j1; j += kThreads) {
    const int c = z[j];
    if (c < c0 || c >= c1) continue;
    unsigned long long* a = la + (c - c0) * kLimbs;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint64_t l0, l1, l2;
      to_limbs(ds[j * 8 + e], l0, l1, l2);
      if (l0) atomicAdd(a + 3 * e, (unsigned long long)l0);
      if (l1) atomicAdd(a + 3 * e + 1, (unsigned long long)l1);
      if (l2) atomicAdd(a + 3 * e + 2, (unsigned long long)l2);
    }
  }
  __syncthreads();
  unsigned long long* out = part + ((int64_t)p * ncb + c0) * kLimbs;
  for (int t = threadIdx.x; t < nc * kLimbs; t += kThreads) out[t] = la[t];
}

// New centre c: the chunks' limbs added (integers, so in any order), converted to fp64 and the
// sum normalised to unit length; a centre without directions keeps its position.
__global__ __launch_bounds__(64) void k_update(const unsigned long long* __restrict__ part, int np, int ncb,
                                               double* __restrict__ cen) {
#pragma clang fp contract(off)
  const int c = blockIdx.x;
  const int lane = threadIdx.x;
  uint64_t l[kLimbs];
#pragma unroll
  for (int t = 0; t < kLimbs; ++t) l[t] = 0;
  for (int p = lane; p < np; p += 64) {
    const unsigned long long* a = part + ((int64_t)p * ncb + c) * kLimbs;
#pragma unroll
    for (int t = 0; t < kLimbs; ++t) l[t] += a[t];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
#pragma unroll
    for (int t = 0; t < kLimbs; ++t) l[t] += __shfl_xor(l[t], o, 64);
  }
  if (lane != 0) return;
  double s[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    uint64_t l0 = l[3 * e], l1 = l[3 * e + 1], l2 = l[3 * e + 2];
    l1 += l0 >> kLimbBits;
    l0 &= kLimbMask;
    l2 += l1 >> kLimbBits;
    l1 &= kLimbMask;
    // l2 < 2^53 and l1, l0 < 2^40 convert exactly; two roundings combine them
    const double hi = ((double)l2 * 0x1p40 + (double)l1) * 0x1p40;
    s[e] = (hi + (double)l0) * 0x1p-100;
  }
  const double norm = sqrt(dot8_pairwise(s, s));
  if (norm > 0.0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) cen[(int64_t)c * 8 + e] = s[e] / norm;
  }
}

__global__ __launch_bounds__(kThreads) void k_centres_to_f16(const double* __restrict__ cen, int64_t count,
                                                             uint16_t* __restrict__ out) {
  const int64_t t = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (t < count) out[t] = d2h(cen[t]);
}

// ------------------------------------------------------------------------------------ host side

inline uint64_t align256(uint64_t x) { return (x + 255) / 256 * 256; }

struct KmPlan {
  int64_t nvec, nb, nab, nfb, ch;
  int ncb, nsplit, per, nr, np;
  uint64_t off_cdf, off_bsum, off_ds, off_z, off_opart, off_cen, off_acc, off_sbest, off_sidx, total;
};

KmPlan km_plan(const sph_format* fmt, int64_t n, int64_t k, int64_t ns) {
  KmPlan P{};
  P.nvec = n * (k / SPH_VEC);
  P.nb = (P.nvec + kScanBlock - 1) / kScanBlock;
  P.nab = (ns + kThreads * kVpt - 1) / (kThreads * kVpt);
  P.nfb = (ns + kThreads - 1) / kThreads;
  P.ncb = 1 << fmt->dir_bits;
  // centre splits of the assignment: enough workgroups for the chip, at least 64 centres each
  int64_t sp = (kTargetBlocks + P.nab - 1) / P.nab;
  sp = std::min<int64_t>(sp, std::max(1, P.ncb / 64));
  P.per = (int)((P.ncb + sp - 1) / sp);
  P.nsplit = (P.ncb + P.per - 1) / P.per;
  // centre ranges x sample chunks of the accumulation: about 128 workgroups
  P.nr = (P.ncb + kAccRange - 1) / kAccRange;
  int64_t np = (128 + P.nr - 1) / P.nr;
  np = std::min<int64_t>(np, (ns + kThreads - 1) / kThreads);
  P.ch = (ns + np - 1) / np;
  P.np = (int)((ns + P.ch - 1) / P.ch);
  uint64_t p = 0;
  P.off_cdf = p;
  p = align256(p + (uint64_t)P.nvec * 8);
  P.off_bsum = p;
  p = align256(p + (uint64_t)P.nb * 8);
  P.off_ds = p;
  p = align256(p + (uint64_t)ns * 64);
  P.off_z = p;
  p = align256(p + (uint64_t)ns * 4);
  P.off_opart = p;
  p = align256(p + (uint64_t)P.nfb * 8);
  P.off_cen = p;
  p = align256(p + (uint64_t)P.ncb * 64);
  P.off_acc = p;
  p = align256(p + (uint64_t)P.np * P.ncb * kLimbs * 8);
  P.off_sbest = p;
  p = align256(p + (uint64_t)P.nsplit * ns * 8);
  P.off_sidx = p;
  p = align256(p + (uint64_t)P.nsplit * ns * 4);
  P.total = p;
  return P;
}

constexpr int64_t kMaxSamples = int64_t(1) << 24;
constexpr int32_t kMaxIters = 10000;

// The encoder and k-means handle 8-D vectors (the 4-D and 16-D formats are decode-only).
int check_fmt8(const sph_format* fmt) {
  const int st = sph_host_check_format(fmt);
  if (st) return st;
  return fmt->vec_dim == SPH_VEC ? SPH_OK : SPH_ERR_UNSUPPORTED_FORMAT;
}

int check_common(const sph_format* fmt, int64_t n, int64_t k, const float* d_w, int64_t ldw) {
  int st = check_fmt8(fmt);
  if (st) return st;
  st = sph_host_check_shape(n, k);
  if (st) return st;
  if (!d_w) return SPH_ERR_NULL;
  if (ldw < k || ldw % 4 != 0 || (uintptr_t)d_w % 16 != 0) return SPH_ERR_SHAPE;
  return SPH_OK;
}

template <typename... A>
bool launch_ok(const void* fn, dim3 grid, dim3 block, hipStream_t s, A... args) {
  void* kargs[] = {(void*)&args...};
  if (hipLaunchKernel(fn, grid, block, kargs, 0, s) != hipSuccess) return false;
  return hipGetLastError() == hipSuccess;
}

}  // namespace

extern "C" {

sph_status sph_encode(const sph_format* fmt, int64_t n, int64_t k, const float* d_w, int64_t ldw,
                      const uint16_t* d_codebook, uint8_t* d_signs, uint16_t* d_dir_idx,
                      uint8_t* d_radius_code, uint16_t* d_group_min, uint16_t* d_group_step,
                      void* stream) {
  if (!fmt || !d_codebook || !d_signs || !d_dir_idx || !d_radius_code || !d_group_min || !d_group_step)
    return SPH_ERR_NULL;
  const int st = check_common(fmt, n, k, d_w, ldw);
  if (st) return (sph_status)st;
  if ((uintptr_t)d_codebook % 2 || (uintptr_t)d_dir_idx % 2 || (uintptr_t)d_group_min % 2 ||
      (uintptr_t)d_group_step % 2)
    return SPH_ERR_SHAPE;
  EncArgs a{};
  a.w = d_w;
  a.ldw = ldw;
  a.nv = k / SPH_VEC;
  a.nvec = n * a.nv;
  a.cb = d_codebook;
  a.ncb = 1 << fmt->dir_bits;
  a.vmax = (1 << fmt->radius_bits) - 1;
  a.signs = d_signs;
  a.dir = d_dir_idx;
  a.q = d_radius_code;
  a.gmin = d_group_min;
  a.gstep = d_group_step;
  if (a.ncb == kMxMaxEntries) {
    // the 2^13-entry codebook: matrix-core search, one 128 KiB codebook copy per CU
    const int64_t nchunks = (a.nvec + kMxVecPerWg - 1) / kMxVecPerWg;
    int dev = 0, cus = 256;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      cus = 256;
    const int64_t grid = std::min<int64_t>(nchunks, cus);
    if (!launch_ok((const void*)k_encode_mx, dim3((unsigned)grid), dim3(64 * kMxWaves), (hipStream_t)stream, a, nchunks))
      return SPH_ERR_HIP;
    return SPH_OK;
  }
  const int64_t grid = (a.nvec + kThreads * kVpt - 1) / (kThreads * kVpt);
  if (!launch_ok((const void*)k_encode, dim3((unsigned)grid), dim3(kThreads), (hipStream_t)stream, a))
    return SPH_ERR_HIP;
  return SPH_OK;
}

sph_status sph_kmeans_workspace_bytes(const sph_format* fmt, int64_t n, int64_t k, int64_t n_samples,
                                      size_t* bytes) {
  if (!fmt || !bytes) return SPH_ERR_NULL;
  int st = check_fmt8(fmt);
  if (st) return (sph_status)st;
  st = sph_host_check_shape(n, k);
  if (st) return (sph_status)st;
  if (n_samples < 1 || n_samples > kMaxSamples) return SPH_ERR_SHAPE;
  *bytes = (size_t)km_plan(fmt, n, k, n_samples).total;
  return SPH_OK;
}

sph_status sph_kmeans_codebook(const sph_format* fmt, int64_t n, int64_t k, const float* d_w, int64_t ldw,
                               const double* d_u, int64_t n_samples, int32_t iters,
                               const uint16_t* d_init, uint16_t* d_codebook, double* d_objective,
                               int64_t* d_sample_idx, void* d_ws, size_t ws_bytes, void* stream) {
  if (!fmt || !d_u || !d_init || !d_codebook || !d_ws) return SPH_ERR_NULL;
  const int st = check_common(fmt, n, k, d_w, ldw);
  if (st) return (sph_status)st;
  if (n_samples < 1 || n_samples > kMaxSamples || iters < 0 || iters > kMaxIters) return SPH_ERR_SHAPE;
  if ((uintptr_t)d_u % 8 || (uintptr_t)d_init % 2 || (uintptr_t)d_codebook % 2 ||
      (uintptr_t)d_objective % 8 || (uintptr_t)d_sample_idx % 8 || (uintptr_t)d_ws % 256)
    return SPH_ERR_SHAPE;
  const KmPlan P = km_plan(fmt, n, k, n_samples);
  if (ws_bytes < P.total) return SPH_ERR_BUFFER_TOO_SMALL;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)d_ws;
  double* cdf = (double*)(ws + P.off_cdf);
  double* bsum = (double*)(ws + P.off_bsum);
  double* ds = (double*)(ws + P.off_ds);
  int32_t* z = (int32_t*)(ws + P.off_z);
  double* opart = (double*)(ws + P.off_opart);
  double* cen = (double*)(ws + P.off_cen);
  unsigned long long* acc = (unsigned long long*)(ws + P.off_acc);
  double* sbest = (double*)(ws + P.off_sbest);
  int32_t* sidx = (int32_t*)(ws + P.off_sidx);
  const int64_t ns = n_samples, nv = k / SPH_VEC, ncb8 = (int64_t)P.ncb * 8;
  const dim3 blk(kThreads);
  const unsigned g_cb = (unsigned)((ncb8 + kThreads - 1) / kThreads);
  const unsigned g_s = (unsigned)((ns + kThreads - 1) / kThreads);
  bool ok = launch_ok((const void*)k_r2, dim3((unsigned)P.nb), blk, s, d_w, ldw, nv, P.nvec, cdf, bsum) &&
            launch_ok((const void*)k_scan_blocks, dim3(1), blk, s, bsum, P.nb) &&
            launch_ok((const void*)k_scan_apply, dim3((unsigned)P.nb), blk, s, cdf, (const double*)bsum, P.nvec) &&
            launch_ok((const void*)k_sample, dim3(g_s), blk, s, d_w, ldw, nv, P.nvec, (const double*)cdf, d_u, ns,
                      ds, d_sample_idx) &&
            launch_ok((const void*)k_init_centres, dim3(g_cb), blk, s, d_init, ncb8, cen);
  const dim3 g_split((unsigned)P.nab, (unsigned)P.nsplit);
  for (int32_t it = 0; ok && it <= iters; ++it) {
    ok = launch_ok((const void*)k_assign_split, g_split, blk, s, (const double*)ds, ns, (const double*)cen, P.ncb,
                   P.per, sbest, sidx) &&
         launch_ok((const void*)k_assign_final, dim3((unsigned)P.nfb), blk, s, (const double*)ds, ns,
                   (const double*)cen, P.nsplit, (const double*)sbest, (const int32_t*)sidx, z, opart);
    if (ok && d_objective)
      ok = launch_ok((const void*)k_objective, dim3(1), dim3(64), s, (const double*)opart, P.nfb,
                     d_objective + it);
    if (ok && it < iters)
      ok = launch_ok((const void*)k_accumulate, dim3((unsigned)P.nr, (unsigned)P.np), blk, s, (const double*)ds, ns,
                     (const int32_t*)z, P.ncb, P.ch, acc) &&
           launch_ok((const void*)k_update, dim3((unsigned)P.ncb), dim3(64), s, (const unsigned long long*)acc, P.np,
                     P.ncb, cen);
  }
  if (ok) ok = launch_ok((const void*)k_centres_to_f16, dim3(g_cb), blk, s, (const double*)cen, ncb8, d_codebook);
  return ok ? SPH_OK : SPH_ERR_HIP;
}

}  // extern "C"
