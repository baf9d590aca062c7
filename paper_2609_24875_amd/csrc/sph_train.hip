// Training side of SPHQuant on the device: the angular codebook (Sec. 3.3, Eq. 9-10) and the
// pseudo-quantised weight of a linear module (Sec. 3.3; App. A steps 7-8 and 10): radius
// r = softplus(rho), group-wise V-bit fake quantisation with a straight-through estimator, and
// w^_i = r^_i s_i (.) c_{z_i}. The radius, its group offset and step (rounded to fp16, as the
// finalised codes store them) and the level are computed in fp64, so each level is decided in
// fp64; weights, gradients and the angular codebook are fp32, the precision of the fine-tuning.
//
// Work layout:
//   angular kernels   one thread per codebook entry (at most 8192).
//   fake quantisation one thread per 8-D vector; 16 neighbouring lanes form one 128-weight group
//                     (groups never straddle a row and start at multiples of 16).
//   radius gradient   one thread per vector, coalesced over dL/dW^.
//   codebook gradient no atomics: the vectors are pre-sorted by direction (a stable counting
//                     sort on the host, once per module, since the indices stay fixed); block
//                     (c, s) sums slice s of centre c's list in order and a fixed lane tree, and
//                     a second kernel adds the slices in order. Repeated calls are bitwise equal.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "sph_fp.h"
#include "sph_host.h"
#include "sph_layout.h"

namespace {

constexpr int kThreads = 256;
constexpr float kHalfPi = 1.57079632679489662f;
constexpr int kTargetBlocks = 1024;
constexpr int kMaxSlices = 64;

__device__ __forceinline__ float sigmoidf(float x) { return 1.0f / (1.0f + expf(-x)); }

// softplus in fp64 as log(e^0 + e^x) without overflow: log1p(e^x) for x < 0, x + log1p(e^-x) for
// x > 0, log 2 at 0
__device__ __forceinline__ double softplus_d(double x) {
  if (x < 0.0) return log1p(exp(x));
  if (x > 0.0) return x + log1p(exp(-x));
  return 0.69314718055994530942;
}

__device__ __forceinline__ float sum8_pairwise(const float* p) {
  return ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
}

// ------------------------------------------------------------------ angular codebook (Eq. 9-10)

// c = C(theta(phi)) for each entry: theta_j = eps + (pi/2 - 2 eps) sigmoid(phi_j),
// c_1 = cos t_1, c_i = (prod_{j<i} sin t_j) cos t_i, c_8 = prod_j sin t_j.
__global__ __launch_bounds__(kThreads) void k_angular_fwd(const float* __restrict__ phi, int ncb, float eps,
                                                          float* __restrict__ cb) {
  const int e = blockIdx.x * kThreads + threadIdx.x;
  if (e >= ncb) return;
  const float span = kHalfPi - 2.0f * eps;
  float sprod = 1.0f;
#pragma unroll
  for (int j = 0; j < 7; ++j) {
    float s, c;
    sincosf(eps + span * sigmoidf(phi[e * 7 + j]), &s, &c);
    cb[e * 8 + j] = sprod * c;
    sprod *= s;
  }
  cb[e * 8 + 7] = sprod;
}

// dL/dphi from dL/dc: dc_i/dt_j = c_i cot t_j for j < i (including c_8), -(prod_{k<i} sin t_k)
// sin t_i for j = i <= 7, and 0 for j > i; dt_j/dphi_j = (pi/2 - 2 eps) s (1 - s).
__global__ __launch_bounds__(kThreads) void k_angular_bwd(const float* __restrict__ phi, int ncb, float eps,
                                                          const float* __restrict__ gc, float* __restrict__ gphi) {
  const int e = blockIdx.x * kThreads + threadIdx.x;
  if (e >= ncb) return;
  const float span = kHalfPi - 2.0f * eps;
  float sg[7], sn[7], cs[7], c[8], pre[7];
  float sprod = 1.0f;
#pragma unroll
  for (int j = 0; j < 7; ++j) {
    sg[j] = sigmoidf(phi[e * 7 + j]);
    sincosf(eps + span * sg[j], &sn[j], &cs[j]);
    pre[j] = sprod;
    c[j] = sprod * cs[j];
    sprod *= sn[j];
  }
  c[7] = sprod;
  float g[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) g[i] = gc[e * 8 + i];
  float later = g[7] * c[7];  // sum over i > j of g_i c_i, built from the back
#pragma unroll
  for (int j = 6; j >= 0; --j) {
    const float dth = later * cs[j] / sn[j] - g[j] * pre[j] * sn[j];
    gphi[e * 7 + j] = dth * span * sg[j] * (1.0f - sg[j]);
    later += g[j] * c[j];
  }
}

// Inverse of Eq. 9-10 for a non-negative unit direction: theta_i = atan2(||c_{i+1..8}||, c_i),
// t = clamp((theta - eps) / (pi/2 - 2 eps), 1e-6, 1 - 1e-6), phi = log t - log(1 - t).
__global__ __launch_bounds__(kThreads) void k_angular_logits(const float* __restrict__ cb, int ncb, float eps,
                                                             float* __restrict__ phi) {
  const int e = blockIdx.x * kThreads + threadIdx.x;
  if (e >= ncb) return;
  const float span = kHalfPi - 2.0f * eps;
  float c[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) c[i] = cb[e * 8 + i];
  float tail2 = c[7] * c[7];
#pragma unroll
  for (int j = 6; j >= 0; --j) {
    const float th = atan2f(sqrtf(tail2), c[j]);
    const float t = fminf(fmaxf((th - eps) / span, 1e-6f), 1.0f - 1e-6f);
    phi[e * 7 + j] = logf(t) - log1pf(-t);
    tail2 += c[j] * c[j];
  }
}

// ------------------------------------------------------------------ pseudo-quantised weights

struct FqArgs {
  int64_t nv, nvec;
  const float* rho;
  const uint8_t* signs;
  const uint16_t* dir;
  const float* cb;
  int vmax;
  float* w_hat;
  int64_t ldw;
  float* r_hat;
  uint8_t* q;
  uint16_t* gmin;
  uint16_t* gstep;
};

// r = softplus(rho); per group of 16 vectors the offset min r and the step (max - min)/(2^V - 1),
// both rounded to fp16; q = clip(round((r - min)/step), 0, 2^V - 1), half to even (0 for a zero
// step); r^ = min + q step; w^ = r^ s (.) c_z. All of it in fp64, then w^ and r^ stored as fp32.
// Optional outputs: r^, and the finalised codes (levels, fp16 offsets and steps).
__global__ __launch_bounds__(kThreads) void k_fq_forward(FqArgs a) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const bool ok = i < a.nvec;  // whole groups are inside or outside together
  const double r = ok ? softplus_d((double)a.rho[i]) : 0.0;
  double lo = r, hi = r;
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) {
    lo = fmin(lo, __shfl_xor(lo, o, 16));
    hi = fmax(hi, __shfl_xor(hi, o, 16));
  }
  const uint16_t lo16 = d2h(lo), st16 = d2h((hi - lo) / (double)a.vmax);
  const double lod = h2d(lo16), std_ = h2d(st16);
  int q = 0;
  if (std_ > 0.0) q = (int)fmin(fmax(rint((r - lod) / std_), 0.0), (double)a.vmax);
  const double rh = lod + (double)q * std_;
  if (!ok) return;
  const int64_t row = i / a.nv, v = i - row * a.nv;
  const uint32_t s = a.signs[i];
  const float4* c4 = reinterpret_cast<const float4*>(a.cb + (int64_t)a.dir[i] * 8);
  const float4 c0 = c4[0], c1 = c4[1];
  const float cc[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
  float w[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float m = (float)(rh * (double)cc[j]);
    w[j] = ((s >> j) & 1) ? -m : m;
  }
  float4* out = reinterpret_cast<float4*>(a.w_hat + row * a.ldw + v * 8);
  out[0] = make_float4(w[0], w[1], w[2], w[3]);
  out[1] = make_float4(w[4], w[5], w[6], w[7]);
  if (a.r_hat) a.r_hat[i] = (float)rh;
  if (a.q) a.q[i] = (uint8_t)q;
  if (a.gmin && (threadIdx.x & 15) == 0) {
    a.gmin[i >> 4] = lo16;
    a.gstep[i >> 4] = st16;
  }
}

// rho from Eq. 6's radius r~ = <|w|, c_z> (floored at 1e-6) through the inverse of softplus.
__global__ __launch_bounds__(kThreads) void k_fq_init_rho(const float* __restrict__ w, int64_t ldw, int64_t nv,
                                                          int64_t nvec, const uint16_t* __restrict__ dir,
                                                          const float* __restrict__ cb, float* __restrict__ rho) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= nvec) return;
  const int64_t row = i / nv, v = i - row * nv;
  const float4* p = reinterpret_cast<const float4*>(w + row * ldw + v * 8);
  const float4* c4 = reinterpret_cast<const float4*>(cb + (int64_t)dir[i] * 8);
  const float4 x0 = p[0], x1 = p[1], c0 = c4[0], c1 = c4[1];
  const float pr[8] = {fabsf(x0.x) * c0.x, fabsf(x0.y) * c0.y, fabsf(x0.z) * c0.z, fabsf(x0.w) * c0.w,
                       fabsf(x1.x) * c1.x, fabsf(x1.y) * c1.y, fabsf(x1.z) * c1.z, fabsf(x1.w) * c1.w};
  const float rt = fmaxf(sum8_pairwise(pr), 1e-6f);
  rho[i] = rt > 20.0f ? rt + log1pf(-expf(-rt)) : logf(expm1f(rt));
}

// dL/drho_i = sigmoid(rho_i) * sum_j dL/dw^_ij s_ij c_{z_i, j} (straight-through: dr^/dr = 1).
__global__ __launch_bounds__(kThreads) void k_fq_grad_rho(int64_t nv, int64_t nvec, const float* __restrict__ rho,
                                                          const uint8_t* __restrict__ signs,
                                                          const uint16_t* __restrict__ dir,
                                                          const float* __restrict__ cb, const float* __restrict__ gw,
                                                          int64_t ldg, float* __restrict__ grho) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= nvec) return;
  const int64_t row = i / nv, v = i - row * nv;
  const float4* g4 = reinterpret_cast<const float4*>(gw + row * ldg + v * 8);
  const float4* c4 = reinterpret_cast<const float4*>(cb + (int64_t)dir[i] * 8);
  const float4 g0 = g4[0], g1 = g4[1], c0 = c4[0], c1 = c4[1];
  const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
  const float c[8] = {c0.x, c0.y, c0.z, c0.w, c1.x, c1.y, c1.z, c1.w};
  const uint32_t s = signs[i];
  float p[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) p[j] = ((s >> j) & 1) ? -g[j] * c[j] : g[j] * c[j];
  grho[i] = sum8_pairwise(p) * sigmoidf(rho[i]);
}

// Slice s of centre c's direction-sorted vector list: sum of r^_i s_i (.) dL/dw^_i in list order
// per thread, then a fixed tree over the block.
__global__ __launch_bounds__(kThreads) void k_fq_grad_cb_part(int64_t nv, const float* __restrict__ r_hat,
                                                              const uint8_t* __restrict__ signs,
                                                              const float* __restrict__ gw, int64_t ldg,
                                                              const int32_t* __restrict__ perm,
                                                              const int64_t* __restrict__ off, int nslice,
                                                              float* __restrict__ part) {
  __shared__ float sh[kThreads / 64][8];
  const int c = blockIdx.x, sl = blockIdx.y;
  const int64_t a0 = off[c], len = off[c + 1] - a0;
  const int64_t b0 = a0 + len * sl / nslice, b1 = a0 + len * (sl + 1) / nslice;
  float acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (int64_t t = b0 + threadIdx.x; t < b1; t += kThreads) {
    const int64_t i = perm[t];
    const int64_t row = i / nv, v = i - row * nv;
    const float4* g4 = reinterpret_cast<const float4*>(gw + row * ldg + v * 8);
    const float4 g0 = g4[0], g1 = g4[1];
    const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
    const float rh = r_hat[i];
    const uint32_t s = signs[i];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] += ((s >> j) & 1) ? -rh * g[j] : rh * g[j];
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] += __shfl_xor(acc[j], o, 64);
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < 8; ++j) sh[wv][j] = acc[j];
  }
  __syncthreads();
  if (threadIdx.x < 8) {
    const int j = threadIdx.x;
    part[((int64_t)c * nslice + sl) * 8 + j] = (sh[0][j] + sh[1][j]) + (sh[2][j] + sh[3][j]);
  }
}

__global__ __launch_bounds__(kThreads) void k_fq_grad_cb_final(const float* __restrict__ part, int ncb, int nslice,
                                                               float* __restrict__ gcb) {
  const int t = blockIdx.x * kThreads + threadIdx.x;
  if (t >= ncb * 8) return;
  const int c = t >> 3, j = t & 7;
  float s = 0.0f;
  for (int sl = 0; sl < nslice; ++sl) s += part[((int64_t)c * nslice + sl) * 8 + j];
  gcb[t] = s;
}

// ------------------------------------------------------------------------------------ host side

int slices_for(int ncb) { return std::max(1, std::min(kMaxSlices, (kTargetBlocks + ncb - 1) / ncb)); }

template <typename... A>
bool launch_ok(const void* fn, dim3 grid, dim3 block, hipStream_t s, A... args) {
  void* kargs[] = {(void*)&args...};
  if (hipLaunchKernel(fn, grid, block, kargs, 0, s) != hipSuccess) return false;
  return hipGetLastError() == hipSuccess;
}

bool dir_bits_ok(int32_t d) { return d >= 1 && d <= 13; }

// The fine-tuning kernels handle 8-D vectors (the 4-D and 16-D formats are decode-only).
int check_fq(const sph_format* fmt, int64_t n, int64_t k) {
  int st = sph_host_check_format(fmt);
  if (st) return st;
  if (fmt->vec_dim != SPH_VEC) return SPH_ERR_UNSUPPORTED_FORMAT;
  return sph_host_check_shape(n, k);
}

bool a16(const void* p) { return (uintptr_t)p % 16 == 0; }

}  // namespace

extern "C" {

sph_status sph_angular_codebook(int32_t dir_bits, const float* d_phi, float eps, float* d_codebook, void* stream) {
  if (!d_phi || !d_codebook) return SPH_ERR_NULL;
  if (!dir_bits_ok(dir_bits) || !(eps >= 0.0f && eps < 0.25f)) return SPH_ERR_SHAPE;
  const int ncb = 1 << dir_bits;
  return launch_ok((const void*)k_angular_fwd, dim3((ncb + kThreads - 1) / kThreads), dim3(kThreads),
                   (hipStream_t)stream, d_phi, ncb, eps, d_codebook)
             ? SPH_OK
             : SPH_ERR_HIP;
}

sph_status sph_angular_codebook_backward(int32_t dir_bits, const float* d_phi, float eps, const float* d_grad_codebook,
                                         float* d_grad_phi, void* stream) {
  if (!d_phi || !d_grad_codebook || !d_grad_phi) return SPH_ERR_NULL;
  if (!dir_bits_ok(dir_bits) || !(eps >= 0.0f && eps < 0.25f)) return SPH_ERR_SHAPE;
  const int ncb = 1 << dir_bits;
  return launch_ok((const void*)k_angular_bwd, dim3((ncb + kThreads - 1) / kThreads), dim3(kThreads),
                   (hipStream_t)stream, d_phi, ncb, eps, d_grad_codebook, d_grad_phi)
             ? SPH_OK
             : SPH_ERR_HIP;
}

sph_status sph_angular_logits(int32_t dir_bits, const float* d_codebook, float eps, float* d_phi, void* stream) {
  if (!d_phi || !d_codebook) return SPH_ERR_NULL;
  if (!dir_bits_ok(dir_bits) || !(eps >= 0.0f && eps < 0.25f)) return SPH_ERR_SHAPE;
  const int ncb = 1 << dir_bits;
  return launch_ok((const void*)k_angular_logits, dim3((ncb + kThreads - 1) / kThreads), dim3(kThreads),
                   (hipStream_t)stream, d_codebook, ncb, eps, d_phi)
             ? SPH_OK
             : SPH_ERR_HIP;
}

sph_status sph_direction_groups(int32_t dir_bits, int64_t count, const uint16_t* dir_idx, int32_t* perm,
                                int64_t* offsets) {
  if (!dir_idx || !perm || !offsets) return SPH_ERR_NULL;
  if (!dir_bits_ok(dir_bits) || count < 1 || count > INT32_MAX) return SPH_ERR_SHAPE;
  const int64_t ncb = int64_t(1) << dir_bits;
  std::vector<int64_t> cnt(ncb + 1, 0);
  for (int64_t i = 0; i < count; ++i) {
    if (dir_idx[i] >= ncb) return SPH_ERR_CODE_RANGE;
    ++cnt[dir_idx[i] + 1];
  }
  for (int64_t c = 0; c < ncb; ++c) cnt[c + 1] += cnt[c];
  for (int64_t c = 0; c <= ncb; ++c) offsets[c] = cnt[c];
  for (int64_t i = 0; i < count; ++i) perm[cnt[dir_idx[i]]++] = (int32_t)i;
  return SPH_OK;
}

sph_status sph_fake_quant_init_rho(const sph_format* fmt, int64_t n, int64_t k, const float* d_w, int64_t ldw,
                                   const uint16_t* d_dir_idx, const float* d_codebook, float* d_rho, void* stream) {
  if (!fmt || !d_w || !d_dir_idx || !d_codebook || !d_rho) return SPH_ERR_NULL;
  const int st = check_fq(fmt, n, k);
  if (st) return (sph_status)st;
  if (ldw < k || ldw % 4 || !a16(d_w) || !a16(d_codebook) || (uintptr_t)d_dir_idx % 2 || (uintptr_t)d_rho % 4)
    return SPH_ERR_SHAPE;
  const int64_t nv = k / SPH_VEC, nvec = n * nv;
  return launch_ok((const void*)k_fq_init_rho, dim3((unsigned)((nvec + kThreads - 1) / kThreads)), dim3(kThreads),
                   (hipStream_t)stream, d_w, ldw, nv, nvec, d_dir_idx, d_codebook, d_rho)
             ? SPH_OK
             : SPH_ERR_HIP;
}

sph_status sph_fake_quant_forward(const sph_format* fmt, int64_t n, int64_t k, const float* d_rho,
                                  const uint8_t* d_signs, const uint16_t* d_dir_idx, const float* d_codebook,
                                  float* d_w_hat, int64_t ldw, float* d_r_hat, uint8_t* d_radius_code,
                                  uint16_t* d_group_min, uint16_t* d_group_step, void* stream) {
  if (!fmt || !d_rho || !d_signs || !d_dir_idx || !d_codebook || !d_w_hat) return SPH_ERR_NULL;
  const int st = check_fq(fmt, n, k);
  if (st) return (sph_status)st;
  if ((d_radius_code || d_group_min || d_group_step) && !(d_radius_code && d_group_min && d_group_step))
    return SPH_ERR_NULL;
  if (ldw < k || ldw % 4 || !a16(d_w_hat) || !a16(d_codebook) || (uintptr_t)d_rho % 4 || (uintptr_t)d_dir_idx % 2 ||
      (uintptr_t)d_r_hat % 4 || (uintptr_t)d_group_min % 2 || (uintptr_t)d_group_step % 2)
    return SPH_ERR_SHAPE;
  FqArgs a{};
  a.nv = k / SPH_VEC;
  a.nvec = n * a.nv;
  a.rho = d_rho;
  a.signs = d_signs;
  a.dir = d_dir_idx;
  a.cb = d_codebook;
  a.vmax = (1 << fmt->radius_bits) - 1;
  a.w_hat = d_w_hat;
  a.ldw = ldw;
  a.r_hat = d_r_hat;
  a.q = d_radius_code;
  a.gmin = d_group_min;
  a.gstep = d_group_step;
  return launch_ok((const void*)k_fq_forward, dim3((unsigned)((a.nvec + kThreads - 1) / kThreads)), dim3(kThreads),
                   (hipStream_t)stream, a)
             ? SPH_OK
             : SPH_ERR_HIP;
}

sph_status sph_fake_quant_backward_workspace_bytes(int32_t dir_bits, size_t* bytes) {
  if (!bytes) return SPH_ERR_NULL;
  if (!dir_bits_ok(dir_bits)) return SPH_ERR_SHAPE;
  const int ncb = 1 << dir_bits;
  *bytes = (size_t)ncb * slices_for(ncb) * 8 * sizeof(float);
  return SPH_OK;
}

sph_status sph_fake_quant_backward(const sph_format* fmt, int64_t n, int64_t k, const float* d_rho,
                                   const uint8_t* d_signs, const uint16_t* d_dir_idx, const float* d_codebook,
                                   const float* d_r_hat, const float* d_grad_w, int64_t ldg, const int32_t* d_perm,
                                   const int64_t* d_offsets, float* d_grad_rho, float* d_grad_codebook, void* d_ws,
                                   size_t ws_bytes, void* stream) {
  if (!fmt || !d_rho || !d_signs || !d_dir_idx || !d_codebook || !d_r_hat || !d_grad_w || !d_perm || !d_offsets ||
      !d_grad_rho || !d_grad_codebook || !d_ws)
    return SPH_ERR_NULL;
  const int st = check_fq(fmt, n, k);
  if (st) return (sph_status)st;
  if (ldg < k || ldg % 4 || !a16(d_grad_w) || !a16(d_codebook) || (uintptr_t)d_rho % 4 || (uintptr_t)d_r_hat % 4 ||
      (uintptr_t)d_dir_idx % 2 || (uintptr_t)d_perm % 4 || (uintptr_t)d_offsets % 8 || (uintptr_t)d_grad_rho % 4 ||
      (uintptr_t)d_grad_codebook % 4 || (uintptr_t)d_ws % 16)
    return SPH_ERR_SHAPE;
  const int ncb = 1 << fmt->dir_bits, ns = slices_for(ncb);
  if (ws_bytes < (size_t)ncb * ns * 8 * sizeof(float)) return SPH_ERR_BUFFER_TOO_SMALL;
  const int64_t nv = k / SPH_VEC, nvec = n * nv;
  hipStream_t s = (hipStream_t)stream;
  float* part = (float*)d_ws;
  const bool ok =
      launch_ok((const void*)k_fq_grad_rho, dim3((unsigned)((nvec + kThreads - 1) / kThreads)), dim3(kThreads), s, nv,
                nvec, d_rho, d_signs, d_dir_idx, d_codebook, d_grad_w, ldg, d_grad_rho) &&
      launch_ok((const void*)k_fq_grad_cb_part, dim3((unsigned)ncb, (unsigned)ns), dim3(kThreads), s, nv, d_r_hat,
                d_signs, d_grad_w, ldg, d_perm, d_offsets, ns, part) &&
      launch_ok((const void*)k_fq_grad_cb_final, dim3((unsigned)((ncb * 8 + kThreads - 1) / kThreads)), dim3(kThreads),
                s, (const float*)part, ncb, ns, d_grad_codebook);
  return ok ? SPH_OK : SPH_ERR_HIP;
}

}  // extern "C"
