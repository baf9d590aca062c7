// Measurement probe, built as its own library (libsph_probe.so) and used by the benchmark only:
// a plain streaming read of a device buffer, the practical HBM read ceiling that the decode
// kernels' packed-weight bandwidth is compared with next to the nominal 8 TB/s.
//
// Three access patterns, so that the ceiling does not rest on one of them:
//  0. grid stride: every thread walks the buffer in a grid-stride loop with four independent
//     16-byte loads in flight per iteration (each wave's four loads lie a grid apart);
//  1. wave blocks: every wave reads contiguous 8 KiB blocks (eight 1 KiB loads in flight), the
//     blocks of consecutive waves adjacent, strided by all the waves of the grid;
//  2. workgroup slices: workgroup b reads the contiguous slice b of `grid` equal slices, 16 KiB
//     per iteration (four 4 KiB loads of the workgroup in flight).
// Loads are folded with XOR; the fold is stored only if it equals a run-time value the data
// never produces, so the loads cannot be removed and nothing is written.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int PROBE_THREADS = 256;

__global__ void __launch_bounds__(PROBE_THREADS) k_probe_read(const uint4* __restrict__ p, uint64_t n16,
                                                              uint32_t* __restrict__ flag, uint32_t never) {
  const uint64_t stride = (uint64_t)gridDim.x * PROBE_THREADS;
  uint64_t i = (uint64_t)blockIdx.x * PROBE_THREADS + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const uint4 a = p[i], b = p[i + stride], c = p[i + 2 * stride], d = p[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n16; i += stride) {
    const uint4 a = p[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  if (acc == never) flag[0] = acc;   // the caller picks a value the fold cannot take
}

__global__ void __launch_bounds__(PROBE_THREADS) k_probe_read_blocks(const uint4* __restrict__ p, uint64_t n16,
                                                                     uint32_t* __restrict__ flag, uint32_t never) {
  constexpr int PER = 8;   // 1 KiB loads per wave block
  const int lane = threadIdx.x & 63;
  const uint64_t wave = (uint64_t)blockIdx.x * (PROBE_THREADS / 64) + (threadIdx.x >> 6);
  const uint64_t waves = (uint64_t)gridDim.x * (PROBE_THREADS / 64);
  const uint64_t nblk = n16 / (64 * PER);
  uint32_t acc = 0;
  for (uint64_t blk = wave; blk < nblk; blk += waves) {
    const uint4* q = p + blk * 64 * PER + lane;
    uint4 v[PER];
#pragma unroll
    for (int j = 0; j < PER; ++j) v[j] = q[64 * j];
#pragma unroll
    for (int j = 0; j < PER; ++j) acc ^= v[j].x ^ v[j].y ^ v[j].z ^ v[j].w;
  }
  // the tail past whole blocks, by the first wave
  for (uint64_t i = nblk * 64 * PER + (wave == 0 ? (uint64_t)lane : n16); i < n16; i += 64) {
    const uint4 a = p[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  if (acc == never) flag[0] = acc;
}

__global__ void __launch_bounds__(PROBE_THREADS) k_probe_read_slices(const uint4* __restrict__ p, uint64_t n16,
                                                                     uint32_t* __restrict__ flag, uint32_t never) {
  const uint64_t per = (n16 + gridDim.x - 1) / gridDim.x;   // 16-byte words per slice
  const uint64_t b0 = (uint64_t)blockIdx.x * per, b1 = b0 + per < n16 ? b0 + per : n16;
  uint32_t acc = 0;
  uint64_t i = b0 + threadIdx.x;
  for (; i + 3 * PROBE_THREADS < b1; i += 4 * PROBE_THREADS) {
    const uint4 a = p[i], b = p[i + PROBE_THREADS], c = p[i + 2 * PROBE_THREADS], d = p[i + 3 * PROBE_THREADS];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < b1; i += PROBE_THREADS) {
    const uint4 a = p[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  if (acc == never) flag[0] = acc;
}

}  // namespace

// Reads `bytes` (a multiple of 16, 16-byte aligned) from d_buf with `grid` workgroups of 256
// threads on `stream`, in access pattern `pattern` (0, 1 or 2, above). d_flag: one device word,
// written only if a thread's XOR fold of its words equals `never` (the caller fills the buffer so
// that it cannot). Returns 0 on success, 1 on a bad argument, 2 on a launch error.
extern "C" int sph_probe_stream_read(const void* d_buf, size_t bytes, int grid, int pattern, void* d_flag,
                                     uint32_t never, void* stream) {
  if (!d_buf || !d_flag || bytes % 16 != 0 || (uintptr_t)d_buf % 16 != 0 || grid < 1 || pattern < 0 ||
      pattern > 2)
    return 1;
  const auto fn = pattern == 0 ? k_probe_read : pattern == 1 ? k_probe_read_blocks : k_probe_read_slices;
  hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(PROBE_THREADS), 0, (hipStream_t)stream, (const uint4*)d_buf,
                     (uint64_t)(bytes / 16), (uint32_t*)d_flag, never);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
