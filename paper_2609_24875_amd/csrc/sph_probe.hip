// Measurement probe, built as its own library (libsph_probe.so) and used by the benchmark only:
// a plain streaming read of a device buffer, the practical HBM read ceiling that the decode
// kernels' packed-weight bandwidth is compared with next to the nominal 8 TB/s.
//
// Every thread walks the buffer in a grid-stride loop with four independent 16-byte loads in
// flight per iteration and folds them with XOR; the fold is stored only if it equals a run-time
// value the data never produces, so the loads cannot be removed and nothing is written.
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

}  // namespace

// Reads `bytes` (a multiple of 16, 16-byte aligned) from d_buf with `grid` workgroups of 256
// threads on `stream`. d_flag: one device word, written only if a thread's XOR fold of its words
// equals `never` (the caller fills the buffer so that it cannot). Returns 0 on success, 1 on a
// bad argument, 2 on a launch error.
extern "C" int sph_probe_stream_read(const void* d_buf, size_t bytes, int grid, void* d_flag, uint32_t never,
                                     void* stream) {
  if (!d_buf || !d_flag || bytes % 16 != 0 || (uintptr_t)d_buf % 16 != 0 || grid < 1) return 1;
  hipLaunchKernelGGL(k_probe_read, dim3((unsigned)grid), dim3(PROBE_THREADS), 0, (hipStream_t)stream,
                     (const uint4*)d_buf, (uint64_t)(bytes / 16), (uint32_t*)d_flag, never);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
