// hbm_read.hip -- a pure streaming read of a device buffer, used by bench.py to measure the
// HBM read ceiling that the GEMV's bandwidth is compared with. Not part of the LogbQuant path.
//
// Every wavefront reads 4 KiB units (four 1 KiB non-temporal 128-bit buffer loads, one per
// 64 lanes x 16 bytes) with one unit in flight ahead of the one being consumed, the access
// pattern and prefetch depth of the M = 1 GEMV. The data is folded into a register and written
// only if it equals a value it cannot take for the inputs bench.py uses, so the kernel stores
// nothing in practice while the compiler cannot drop the loads.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnit = 4096;

__global__ __launch_bounds__(512) void k_read(const uint8_t* __restrict__ buf, int64_t units,
                                              uint32_t* __restrict__ sink) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t gw = (int64_t)blockIdx.x * 8 + wave;
  const int64_t nw = (int64_t)gridDim.x * 8;
  auto load = [&](int64_t u, u32x4 (&q)[4]) {
    const bool live = u < units;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(buf + (live ? u * kUnit : 0)), (short)0, live ? kUnit : 0, 0x00020000);
#pragma unroll
    for (int i = 0; i < 4; ++i) q[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, 16 * lane + 1024 * i, 0, 2);
  };
  u32x4 a[4], b[4];
  uint32_t acc = 0;
  load(gw, a);
  for (int64_t u = gw; u < units; u += 2 * nw) {
    load(u + nw, b);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc ^= a[i].x ^ a[i].y ^ a[i].z ^ a[i].w;
    load(u + 2 * nw, a);
    if (u + nw < units) {
#pragma unroll
      for (int i = 0; i < 4; ++i) acc ^= b[i].x ^ b[i].y ^ b[i].z ^ b[i].w;
    }
  }
  if (acc == 0x9E3779B9u) sink[(int64_t)blockIdx.x * 512 + threadIdx.x] = acc;
}

}  // namespace

// Reads `bytes` (a multiple of 4096) from device buffer `buf` once. `sink` is a device buffer
// of grid * 512 uint32 (grid = the number of compute units) that is written only in the case
// described above. Returns 0, or 1 on a bad argument, 2 on a launch failure.
extern "C" int32_t hbm_read(const void* buf, int64_t bytes, uint32_t* sink, int32_t grid,
                            void* stream) {
  if (!buf || !sink || bytes <= 0 || bytes % kUnit != 0 || grid <= 0) return 1;
  hipLaunchKernelGGL(k_read, dim3((unsigned)grid), dim3(512), 0, (hipStream_t)stream,
                     (const uint8_t*)buf, bytes / kUnit, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
