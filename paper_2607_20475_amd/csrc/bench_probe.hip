// bench_probe.hip -- measurement aids of the benchmark, not part of the
// sampler library:
//   bench_read   a plain streaming read of a device buffer: the practical HBM
//                ceiling the sampler's streaming pass is compared with, and the
//                known byte count that scales the FETCH_SIZE counter;
//   bench_write  a plain streaming write of a known byte count, which scales
//                the WRITE_SIZE counter.
// The read folds every 16-byte word into one register and writes a word only
// when the fold equals a value the caller never passes, so its loads cannot
// be removed and it writes nothing.
#include <hip/hip_runtime.h>
#include <stdint.h>

__global__ __launch_bounds__(256) void bench_read_kernel(const uint4* __restrict__ p, size_t n, uint32_t never,
                                                         uint32_t* sink) {
  uint32_t acc = 0u;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const uint4 a = p[i], b = p[i + stride], c = p[i + 2 * stride], d = p[i + 3 * stride];
    acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
  }
  for (; i < n; i += stride) {
    const uint4 a = p[i];
    acc ^= a.x ^ a.y ^ a.z ^ a.w;
  }
  if (acc == never) sink[threadIdx.x] = acc;
}

__global__ __launch_bounds__(256) void bench_write_kernel(uint4* __restrict__ p, size_t n, uint32_t v) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = make_uint4(v, v, v, v);
}

// Reads `bytes` (a multiple of 16) from `p` on `stream` with `blocks` workgroups.
extern "C" int bench_read(const void* p, size_t bytes, int blocks, uint32_t never, uint32_t* sink, void* stream) {
  if (!p || !sink || (bytes & 15u) || blocks <= 0) return -1;
  hipLaunchKernelGGL(bench_read_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     reinterpret_cast<const uint4*>(p), bytes / 16, never, sink);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

// Writes `bytes` (a multiple of 16) to `p` on `stream` with `blocks` workgroups.
extern "C" int bench_write(void* p, size_t bytes, int blocks, uint32_t v, void* stream) {
  if (!p || (bytes & 15u) || blocks <= 0) return -1;
  hipLaunchKernelGGL(bench_write_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                     reinterpret_cast<uint4*>(p), bytes / 16, v);
  return hipGetLastError() == hipSuccess ? 0 : -2;
}
