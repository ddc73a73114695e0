// ss_aux.hip -- verification assembly, the materialising pass of
// ss_process_logits and the workspace fill kernel.
#include "ss_impl.hpp"
#include "ss_launch.hpp"

namespace ss {

// row's correction (or the bonus token), then -1.
__global__ __launch_bounds__(kBlock) void ss_assemble_kernel(KArgs a) {
  const int b = blockIdx.x * kBlock + threadIdx.x;
  if (b >= a.B) return;
  const int L = a.L;
  int n = 0;
  int fl = 0;
  int32_t* out = a.out_tokens + (size_t)b * (L + 1);
  int l = 0;
  for (; l <= L; ++l) {
    const RowResult rr = a.res[(size_t)b * (L + 1) + l];
    fl |= rr.flags;
    if (l < L && rr.accept) {
      out[l] = a.draft_tokens[(size_t)b * L + l];
      ++n;
      continue;
    }
    out[l] = rr.emit;
    ++l;
    break;
  }
  for (; l <= L; ++l) out[l] = -1;
  a.out_nacc[b] = n;
  if (a.flags) a.flags[b] = fl;
}

__global__ void ss_zero_kernel(uint32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}
template <int DT>
void launch_materialize(const KArgs& k, dim3 grid, dim3 block, hipStream_t st) {
  hipLaunchKernelGGL(ss_materialize_kernel<DT>, grid, block, 0, st, k);
}
template void launch_materialize<SS_F32>(const KArgs&, dim3, dim3, hipStream_t);
template void launch_materialize<SS_BF16>(const KArgs&, dim3, dim3, hipStream_t);

void launch_assemble(const KArgs& k, dim3 grid, dim3 block, hipStream_t st) {
  hipLaunchKernelGGL(ss_assemble_kernel, grid, block, 0, st, k);
}
void launch_zero(uint32_t* p, size_t n, dim3 grid, dim3 block, hipStream_t st) {
  hipLaunchKernelGGL(ss_zero_kernel, grid, block, 0, st, p, n);
}

}  // namespace ss
