// ss_merge.hip -- one instantiation of the row merge kernel, chosen at compile
// time by SS_MERGE_DT (element type) and SS_MERGE_OP (operation); the build
// compiles this file once per pair so the instantiations compile in parallel.
#include "ss_impl.hpp"
#include "ss_launch.hpp"

#if !defined(SS_MERGE_DT) || !defined(SS_MERGE_OP)
#error "SS_MERGE_DT and SS_MERGE_OP select the merge instantiation"
#endif

namespace ss {

template <int DT, int OP>
void launch_merge(const KArgs& k, dim3 grid, dim3 block, int smem, hipStream_t st) {
  hipLaunchKernelGGL((ss_merge_kernel<DT, OP>), grid, block, smem, st, k);
}
template <int DT, int OP>
hipError_t merge_smem_limit(int bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&ss_merge_kernel<DT, OP>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}
template void launch_merge<SS_MERGE_DT, SS_MERGE_OP>(const KArgs&, dim3, dim3, int, hipStream_t);
template hipError_t merge_smem_limit<SS_MERGE_DT, SS_MERGE_OP>(int);

}  // namespace ss
