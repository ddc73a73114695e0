// ss_launch.hpp -- host launchers of the kernels, one definition per
// translation unit (each kernel instantiation is compiled on its own).
#pragma once
#include <hip/hip_runtime.h>

namespace ss {

struct KArgs;

template <int DT, bool LP>
void launch_stream(const KArgs& k, dim3 grid, dim3 block, int smem, hipStream_t st);
template <int DT, int OP>
void launch_merge(const KArgs& k, dim3 grid, dim3 block, int smem, hipStream_t st);
template <int DT, int OP>
hipError_t merge_smem_limit(int bytes);
template <int DT>
void launch_materialize(const KArgs& k, dim3 grid, dim3 block, hipStream_t st);
void launch_assemble(const KArgs& k, dim3 grid, dim3 block, hipStream_t st);
void launch_zero(uint32_t* p, size_t n, dim3 grid, dim3 block, hipStream_t st);

#define SS_EXTERN_MERGE(DT, OP)                                                            \
  extern template void launch_merge<DT, OP>(const KArgs&, dim3, dim3, int, hipStream_t); \
  extern template hipError_t merge_smem_limit<DT, OP>(int);
SS_EXTERN_MERGE(0, 0)
SS_EXTERN_MERGE(0, 1)
SS_EXTERN_MERGE(0, 2)
SS_EXTERN_MERGE(0, 3)
SS_EXTERN_MERGE(0, 4)
SS_EXTERN_MERGE(0, 5)
SS_EXTERN_MERGE(1, 0)
SS_EXTERN_MERGE(1, 1)
SS_EXTERN_MERGE(1, 2)
SS_EXTERN_MERGE(1, 3)
SS_EXTERN_MERGE(1, 4)
SS_EXTERN_MERGE(1, 5)
#undef SS_EXTERN_MERGE
extern template void launch_stream<0, false>(const KArgs&, dim3, dim3, int, hipStream_t);
extern template void launch_stream<1, false>(const KArgs&, dim3, dim3, int, hipStream_t);
extern template void launch_stream<0, true>(const KArgs&, dim3, dim3, int, hipStream_t);
extern template void launch_stream<1, true>(const KArgs&, dim3, dim3, int, hipStream_t);
extern template void launch_materialize<0>(const KArgs&, dim3, dim3, hipStream_t);
extern template void launch_materialize<1>(const KArgs&, dim3, dim3, hipStream_t);

}  // namespace ss
