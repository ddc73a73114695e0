// ss_stream.hip -- the streaming kernel for both logit element types.
#include "ss_impl.hpp"
#include "ss_launch.hpp"

namespace ss {

template <int DT, bool LP>
void launch_stream(const KArgs& k, dim3 grid, dim3 block, int smem, hipStream_t st) {
  hipLaunchKernelGGL((ss_stream_kernel<DT, LP>), grid, block, smem, st, k);
}
template void launch_stream<SS_F32, false>(const KArgs&, dim3, dim3, int, hipStream_t);
template void launch_stream<SS_BF16, false>(const KArgs&, dim3, dim3, int, hipStream_t);
template void launch_stream<SS_F32, true>(const KArgs&, dim3, dim3, int, hipStream_t);
template void launch_stream<SS_BF16, true>(const KArgs&, dim3, dim3, int, hipStream_t);

}  // namespace ss
