// The fused step's instances for 64-token pages (block-mean selection workloads).
#include "prr_fused_impl.h"

namespace prr {

template hipError_t launch_fused_inst<true, 64, 1>(int, const FusedLaunch&, hipStream_t);
template int resident_inst<true, 64, 1>();
template hipError_t launch_fused_inst<false, 64, 1>(int, const FusedLaunch&, hipStream_t);
template int resident_inst<false, 64, 1>();

}  // namespace prr
