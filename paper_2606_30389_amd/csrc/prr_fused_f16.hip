// The fused step's float16 instances for 16-token pages.
#include "prr_fused_impl.h"

namespace prr {

template hipError_t launch_fused_inst<false, 16, 1>(int, const FusedLaunch&, hipStream_t);
template int resident_inst<false, 16, 1>();
template hipError_t launch_fused_inst<false, 16, 2>(int, const FusedLaunch&, hipStream_t);
template int resident_inst<false, 16, 2>();

}  // namespace prr
