// The fused step's bfloat16 instances for 16-token pages, and the dispatcher.
#include "prr_fused_impl.h"

namespace prr {

template hipError_t launch_fused_inst<true, 16, 1>(int, const FusedLaunch&, hipStream_t);
template int resident_inst<true, 16, 1>();
template hipError_t launch_fused_inst<true, 16, 2>(int, const FusedLaunch&, hipStream_t);
template int resident_inst<true, 16, 2>();

int fused_grid(const FusedLaunch& a) {
  const int H = a.num_kv_heads;
  int per = a.n_score + 1;
  if (a.schedule != 0) per += 1;
  if (a.schedule == 1) per += a.n_spec + a.n_late;
  if (a.schedule != 2) per += a.miss_wgs + a.group;
  return H * per;
}

int fused_resident(bool bf16, int page_size, int chunk) {
  const int npw = (chunk + kFusedWaves - 1) / kFusedWaves;
  if (page_size == 16) {
    if (npw <= 1) return bf16 ? resident_inst<true, 16, 1>() : resident_inst<false, 16, 1>();
    return bf16 ? resident_inst<true, 16, 2>() : resident_inst<false, 16, 2>();
  }
  return bf16 ? resident_inst<true, 64, 1>() : resident_inst<false, 64, 1>();
}

hipError_t launch_fused(const FusedLaunch& a, bool bf16, int page_size, hipStream_t stream) {
  const int grid = fused_grid(a);
  const int npw = (a.chunk + kFusedWaves - 1) / kFusedWaves;
  if (page_size == 16) {
    if (npw <= 1)
      return bf16 ? launch_fused_inst<true, 16, 1>(grid, a, stream) : launch_fused_inst<false, 16, 1>(grid, a, stream);
    return bf16 ? launch_fused_inst<true, 16, 2>(grid, a, stream) : launch_fused_inst<false, 16, 2>(grid, a, stream);
  }
  return bf16 ? launch_fused_inst<true, 64, 1>(grid, a, stream) : launch_fused_inst<false, 64, 1>(grid, a, stream);
}

}  // namespace prr
