// prr_score_topk_static: the selection entry point without a workspace argument and
// without any allocation, for callers that cannot allocate device memory (code under
// HIP graph capture, tight serving loops).  Its only scratch -- one arrival counter per KV
// head, with which the last score workgroup of a head finds that every score is written
// -- lives in a file-scope device array of fixed size, one copy per GPU.
#include <mutex>

#include "prr_launch.h"

namespace {

constexpr int kScratchWords = PRR_STATIC_MAX_KV_HEADS;

// One arrival counter per KV head.  In host code this name stands for the array, not for
// its device address: the address is looked up per device (scratch_of) and only that is
// passed to kernels or fill launches.
__device__ __align__(256) uint32_t scratch[kScratchWords];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
uint32_t* g_scratch_ptr[kMaxDevices] = {};

// The device address of the current device's copy of `scratch`, looked up once per device
// with that device current.
prr_status scratch_of(uint32_t** out) {
  int dev = -1;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return prr::api_fail(PRR_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return prr::api_fail(PRR_ERR_HIP, "device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (r != hipSuccess || !p)
      return prr::api_fail(PRR_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(r));
    g_scratch_ptr[dev] = static_cast<uint32_t*>(p);
  }
  *out = g_scratch_ptr[dev];
  return PRR_OK;
}

}  // namespace

extern "C" prr_status prr_score_topk_static(const prr_dims* dims, const void* q, const void* meta, int32_t num_pages,
                                             int32_t k_select, const int32_t* forced, int32_t n_forced,
                                             int32_t forced_in_budget, float* scores, int32_t* selected,
                                             int32_t* selected_count, int32_t cap, hipStream_t stream) {
  prr::ScoreLaunch a;
  const prr_status st = prr::prepare_score(dims, q, meta, num_pages, k_select, forced, n_forced, forced_in_budget,
                                           scores, selected, selected_count, cap, a);
  if (st != PRR_OK) return st;
  if (dims->num_kv_heads > kScratchWords)
    return prr::api_fail(PRR_ERR_INVALID_ARG, "num_kv_heads %d exceeds the %d KV heads of the static scratch",
                         dims->num_kv_heads, kScratchWords);
  uint32_t* ptr = nullptr;
  const prr_status sp = scratch_of(&ptr);
  if (sp != PRR_OK) return sp;
  // the counters start at zero: cleared on this stream before every call (a fill kernel,
  // not a memset node, so that the call can be captured in a graph)
  hipError_t e = prr::launch_fill_zero(ptr, sizeof(uint32_t) * kScratchWords, stream);
  if (e == hipSuccess) {
    a.counters = ptr;
    e = prr::launch_score_topk(a, stream);
  }
  if (e != hipSuccess) return prr::api_fail(PRR_ERR_HIP, "score_topk_static launch: %s", hipGetErrorString(e));
  return prr::api_ok();
}
