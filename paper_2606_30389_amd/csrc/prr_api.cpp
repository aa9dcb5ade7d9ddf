// C ABI of libprr: argument validation, workspace carving, dispatch to the launchers.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <stddef.h>

#include <algorithm>
#include <mutex>

#include "prr.h"
#include "prr_launch.h"

// (alpha, beta, gamma) of the step parameters are read as one float[3]
static_assert(offsetof(prr_step_params, beta) == offsetof(prr_step_params, alpha) + sizeof(float) &&
                  offsetof(prr_step_params, gamma) == offsetof(prr_step_params, alpha) + 2 * sizeof(float),
              "alpha, beta, gamma are consecutive");

namespace {

thread_local char g_last_error[512] = "";

prr_status fail(prr_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

prr_status ok() {
  g_last_error[0] = '\0';
  return PRR_OK;
}

prr_status hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(PRR_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int div_up(int a, int b) { return (a + b - 1) / b; }

// a chunk (unit) holds at most 16 tiles of 16 tokens: four per wave
bool chunk_ok(const prr_dims* d, int chunk) { return chunk >= 1 && chunk * (d->page_size / 16) <= 16; }

prr_status check_dims(const prr_dims* d) {
  if (!d) return fail(PRR_ERR_INVALID_ARG, "dims is NULL");
  if (d->head_dim != 128) return fail(PRR_ERR_UNSUPPORTED, "head_dim %d: only 128 is compiled", d->head_dim);
  if (d->page_size != 16 && d->page_size != 32 && d->page_size != 64 && d->page_size != 128 && d->page_size != 256)
    return fail(PRR_ERR_UNSUPPORTED, "page_size %d: only 16, 32, 64, 128 and 256 are compiled", d->page_size);
  if (d->num_kv_heads < 1) return fail(PRR_ERR_INVALID_ARG, "num_kv_heads %d < 1", d->num_kv_heads);
  if (d->num_q_heads < 1 || d->num_q_heads % d->num_kv_heads != 0)
    return fail(PRR_ERR_INVALID_ARG, "num_q_heads %d is not a multiple of num_kv_heads %d", d->num_q_heads,
                d->num_kv_heads);
  const int g = d->num_q_heads / d->num_kv_heads;
  if (g > 16) return fail(PRR_ERR_UNSUPPORTED, "group size %d > 16", g);
  if (d->max_pages < 1) return fail(PRR_ERR_INVALID_ARG, "max_pages %d < 1", d->max_pages);
  if (d->dtype != PRR_F16 && d->dtype != PRR_BF16) return fail(PRR_ERR_INVALID_ARG, "dtype %d", d->dtype);
  if (d->meta_kind != PRR_META_MINMAX && d->meta_kind != PRR_META_MEAN)
    return fail(PRR_ERR_INVALID_ARG, "meta_kind %d", d->meta_kind);
  return ok();
}

prr_status check_ptr(const void* p, const char* name, size_t align) {
  if (!p) return fail(PRR_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned(p, align)) return fail(PRR_ERR_INVALID_ARG, "%s is not %zu-byte aligned", name, align);
  return ok();
}

#define PRR_TRY(expr)              \
  do {                             \
    const prr_status _s = (expr);  \
    if (_s != PRR_OK) return _s;   \
  } while (0)

struct WsLayout {
  size_t flags, sel_cnt, rep_cnt, rep_o, rep_ml, f_score, f_thr, f_mcnt, f_mlist, f_part, f_parto, f_candk,
      f_candp, f_pkey, f_win, f_lcnt, f_pbits, total;
  int nchunks, nwork_max, nparts;
};

bool ws_layout(const prr_dims* d, int cap, int chunk, WsLayout& L) {
  if (check_dims(d) != PRR_OK || cap < 1 || cap > PRR_MAX_CAP || !chunk_ok(d, chunk)) return false;
  const int hkv = d->num_kv_heads, g = d->num_q_heads / d->num_kv_heads;
  L.nchunks = div_up(cap, chunk);
  L.nwork_max = 2 * L.nchunks;
  size_t off = 0;
  L.flags = off;
  off += 256;
  L.sel_cnt = off;
  off = align_up(off + (size_t)hkv * 4, 256);
  L.rep_cnt = off;
  off = align_up(off + (size_t)2 * hkv * 4, 256);
  L.rep_o = off;
  off = align_up(off + (size_t)hkv * L.nwork_max * g * 128 * 4, 256);
  L.rep_ml = off;
  off = align_up(off + (size_t)hkv * L.nwork_max * g * 2 * 4, 256);
  // fused step: tagged scores, threshold, missed count and list, partial states
  L.nparts = 3 * L.nchunks;
  L.f_score = off;
  off = align_up(off + (size_t)hkv * d->max_pages * 8, 256);
  // the threshold, missed and late counts: 8 copies of 256 bytes per KV head
  L.f_thr = off;
  off = align_up(off + (size_t)hkv * 8 * 256, 256);
  L.f_mcnt = off;
  off = align_up(off + (size_t)hkv * 8 * 256, 256);
  L.f_mlist = off;
  off = align_up(off + (size_t)hkv * cap * 8, 256);
  L.f_part = off;
  off = align_up(off + (size_t)hkv * L.nparts * g * 2 * 8, 256);
  L.f_parto = off;
  off = align_up(off + (size_t)hkv * L.nparts * g * 128 * 4, 256);
  const size_t nsc = (size_t)div_up(d->max_pages, prr::kFusedScorePages);
  L.f_candk = off;  // per list: the count, then the keys
  off = align_up(off + 3 * (size_t)hkv * nsc * (prr::kFusedScorePages + 4) * 8, 256);
  L.f_candp = off;
  off = align_up(off + 3 * (size_t)hkv * nsc * prr::kFusedScorePages * 8, 256);
  L.f_pkey = off;
  off = align_up(off + (size_t)hkv * d->max_pages * 8, 256);
  L.f_win = off;
  off = align_up(off + (size_t)hkv * 4 * 4, 256);
  L.f_lcnt = off;
  off = align_up(off + (size_t)hkv * 8 * 256, 256);
  L.f_pbits = off;
  off = align_up(off + 2 * (size_t)hkv * ((d->max_pages + 31) / 32) * 4, 256);
  L.total = off;
  return true;
}

prr_status check_forced(const int32_t* forced, int n_forced, int num_pages) {
  if (n_forced < 0 || n_forced > PRR_MAX_FORCED)
    return fail(PRR_ERR_INVALID_ARG, "n_forced %d outside [0, %d]", n_forced, PRR_MAX_FORCED);
  if (n_forced > 0 && !forced) return fail(PRR_ERR_INVALID_ARG, "forced is NULL with n_forced %d", n_forced);
  for (int i = 0; i < n_forced; ++i) {
    if (forced[i] < 0 || forced[i] >= num_pages)
      return fail(PRR_ERR_INVALID_ARG, "forced[%d] = %d outside [0, %d)", i, forced[i], num_pages);
    for (int j = 0; j < i; ++j)
      if (forced[j] == forced[i]) return fail(PRR_ERR_INVALID_ARG, "forced page %d listed twice", forced[i]);
  }
  return ok();
}

// (alpha, beta, gamma) of the EMA predictor in (0, 1], (0, 1], [0, 1].
prr_status check_theta(const float* th) {
  if (!(th[0] > 0.f && th[0] <= 1.f) || !(th[1] > 0.f && th[1] <= 1.f) || !(th[2] >= 0.f && th[2] <= 1.f))
    return fail(PRR_ERR_INVALID_ARG, "alpha %g, beta %g, gamma %g outside (0,1], (0,1], [0,1]", th[0], th[1], th[2]);
  return ok();
}

// Late-speculation workgroups per KV head: one per chunk of the list capacity, or fewer
// when that keeps every role dispatched up to the late workgroups (score, select,
// predict, speculation, late) within the workgroups the chip holds at once, so that no
// late workgroup waits for a slot.  Late pages beyond the capacity are attended after the
// threshold, as missed pages; a cut deeper than half is not made.
int late_slots(const prr_dims* d, int n_score, int nchunks, int chunk) {
  const int resident = prr::fused_resident(d->dtype == PRR_BF16, d->page_size, chunk);
  if (resident <= 0) return nchunks;
  const int fit = resident / d->num_kv_heads - n_score - 2 - nchunks;
  if (fit >= nchunks || fit < (nchunks + 1) / 2) return nchunks;
  return fit;
}

// Missed-list workgroups per KV head.  With late speculation the missed list is short (the
// pages of A that neither P nor the late window attended before the threshold), so a few
// workgroups take its chunks in turn instead of one idle workgroup per chunk of the list
// capacity; without it every chunk has a workgroup of its own.
// (Instances of two pages per wave, chunks above kFusedWaves pages, take one chunk per
// workgroup.)
constexpr int kLateMissWorkgroups = 4;
int miss_workgroups(bool late, int nchunks, int chunk) {
  return late && chunk <= prr::kFusedWaves ? std::min(nchunks, kLateMissWorkgroups) : nchunks;
}

// |A| for a budget and forced set, and the number of non-forced pages to pick.
void budget(int k_select, int n_forced, int forced_in_budget, int num_pages, int& total, int& kextra) {
  kextra = forced_in_budget ? std::max(0, k_select - n_forced) : k_select;
  total = std::min(num_pages, n_forced + kextra);
}

// Events and stream-memory words of prr_stream_chain (words 0, 1) and of the two-stream
// step without events (words 2-5: fork, selection, speculation, join), made once per device
// and kept until the process ends (a stream may still wait on them when a call returns).
// Every value written is larger than the one before, so each word only grows.
constexpr int kChainMaxHops = 256;
constexpr int kChainMaxDevices = 16;
constexpr int kStreamWords = 6;
struct ChainState {
  bool events = false, words = false;
  hipEvent_t ev[kChainMaxHops] = {};
  void* word[kStreamWords] = {};
  uint64_t value = 0;  // the last value written
};
std::mutex g_chain_mu;
ChainState g_chain[kChainMaxDevices];

}  // namespace

namespace prr {

prr_status api_fail(prr_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return st;
}

prr_status api_ok() { return ok(); }

prr_status prepare_score(const prr_dims* dims, const void* q, const void* meta, int32_t num_pages, int32_t k_select,
                         const int32_t* forced, int32_t n_forced, int32_t forced_in_budget, float* scores,
                         int32_t* selected, int32_t* selected_count, int32_t cap, ScoreLaunch& a) {
  PRR_TRY(check_dims(dims));
  PRR_TRY(check_ptr(q, "q", 16));
  PRR_TRY(check_ptr(meta, "meta", 16));
  PRR_TRY(check_ptr(scores, "scores", 4));
  PRR_TRY(check_ptr(selected, "selected", 4));
  PRR_TRY(check_ptr(selected_count, "selected_count", 4));
  if (num_pages < 1 || num_pages > PRR_MAX_PAGES || num_pages > dims->max_pages)
    return fail(PRR_ERR_INVALID_ARG, "num_pages %d outside [1, min(max_pages, %d)]", num_pages, PRR_MAX_PAGES);
  if (k_select < 0) return fail(PRR_ERR_INVALID_ARG, "k_select %d < 0", k_select);
  PRR_TRY(check_forced(forced, n_forced, num_pages));
  if (cap < 1 || cap > PRR_MAX_CAP) return fail(PRR_ERR_INVALID_ARG, "cap %d outside [1, %d]", cap, PRR_MAX_CAP);
  int total, kextra;
  budget(k_select, n_forced, forced_in_budget, num_pages, total, kextra);
  if (total > cap) return fail(PRR_ERR_INVALID_ARG, "|A| = %d exceeds cap %d", total, cap);
  memset(&a, 0, sizeof(a));
  a.q = q;
  a.meta = meta;
  a.scores = scores;
  a.selected = selected;
  a.selected_count = selected_count;
  a.num_kv_heads = dims->num_kv_heads;
  a.group = dims->num_q_heads / dims->num_kv_heads;
  a.max_pages = dims->max_pages;
  a.num_pages = num_pages;
  a.kextra = kextra;
  a.cap = cap;
  a.n_forced = n_forced;
  a.bf16 = dims->dtype == PRR_BF16;
  a.meta_mean = dims->meta_kind == PRR_META_MEAN;
  for (int i = 0; i < n_forced; ++i) a.forced[i] = forced[i];
  return ok();
}

}  // namespace prr

extern "C" {

const char* prr_status_string(prr_status s) {
  switch (s) {
    case PRR_OK: return "PRR_OK";
    case PRR_ERR_INVALID_ARG: return "PRR_ERR_INVALID_ARG";
    case PRR_ERR_UNSUPPORTED: return "PRR_ERR_UNSUPPORTED";
    case PRR_ERR_WORKSPACE: return "PRR_ERR_WORKSPACE";
    case PRR_ERR_HIP: return "PRR_ERR_HIP";
    default: return "PRR_ERR_UNKNOWN";
  }
}

const char* prr_last_error(void) { return g_last_error; }

size_t prr_workspace_size(const prr_dims* dims, int32_t cap, int32_t chunk_pages) {
  WsLayout L;
  if (!ws_layout(dims, cap, chunk_pages, L)) return 0;
  return L.total;
}

prr_status prr_workspace_init(void* workspace, size_t bytes, hipStream_t stream) {
  PRR_TRY(check_ptr(workspace, "workspace", 256));
  if (bytes % 16 != 0) return fail(PRR_ERR_WORKSPACE, "workspace size %zu is not a multiple of 16", bytes);
  return hip_status(prr::launch_fill_zero(workspace, bytes, stream), "workspace fill");
}

prr_status prr_empty_launch(int32_t grid, int32_t threads, hipStream_t stream) {
  if (grid < 1 || grid > (1 << 20)) return fail(PRR_ERR_INVALID_ARG, "grid %d outside [1, 2^20]", grid);
  if (threads < 1 || threads > 1024) return fail(PRR_ERR_INVALID_ARG, "threads %d outside [1, 1024]", threads);
  return hip_status(prr::launch_empty(grid, threads, stream), "empty launch");
}

prr_status prr_read_stream(const void* buf, size_t bytes, uint32_t* sink, int32_t grid, hipStream_t stream) {
  PRR_TRY(check_ptr(buf, "buf", 16));
  PRR_TRY(check_ptr(sink, "sink", 4));
  if (bytes == 0 || bytes % 16 != 0) return fail(PRR_ERR_INVALID_ARG, "bytes %zu is not a positive multiple of 16", bytes);
  if (grid < 1 || grid > (1 << 20)) return fail(PRR_ERR_INVALID_ARG, "grid %d outside [1, 2^20]", grid);
  return hip_status(prr::launch_read_stream(buf, bytes, sink, grid, stream), "read stream");
}

}  // extern "C"

namespace {

// This device's events and stream-memory words (the caller locks g_chain_mu to use them).
prr_status chain_state(ChainState*& st) {
  int dev = 0;
  PRR_TRY(hip_status(hipGetDevice(&dev), "get device"));
  if (dev < 0 || dev >= kChainMaxDevices) return fail(PRR_ERR_UNSUPPORTED, "device %d", dev);
  st = &g_chain[dev];
  return ok();
}

// The stream-memory words, allocated and zeroed on first use (a set-up that failed
// part-way resumes where it stopped); called with g_chain_mu held.
prr_status stream_words(ChainState& st, hipStream_t s) {
  if (st.words) return ok();
  int dev = 0, can = 0;
  PRR_TRY(hip_status(hipGetDevice(&dev), "get device"));
  PRR_TRY(hip_status(hipDeviceGetAttribute(&can, hipDeviceAttributeCanUseStreamWaitValue, dev), "attribute"));
  if (!can) return fail(PRR_ERR_UNSUPPORTED, "the device has no stream memory waits");
  for (int k = 0; k < kStreamWords; ++k)
    if (!st.word[k])
      PRR_TRY(hip_status(hipExtMallocWithFlags(&st.word[k], sizeof(uint64_t), hipMallocSignalMemory),
                         "stream memory word"));
  // zero every word and wait, so that no first wait compares against what the new memory held
  for (int k = 0; k < kStreamWords; ++k)
    PRR_TRY(hip_status(hipStreamWriteValue64(s, st.word[k], 0ull, 0), "stream write"));
  PRR_TRY(hip_status(hipStreamSynchronize(s), "stream synchronize"));
  st.words = true;
  return ok();
}

// `to` waits until `from` has reached this point: an event, or a stream-memory word.
prr_status stream_dep(hipStream_t from, hipStream_t to, hipEvent_t ev, ChainState* mem, int word) {
  if (!mem) {
    PRR_TRY(hip_status(hipEventRecord(ev, from), "event record"));
    return hip_status(hipStreamWaitEvent(to, ev, 0), "stream wait");
  }
  const uint64_t v = ++mem->value;
  PRR_TRY(hip_status(hipStreamWriteValue64(from, mem->word[word], v, 0), "stream write"));
  return hip_status(hipStreamWaitValue64(to, mem->word[word], v, hipStreamWaitValueGte, ~0ull), "stream wait");
}

}  // namespace

extern "C" {

prr_status prr_stream_chain(int32_t n_hops, int32_t mode, hipStream_t a, hipStream_t b) {
  if (n_hops < 2 || n_hops > kChainMaxHops || n_hops % 2 != 0)
    return fail(PRR_ERR_INVALID_ARG, "n_hops %d is not even in [2, %d]", n_hops, kChainMaxHops);
  if (mode < PRR_CHAIN_ONE_STREAM || mode > PRR_CHAIN_STREAM_MEMORY) return fail(PRR_ERR_INVALID_ARG, "mode %d", mode);
  if (mode == PRR_CHAIN_ONE_STREAM) {
    for (int i = 0; i < n_hops; ++i) PRR_TRY(hip_status(prr::launch_empty(1, 64, a), "empty launch"));
    return ok();
  }
  if (a == b) return fail(PRR_ERR_INVALID_ARG, "a dependency needs two different streams");
  ChainState* stp = nullptr;
  PRR_TRY(chain_state(stp));
  std::lock_guard<std::mutex> guard(g_chain_mu);
  ChainState& st = *stp;
  if (!st.events) {  // (a set-up that failed part-way resumes where it stopped)
    for (int i = 0; i < kChainMaxHops; ++i)
      if (!st.ev[i]) PRR_TRY(hip_status(hipEventCreateWithFlags(&st.ev[i], hipEventDisableTiming), "event create"));
    st.events = true;
  }
  if (mode == PRR_CHAIN_STREAM_MEMORY) PRR_TRY(stream_words(st, a));
  for (int i = 0; i < n_hops; ++i) {
    hipStream_t x = (i & 1) ? b : a, y = (i & 1) ? a : b;
    PRR_TRY(hip_status(prr::launch_empty(1, 64, x), "empty launch"));
    if (mode == PRR_CHAIN_EVENTS) {
      PRR_TRY(hip_status(hipEventRecord(st.ev[i], x), "event record"));
      PRR_TRY(hip_status(hipStreamWaitEvent(y, st.ev[i], 0), "stream wait"));
    } else {
      const uint64_t v = ++st.value;
      PRR_TRY(hip_status(hipStreamWriteValue64(x, st.word[i & 1], v, 0), "stream write"));
      PRR_TRY(hip_status(hipStreamWaitValue64(y, st.word[i & 1], v, hipStreamWaitValueGte, ~0ull), "stream wait"));
    }
  }
  return ok();
}

int32_t prr_fused_grid(const prr_dims* dims, const prr_step_params* sp, int32_t schedule) {
  if (check_dims(dims) != PRR_OK || !sp || schedule < PRR_SCHED_FUSED_SERIAL || schedule > PRR_SCHED_FUSED_PREFILL ||
      (dims->page_size != 16 && dims->page_size != 64))
    return 0;
  WsLayout L;
  if (!ws_layout(dims, sp->cap, sp->chunk_pages, L) || sp->num_pages < 1) return 0;
  prr::FusedLaunch a;
  memset(&a, 0, sizeof(a));
  a.schedule = schedule == PRR_SCHED_FUSED_PRR ? 1 : (schedule == PRR_SCHED_FUSED_PREFILL ? 2 : 0);
  a.num_kv_heads = dims->num_kv_heads;
  a.group = dims->num_q_heads / dims->num_kv_heads;
  a.n_score = div_up(sp->num_pages, prr::kFusedScorePages);
  a.n_spec = L.nchunks;
  a.n_miss = L.nchunks;
  a.late = a.schedule == 1 && sp->late_spec && sp->mode != PRR_RECOMPUTE_ON_MISS;
  a.n_late = a.late ? late_slots(dims, a.n_score, L.nchunks, sp->chunk_pages) : 0;
  a.miss_wgs = miss_workgroups(a.late, L.nchunks, sp->chunk_pages);
  return prr::fused_grid(a);
}

prr_status prr_epoch_advance(uint32_t* epoch_dev, hipStream_t stream) {
  PRR_TRY(check_ptr(epoch_dev, "epoch_dev", 4));
  return hip_status(prr::launch_epoch_advance(epoch_dev, stream), "epoch advance");
}

size_t prr_spec_state_floats(const prr_dims* dims, int32_t cap, int32_t chunk_pages, size_t* part_o_floats,
                             size_t* part_ml_floats, size_t* page_m_floats) {
  if (check_dims(dims) != PRR_OK || cap < 1 || cap > PRR_MAX_CAP || !chunk_ok(dims, chunk_pages)) return 0;
  const size_t hkv = dims->num_kv_heads, g = dims->num_q_heads / dims->num_kv_heads;
  const size_t nch = (size_t)div_up(cap, chunk_pages);
  const size_t po = hkv * nch * g * 128, pml = hkv * nch * g, pm = hkv * (size_t)cap * g;
  if (part_o_floats) *part_o_floats = po;
  if (part_ml_floats) *part_ml_floats = pml;
  if (page_m_floats) *page_m_floats = pm;
  return po + 2 * pml + pm;
}

prr_status prr_build_page_meta(const prr_dims* dims, const void* k_cache, const int32_t* page_table,
                               int32_t num_tokens, int32_t page_begin, int32_t page_end, void* meta,
                               hipStream_t stream) {
  PRR_TRY(check_dims(dims));
  PRR_TRY(check_ptr(k_cache, "k_cache", 16));
  PRR_TRY(check_ptr(meta, "meta", 16));
  if (page_table && !aligned(page_table, 4)) return fail(PRR_ERR_INVALID_ARG, "page_table misaligned");
  if (num_tokens < 1 || (int64_t)num_tokens > (int64_t)dims->max_pages * dims->page_size)
    return fail(PRR_ERR_INVALID_ARG, "num_tokens %d outside [1, max_pages*page_size]", num_tokens);
  const int npages = div_up(num_tokens, dims->page_size);
  if (page_begin < 0 || page_end > npages || page_begin > page_end)
    return fail(PRR_ERR_INVALID_ARG, "page range [%d, %d) outside [0, %d]", page_begin, page_end, npages);
  prr::MetaLaunch a;
  a.k_cache = k_cache;
  a.page_table = page_table;
  a.meta = meta;
  a.num_kv_heads = dims->num_kv_heads;
  a.max_pages = dims->max_pages;
  a.page_size = dims->page_size;
  a.num_tokens = num_tokens;
  a.page_begin = page_begin;
  a.page_end = page_end;
  a.bf16 = dims->dtype == PRR_BF16;
  a.meta_mean = dims->meta_kind == PRR_META_MEAN;
  return hip_status(prr::launch_meta(a, stream), "build_page_meta launch");
}

prr_status prr_score_topk(const prr_dims* dims, const void* q, const void* meta, int32_t num_pages, int32_t k_select,
                          const int32_t* forced, int32_t n_forced, int32_t forced_in_budget, float* scores,
                          int32_t* selected, int32_t* selected_count, int32_t cap, void* workspace, size_t ws_bytes,
                          hipStream_t stream) {
  prr::ScoreLaunch a;
  PRR_TRY(prr::prepare_score(dims, q, meta, num_pages, k_select, forced, n_forced, forced_in_budget, scores, selected,
                             selected_count, cap, a));
  PRR_TRY(check_ptr(workspace, "workspace", 256));
  WsLayout L;
  if (!ws_layout(dims, cap, 1, L) || ws_bytes < L.rep_cnt)
    return fail(PRR_ERR_WORKSPACE, "workspace of %zu bytes too small", ws_bytes);
  a.counters = reinterpret_cast<uint32_t*>(static_cast<char*>(workspace) + L.sel_cnt);
  return hip_status(prr::launch_score_topk(a, stream), "score_topk launch");
}

prr_status prr_predict(const prr_dims* dims, float* ema_level, float* ema_trend, uint32_t* ema_init_bits,
                       const float* scores, int32_t num_pages, float alpha, float beta, float gamma, int32_t p_select,
                       const int32_t* forced, int32_t n_forced, int32_t forced_in_budget, int32_t* predicted,
                       int32_t* predicted_count, int32_t cap, hipStream_t stream) {
  PRR_TRY(check_dims(dims));
  PRR_TRY(check_ptr(ema_level, "ema_level", 4));
  PRR_TRY(check_ptr(ema_trend, "ema_trend", 4));
  PRR_TRY(check_ptr(ema_init_bits, "ema_init_bits", 4));
  if (scores && !aligned(scores, 4)) return fail(PRR_ERR_INVALID_ARG, "scores misaligned");
  PRR_TRY(check_ptr(predicted, "predicted", 4));
  PRR_TRY(check_ptr(predicted_count, "predicted_count", 4));
  if (num_pages < 1 || num_pages > PRR_MAX_PAGES || num_pages > dims->max_pages)
    return fail(PRR_ERR_INVALID_ARG, "num_pages %d outside [1, min(max_pages, %d)]", num_pages, PRR_MAX_PAGES);
  if (!(alpha > 0.f && alpha <= 1.f) || !(beta > 0.f && beta <= 1.f) || !(gamma >= 0.f && gamma <= 1.f))
    return fail(PRR_ERR_INVALID_ARG, "alpha %g, beta %g, gamma %g outside (0,1], (0,1], [0,1]", alpha, beta, gamma);
  if (p_select < 0) return fail(PRR_ERR_INVALID_ARG, "p_select %d < 0", p_select);
  PRR_TRY(check_forced(forced, n_forced, num_pages));
  if (cap < 1 || cap > PRR_MAX_CAP) return fail(PRR_ERR_INVALID_ARG, "cap %d outside [1, %d]", cap, PRR_MAX_CAP);
  int total, kextra;
  budget(p_select, n_forced, forced_in_budget, num_pages, total, kextra);
  if (total > cap) return fail(PRR_ERR_INVALID_ARG, "|P| = %d exceeds cap %d", total, cap);
  prr::PredictLaunch a;
  memset(&a, 0, sizeof(a));
  a.level = ema_level;
  a.trend = ema_trend;
  a.init_bits = ema_init_bits;
  a.scores = scores;
  a.predicted = predicted;
  a.predicted_count = predicted_count;
  a.alpha = alpha;
  a.beta = beta;
  a.gamma = gamma;
  a.num_kv_heads = dims->num_kv_heads;
  a.max_pages = dims->max_pages;
  a.num_pages = num_pages;
  a.kextra = kextra;
  a.cap = cap;
  a.n_forced = n_forced;
  for (int i = 0; i < n_forced; ++i) a.forced[i] = forced[i];
  return hip_status(prr::launch_predict(a, stream), "predict launch");
}

prr_status prr_spec_attn(const prr_dims* dims, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* page_table, int32_t num_tokens, const int32_t* pages,
                         const int32_t* page_count, int32_t cap, int32_t chunk_pages, float* part_o, float* part_m,
                         float* part_l, float* page_m, hipStream_t stream) {
  PRR_TRY(check_dims(dims));
  PRR_TRY(check_ptr(q, "q", 16));
  PRR_TRY(check_ptr(k_cache, "k_cache", 16));
  PRR_TRY(check_ptr(v_cache, "v_cache", 16));
  PRR_TRY(check_ptr(pages, "pages", 4));
  PRR_TRY(check_ptr(page_count, "page_count", 4));
  PRR_TRY(check_ptr(part_o, "part_o", 16));
  PRR_TRY(check_ptr(part_m, "part_m", 4));
  PRR_TRY(check_ptr(part_l, "part_l", 4));
  if (page_m && !aligned(page_m, 4)) return fail(PRR_ERR_INVALID_ARG, "page_m misaligned");
  if (page_table && !aligned(page_table, 4)) return fail(PRR_ERR_INVALID_ARG, "page_table misaligned");
  if (num_tokens < 1 || (int64_t)num_tokens > (int64_t)dims->max_pages * dims->page_size)
    return fail(PRR_ERR_INVALID_ARG, "num_tokens %d outside [1, max_pages*page_size]", num_tokens);
  if (cap < 1 || cap > PRR_MAX_CAP) return fail(PRR_ERR_INVALID_ARG, "cap %d outside [1, %d]", cap, PRR_MAX_CAP);
  if (!chunk_ok(dims, chunk_pages))
    return fail(PRR_ERR_INVALID_ARG, "chunk_pages %d outside [1, 256 / page_size]", chunk_pages);
  prr::SpecLaunch a;
  memset(&a, 0, sizeof(a));
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.page_table = page_table;
  a.pages = pages;
  a.page_count = page_count;
  a.part_o = part_o;
  a.part_m = part_m;
  a.part_l = part_l;
  a.page_m = page_m;
  a.num_kv_heads = dims->num_kv_heads;
  a.group = dims->num_q_heads / dims->num_kv_heads;
  a.max_pages = dims->max_pages;
  a.num_pages = div_up(num_tokens, dims->page_size);
  a.num_tokens = num_tokens;
  a.page_size = dims->page_size;
  a.cap = cap;
  a.chunk = chunk_pages;
  a.nchunks = div_up(cap, chunk_pages);
  a.bf16 = dims->dtype == PRR_BF16;
  return hip_status(prr::launch_spec_attn(a, stream), "spec_attn launch");
}

prr_status prr_repair(const prr_dims* dims, const void* q, const void* k_cache, const void* v_cache,
                      const int32_t* page_table, int32_t num_tokens, int32_t num_pages, const int32_t* selected,
                      const int32_t* selected_count, const int32_t* predicted, const int32_t* predicted_count,
                      int32_t cap, int32_t chunk_pages, const float* part_o, const float* part_m, const float* part_l,
                      const float* page_m, int32_t mode, float* out_o32, void* out_o, float* out_m, float* out_l,
                      int32_t* missed_count, int32_t* wasted_count, void* workspace, size_t ws_bytes,
                      hipStream_t stream) {
  PRR_TRY(check_dims(dims));
  PRR_TRY(check_ptr(q, "q", 16));
  PRR_TRY(check_ptr(k_cache, "k_cache", 16));
  PRR_TRY(check_ptr(v_cache, "v_cache", 16));
  PRR_TRY(check_ptr(selected, "selected", 4));
  PRR_TRY(check_ptr(selected_count, "selected_count", 4));
  if ((predicted == nullptr) != (predicted_count == nullptr))
    return fail(PRR_ERR_INVALID_ARG, "predicted and predicted_count must both be set or both be NULL");
  if (predicted) {
    PRR_TRY(check_ptr(predicted, "predicted", 4));
    PRR_TRY(check_ptr(predicted_count, "predicted_count", 4));
    PRR_TRY(check_ptr(part_o, "part_o", 16));
    PRR_TRY(check_ptr(part_m, "part_m", 4));
    PRR_TRY(check_ptr(part_l, "part_l", 4));
    if (page_m && !aligned(page_m, 4)) return fail(PRR_ERR_INVALID_ARG, "page_m misaligned");
  }
  PRR_TRY(check_ptr(out_o32, "out_o32", 4));
  if (out_o && !aligned(out_o, 2)) return fail(PRR_ERR_INVALID_ARG, "out_o misaligned");
  PRR_TRY(check_ptr(out_m, "out_m", 4));
  PRR_TRY(check_ptr(out_l, "out_l", 4));
  if (page_table && !aligned(page_table, 4)) return fail(PRR_ERR_INVALID_ARG, "page_table misaligned");
  if (mode != PRR_EXACT_SELECTED && mode != PRR_KEEP_WASTED) return fail(PRR_ERR_INVALID_ARG, "mode %d", mode);
  if (num_tokens < 1 || (int64_t)num_tokens > (int64_t)dims->max_pages * dims->page_size)
    return fail(PRR_ERR_INVALID_ARG, "num_tokens %d outside [1, max_pages*page_size]", num_tokens);
  const int npages_tok = div_up(num_tokens, dims->page_size);
  if (num_pages < 1 || num_pages > npages_tok || num_pages > PRR_MAX_PAGES)
    return fail(PRR_ERR_INVALID_ARG, "num_pages %d outside [1, min(ceil(num_tokens/page_size), %d)]", num_pages,
                PRR_MAX_PAGES);
  if (cap < 1 || cap > PRR_MAX_CAP) return fail(PRR_ERR_INVALID_ARG, "cap %d outside [1, %d]", cap, PRR_MAX_CAP);
  if (!chunk_ok(dims, chunk_pages))
    return fail(PRR_ERR_INVALID_ARG, "chunk_pages %d outside [1, 256 / page_size]", chunk_pages);
  PRR_TRY(check_ptr(workspace, "workspace", 256));
  WsLayout L;
  if (!ws_layout(dims, cap, chunk_pages, L) || ws_bytes < L.total)
    return fail(PRR_ERR_WORKSPACE, "workspace of %zu bytes too small (need %zu)", ws_bytes,
                ws_layout(dims, cap, chunk_pages, L) ? L.total : (size_t)0);
  const int g = dims->num_q_heads / dims->num_kv_heads;
  prr::RepairLaunch a;
  memset(&a, 0, sizeof(a));
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.page_table = page_table;
  a.selected = selected;
  a.selected_count = selected_count;
  a.predicted = predicted;
  a.predicted_count = predicted_count;
  a.part_o = part_o;
  a.part_m = part_m;
  a.part_l = part_l;
  a.page_m = predicted ? page_m : nullptr;
  a.out_o32 = out_o32;
  a.out_o = out_o;
  a.out_m = out_m;
  a.out_l = out_l;
  a.missed_count = missed_count;
  a.wasted_count = wasted_count;
  char* ws = static_cast<char*>(workspace);
  a.ws_o = reinterpret_cast<float*>(ws + L.rep_o);
  a.ws_ml = reinterpret_cast<float*>(ws + L.rep_ml);
  a.ws_cnt = reinterpret_cast<uint32_t*>(ws + L.rep_cnt);
  a.flags = reinterpret_cast<uint32_t*>(ws + L.flags);
  a.num_kv_heads = dims->num_kv_heads;
  a.group = g;
  a.max_pages = dims->max_pages;
  a.num_pages = num_pages;
  a.num_tokens = num_tokens;
  a.page_size = dims->page_size;
  a.cap = cap;
  a.chunk = chunk_pages;
  a.nchunks = L.nchunks;
  a.nwork = (predicted && mode == PRR_EXACT_SELECTED) ? 2 * L.nchunks : L.nchunks;
  a.nmerge_per_kv = div_up(g, 2);
  a.mode = mode;
  a.bf16 = dims->dtype == PRR_BF16;
  return hip_status(prr::launch_repair(a, stream), "repair launch");
}

prr_status prr_calibrate(const float* scores, int32_t n_traj, int32_t n_rows, int32_t n_blocks,
                         const int32_t* form_row, int32_t k_select, int32_t p_select, const float* grid, int32_t n_grid,
                         int32_t n_threads, float* best_theta, double* objective_out) {
  if (!scores || !grid || !best_theta) return fail(PRR_ERR_INVALID_ARG, "scores, grid or best_theta is NULL");
  if (n_traj < 1 || n_rows < 2 || n_blocks < 1 || n_grid < 1)
    return fail(PRR_ERR_INVALID_ARG, "n_traj %d, n_rows %d (>= 2), n_blocks %d, n_grid %d", n_traj, n_rows, n_blocks,
                n_grid);
  if (k_select < 0 || p_select < 0) return fail(PRR_ERR_INVALID_ARG, "k_select %d / p_select %d < 0", k_select, p_select);
  if (form_row) {
    for (int b = 0; b < n_blocks; ++b)
      if (form_row[b] < 0) return fail(PRR_ERR_INVALID_ARG, "form_row[%d] = %d < 0", b, form_row[b]);
  }
  for (int g = 0; g < n_grid; ++g) {
    const float a = grid[3 * g], b = grid[3 * g + 1], c = grid[3 * g + 2];
    if (!(a > 0.f && a <= 1.f) || !(b > 0.f && b <= 1.f) || !(c >= 0.f && c <= 1.f))
      return fail(PRR_ERR_INVALID_ARG, "grid point %d (%g, %g, %g) outside (0,1] x (0,1] x [0,1]", g, a, b, c);
  }
  prr::calibrate_grid(scores, n_traj, n_rows, n_blocks, form_row, k_select, p_select, grid, n_grid, n_threads,
                      best_theta, objective_out);
  return ok();
}

prr_status prr_pick_delta(const int32_t* context, const float* delta, const float* select_us, const float* spec_us,
                          int32_t n_rows, int32_t query_context, int32_t degree, float* delta_out, float* select_est,
                          float* spec_est) {
  if (!delta_out) return fail(PRR_ERR_INVALID_ARG, "delta_out is NULL");
  if (n_rows < 0) return fail(PRR_ERR_INVALID_ARG, "n_rows %d < 0", n_rows);
  if (n_rows > 0 && (!context || !delta || !select_us || !spec_us))
    return fail(PRR_ERR_INVALID_ARG, "a table column is NULL");
  if (query_context < 1) return fail(PRR_ERR_INVALID_ARG, "query_context %d < 1", query_context);
  if (degree < 0 || degree > 3) return fail(PRR_ERR_INVALID_ARG, "degree %d outside [0, 3]", degree);
  for (int i = 0; i < n_rows; ++i) {
    if (context[i] < 1 || !(delta[i] >= 1.0f) || !(select_us[i] >= 0.0f) || !(spec_us[i] >= 0.0f))
      return fail(PRR_ERR_INVALID_ARG, "table row %d: context %d, delta %g, select %g us, spec %g us", i, context[i],
                  delta[i], select_us[i], spec_us[i]);
  }
  if (select_est) *select_est = NAN;
  if (spec_est) *spec_est = NAN;
  *delta_out = n_rows > 0 ? prr::pick_delta(context, delta, select_us, spec_us, n_rows, query_context, degree,
                                            select_est, spec_est)
                          : 1.0f;
  return ok();
}

prr_status prr_merge_states(int32_t n_states, int32_t rows, int32_t d, const float* o, const float* m, const float* l,
                            float* out_o, float* out_m, float* out_l, hipStream_t stream) {
  if (n_states < 0 || rows < 1 || d < 1 || d > 1024)
    return fail(PRR_ERR_INVALID_ARG, "n_states %d, rows %d, d %d", n_states, rows, d);
  if (n_states > 0) {
    PRR_TRY(check_ptr(o, "o", 4));
    PRR_TRY(check_ptr(m, "m", 4));
    PRR_TRY(check_ptr(l, "l", 4));
  }
  PRR_TRY(check_ptr(out_o, "out_o", 4));
  PRR_TRY(check_ptr(out_m, "out_m", 4));
  PRR_TRY(check_ptr(out_l, "out_l", 4));
  return hip_status(prr::launch_merge_states(n_states, rows, d, o, m, l, out_o, out_m, out_l, stream),
                    "merge_states launch");
}

// One layer of a fused schedule: every argument checked as by the individual entry
// points, then one launch.
static prr_status fused_layer(const prr_dims* dims, const prr_step_params* sp, const prr_layer_io& y, int parity,
                              int schedule, hipStream_t stream, int layer) {
  const bool prr = schedule == PRR_SCHED_FUSED_PRR, prefill = schedule == PRR_SCHED_FUSED_PREFILL;
  PRR_TRY(check_ptr(y.q, "q", 16));
  PRR_TRY(check_ptr(y.meta, "meta", 16));
  PRR_TRY(check_ptr(y.scores, "scores", 4));
  PRR_TRY(check_ptr(y.selected, "selected", 4));
  PRR_TRY(check_ptr(y.selected_count, "selected_count", 4));
  if (y.page_table && !aligned(y.page_table, 4)) return fail(PRR_ERR_INVALID_ARG, "page_table misaligned");
  if (!prefill) {
    PRR_TRY(check_ptr(y.k_cache, "k_cache", 16));
    PRR_TRY(check_ptr(y.v_cache, "v_cache", 16));
    PRR_TRY(check_ptr(y.out_o32, "out_o32", 4));
    if (y.out_o && !aligned(y.out_o, 2)) return fail(PRR_ERR_INVALID_ARG, "out_o misaligned");
    PRR_TRY(check_ptr(y.out_m, "out_m", 4));
    PRR_TRY(check_ptr(y.out_l, "out_l", 4));
    if (y.missed_count && !aligned(y.missed_count, 4)) return fail(PRR_ERR_INVALID_ARG, "missed_count misaligned");
    if (y.wasted_count && !aligned(y.wasted_count, 4)) return fail(PRR_ERR_INVALID_ARG, "wasted_count misaligned");
    if (y.covered_count && !aligned(y.covered_count, 4)) return fail(PRR_ERR_INVALID_ARG, "covered_count misaligned");
  }
  if (prr || prefill) {
    PRR_TRY(check_ptr(y.ema_level, "ema_level", 4));
    PRR_TRY(check_ptr(y.ema_trend, "ema_trend", 4));
    PRR_TRY(check_ptr(y.ema_init_bits, "ema_init_bits", 4));
    PRR_TRY(check_ptr(y.predicted[1 - parity], "predicted[next]", 4));
    PRR_TRY(check_ptr(y.predicted_count[1 - parity], "predicted_count[next]", 4));
  }
  if (prr) {
    PRR_TRY(check_ptr(y.predicted[parity], "predicted[current]", 4));
    PRR_TRY(check_ptr(y.predicted_count[parity], "predicted_count[current]", 4));
  }
  if (sp->num_tokens < 1 || (int64_t)sp->num_tokens > (int64_t)dims->max_pages * dims->page_size)
    return fail(PRR_ERR_INVALID_ARG, "num_tokens %d outside [1, max_pages*page_size]", sp->num_tokens);
  const int npages_tok = div_up(sp->num_tokens, dims->page_size);
  if (sp->num_pages < 1 || sp->num_pages > npages_tok || sp->num_pages > PRR_MAX_PAGES)
    return fail(PRR_ERR_INVALID_ARG, "num_pages %d outside [1, min(ceil(num_tokens/page_size), %d)]", sp->num_pages,
                PRR_MAX_PAGES);
  if (sp->num_pages > prr::kFusedMaxPages)
    return fail(PRR_ERR_UNSUPPORTED, "fused schedules take at most %d pages (num_pages %d)", prr::kFusedMaxPages,
                sp->num_pages);
  if (sp->k_select < 0 || sp->p_select < 0)
    return fail(PRR_ERR_INVALID_ARG, "k_select %d / p_select %d < 0", sp->k_select, sp->p_select);
  PRR_TRY(check_forced(sp->forced, sp->n_forced, sp->num_pages));
  if (sp->cap < 1 || sp->cap > PRR_MAX_CAP) return fail(PRR_ERR_INVALID_ARG, "cap %d outside [1, %d]", sp->cap, PRR_MAX_CAP);
  if (!chunk_ok(dims, sp->chunk_pages))
    return fail(PRR_ERR_INVALID_ARG, "chunk_pages %d outside [1, 256 / page_size]", sp->chunk_pages);
  if (sp->mode != PRR_EXACT_SELECTED && sp->mode != PRR_KEEP_WASTED && sp->mode != PRR_RECOMPUTE_ON_MISS)
    return fail(PRR_ERR_INVALID_ARG, "mode %d", sp->mode);
  if (sp->late_spec < 0 || sp->late_spec > 2) return fail(PRR_ERR_INVALID_ARG, "late_spec %d", sp->late_spec);
  if (sp->epoch_dev) {
    PRR_TRY(check_ptr(sp->epoch_dev, "epoch_dev", 4));
  } else if (sp->epoch == 0) {
    return fail(PRR_ERR_INVALID_ARG, "epoch 0 is reserved (a zeroed workspace carries it)");
  }
  if (prr || prefill) PRR_TRY(check_theta(y.theta ? y.theta : &sp->alpha));
  int total_a, kextra_a, total_p, kextra_p;
  budget(sp->k_select, sp->n_forced, sp->forced_in_budget, sp->num_pages, total_a, kextra_a);
  budget(sp->p_select, sp->n_forced, sp->forced_in_budget, sp->num_pages, total_p, kextra_p);
  if (total_a > sp->cap) return fail(PRR_ERR_INVALID_ARG, "|A| = %d exceeds cap %d", total_a, sp->cap);
  if ((prr || prefill) && total_p > sp->cap) return fail(PRR_ERR_INVALID_ARG, "|P| = %d exceeds cap %d", total_p, sp->cap);
  PRR_TRY(check_ptr(y.workspace, "workspace", 256));
  WsLayout L;
  if (!ws_layout(dims, sp->cap, sp->chunk_pages, L) || y.ws_bytes < L.total)
    return fail(PRR_ERR_WORKSPACE, "workspace of %zu bytes too small (need %zu)", y.ws_bytes,
                ws_layout(dims, sp->cap, sp->chunk_pages, L) ? L.total : (size_t)0);
  prr::FusedLaunch a;
  memset(&a, 0, sizeof(a));
  a.q = y.q;
  a.meta = y.meta;
  a.k_cache = y.k_cache;
  a.v_cache = y.v_cache;
  a.page_table = y.page_table;
  a.level = y.ema_level;
  a.trend = y.ema_trend;
  a.init_bits = y.ema_init_bits;
  a.pred_cur = prr ? y.predicted[parity] : nullptr;
  a.pred_cur_count = prr ? y.predicted_count[parity] : nullptr;
  a.pred_nxt = y.predicted[1 - parity];
  a.pred_nxt_count = y.predicted_count[1 - parity];
  a.scores = y.scores;
  a.selected = y.selected;
  a.selected_count = y.selected_count;
  a.out_o32 = y.out_o32;
  a.out_o = y.out_o;
  a.out_m = y.out_m;
  a.out_l = y.out_l;
  a.missed_count = y.missed_count;
  a.wasted_count = y.wasted_count;
  a.covered_count = y.covered_count;
  char* ws = static_cast<char*>(y.workspace);
  a.t_score = reinterpret_cast<uint64_t*>(ws + L.f_score);
  a.t_thr = reinterpret_cast<uint64_t*>(ws + L.f_thr);
  a.t_mcnt = reinterpret_cast<uint64_t*>(ws + L.f_mcnt);
  a.t_mlist = reinterpret_cast<uint64_t*>(ws + L.f_mlist);
  a.t_part = reinterpret_cast<uint64_t*>(ws + L.f_part);
  a.part_o = reinterpret_cast<float*>(ws + L.f_parto);
  a.t_candk = reinterpret_cast<uint64_t*>(ws + L.f_candk);
  a.t_candp = reinterpret_cast<uint64_t*>(ws + L.f_candp);
  a.t_pkey = reinterpret_cast<uint64_t*>(ws + L.f_pkey);
  a.win = reinterpret_cast<uint32_t*>(ws + L.f_win);
  a.t_lcnt = reinterpret_cast<uint64_t*>(ws + L.f_lcnt);
  {
    uint32_t* pb = reinterpret_cast<uint32_t*>(ws + L.f_pbits);
    const size_t nwp = (size_t)dims->num_kv_heads * ((dims->max_pages + 31) / 32);
    a.pbits_cur = pb + (size_t)parity * nwp;
    a.pbits_nxt = pb + (size_t)(1 - parity) * nwp;
  }
  a.flags = reinterpret_cast<uint32_t*>(ws + L.flags);
  a.stamps = sp->phase_stamps ? reinterpret_cast<unsigned long long*>(sp->phase_stamps) +
                                    (size_t)layer * prr::kStampSlots * prr::kStampMaxWorkgroups
                              : nullptr;
  a.alpha = y.theta ? y.theta[0] : sp->alpha;
  a.beta = y.theta ? y.theta[1] : sp->beta;
  a.gamma = y.theta ? y.theta[2] : sp->gamma;
  a.epoch = sp->epoch;
  a.epoch_dev = sp->epoch_dev;
  a.schedule = prr ? 1 : (prefill ? 2 : 0);
  a.mode = sp->mode;
  a.num_kv_heads = dims->num_kv_heads;
  a.group = dims->num_q_heads / dims->num_kv_heads;
  a.max_pages = dims->max_pages;
  a.num_pages = sp->num_pages;
  a.num_tokens = sp->num_tokens;
  a.kextra_a = kextra_a;
  a.kextra_p = kextra_p;
  a.cap = sp->cap;
  a.chunk = sp->chunk_pages;
  a.n_score = div_up(sp->num_pages, prr::kFusedScorePages);
  a.n_spec = L.nchunks;
  a.n_miss = L.nchunks;
  a.late = prr && sp->late_spec && sp->mode != PRR_RECOMPUTE_ON_MISS;
  a.readahead = a.late && sp->late_spec == 1;  // (kept only if the grid is resident at once)
  a.n_late = a.late ? late_slots(dims, a.n_score, L.nchunks, sp->chunk_pages) : 0;
  a.miss_wgs = miss_workgroups(a.late, L.nchunks, sp->chunk_pages);
  a.nparts = L.nparts;
  a.n_forced = sp->n_forced;
  a.meta_mean = dims->meta_kind == PRR_META_MEAN;
  for (int i = 0; i < sp->n_forced; ++i) a.forced[i] = sp->forced[i];
  if (a.stamps && prr::fused_grid(a) > prr::kStampMaxWorkgroups)
    return fail(PRR_ERR_UNSUPPORTED, "phase_stamps record at most %d workgroups (grid %d)", prr::kStampMaxWorkgroups,
                prr::fused_grid(a));
  return hip_status(prr::launch_fused(a, dims->dtype == PRR_BF16, dims->page_size, stream), "fused step launch");
}

prr_status prr_decode_step(const prr_dims* dims, const prr_step_params* sp, const prr_layer_io* layers,
                           int32_t n_layers, int32_t parity, int32_t schedule, hipStream_t stream,
                           hipStream_t spec_stream, hipEvent_t* events) {
  PRR_TRY(check_dims(dims));
  if (!sp || !layers) return fail(PRR_ERR_INVALID_ARG, "params or layers is NULL");
  if (n_layers < 1) return fail(PRR_ERR_INVALID_ARG, "n_layers %d < 1", n_layers);
  if (parity != 0 && parity != 1) return fail(PRR_ERR_INVALID_ARG, "parity %d", parity);
  if (schedule < PRR_SCHED_SERIAL || schedule > PRR_SCHED_FUSED_PREFILL)
    return fail(PRR_ERR_INVALID_ARG, "schedule %d", schedule);
  if (schedule >= PRR_SCHED_FUSED_SERIAL) {
    if (dims->page_size != 16 && dims->page_size != 64)
      return fail(PRR_ERR_UNSUPPORTED, "page_size %d: the fused schedules are compiled for 16 and 64", dims->page_size);
    if (sp->phase_stamps && !aligned(sp->phase_stamps, 8)) return fail(PRR_ERR_INVALID_ARG, "phase_stamps misaligned");
    for (int l = 0; l < n_layers; ++l) PRR_TRY(fused_layer(dims, sp, layers[l], parity, schedule, stream, l));
    return ok();
  }
  // PRR_SCHED_TWO_STREAM without events: the library's stream-memory words order the streams
  ChainState* mem = nullptr;
  std::unique_lock<std::mutex> mem_lock(g_chain_mu, std::defer_lock);
  if (schedule == PRR_SCHED_TWO_STREAM && !events) {
    PRR_TRY(chain_state(mem));
    mem_lock.lock();
    PRR_TRY(stream_words(*mem, stream));
  }
  const int nxt = 1 - parity;
  for (int l = 0; l < n_layers; ++l) {
    const prr_layer_io& y = layers[l];
    const float* th = y.theta ? y.theta : &sp->alpha;  // (alpha, beta, gamma are consecutive)
    if (schedule != PRR_SCHED_SERIAL) PRR_TRY(check_theta(th));
    if (schedule == PRR_SCHED_SERIAL) {
      PRR_TRY(prr_score_topk(dims, y.q, y.meta, sp->num_pages, sp->k_select, sp->forced, sp->n_forced,
                             sp->forced_in_budget, y.scores, y.selected, y.selected_count, sp->cap, y.workspace,
                             y.ws_bytes, stream));
      PRR_TRY(prr_repair(dims, y.q, y.k_cache, y.v_cache, y.page_table, sp->num_tokens, sp->num_pages, y.selected,
                         y.selected_count, nullptr, nullptr, sp->cap, sp->chunk_pages, nullptr, nullptr, nullptr,
                         nullptr, sp->mode, y.out_o32, y.out_o, y.out_m, y.out_l, y.missed_count, y.wasted_count,
                         y.workspace, y.ws_bytes, stream));
    } else if (schedule == PRR_SCHED_PREFILL) {
      PRR_TRY(prr_score_topk(dims, y.q, y.meta, sp->num_pages, sp->k_select, sp->forced, sp->n_forced,
                             sp->forced_in_budget, y.scores, y.selected, y.selected_count, sp->cap, y.workspace,
                             y.ws_bytes, stream));
      PRR_TRY(prr_predict(dims, y.ema_level, y.ema_trend, y.ema_init_bits, y.scores, sp->num_pages, th[0], th[1],
                          th[2], sp->p_select, sp->forced, sp->n_forced, sp->forced_in_budget,
                          y.predicted[nxt], y.predicted_count[nxt], sp->cap, stream));
    } else {
      hipEvent_t fork = mem ? nullptr : events[3 * l], sel = mem ? nullptr : events[3 * l + 1],
                 spec = mem ? nullptr : events[3 * l + 2];
      PRR_TRY(stream_dep(stream, spec_stream, fork, mem, 2));
      PRR_TRY(prr_score_topk(dims, y.q, y.meta, sp->num_pages, sp->k_select, sp->forced, sp->n_forced,
                             sp->forced_in_budget, y.scores, y.selected, y.selected_count, sp->cap, y.workspace,
                             y.ws_bytes, stream));
      // (the selection's point on `stream`, waited for by the prediction below)
      const uint64_t sel_value = mem ? ++mem->value : 0;
      if (mem) PRR_TRY(hip_status(hipStreamWriteValue64(stream, mem->word[3], sel_value, 0), "stream write"));
      else PRR_TRY(hip_status(hipEventRecord(sel, stream), "event record"));
      PRR_TRY(prr_spec_attn(dims, y.q, y.k_cache, y.v_cache, y.page_table, sp->num_tokens, y.predicted[parity],
                            y.predicted_count[parity], sp->cap, sp->chunk_pages, y.part_o, y.part_m, y.part_l,
                            y.page_m, spec_stream));
      PRR_TRY(stream_dep(spec_stream, stream, spec, mem, 4));
      PRR_TRY(prr_repair(dims, y.q, y.k_cache, y.v_cache, y.page_table, sp->num_tokens, sp->num_pages, y.selected,
                         y.selected_count, y.predicted[parity], y.predicted_count[parity], sp->cap, sp->chunk_pages,
                         y.part_o, y.part_m, y.part_l, y.page_m, sp->mode, y.out_o32, y.out_o, y.out_m, y.out_l,
                         y.missed_count, y.wasted_count, y.workspace, y.ws_bytes, stream));
      if (mem)
        PRR_TRY(hip_status(hipStreamWaitValue64(spec_stream, mem->word[3], sel_value, hipStreamWaitValueGte, ~0ull),
                           "stream wait"));
      else PRR_TRY(hip_status(hipStreamWaitEvent(spec_stream, sel, 0), "stream wait"));
      PRR_TRY(prr_predict(dims, y.ema_level, y.ema_trend, y.ema_init_bits, y.scores, sp->num_pages, th[0], th[1],
                          th[2], sp->p_select, sp->forced, sp->n_forced, sp->forced_in_budget,
                          y.predicted[nxt], y.predicted_count[nxt], sp->cap, spec_stream));
    }
  }
  if (schedule == PRR_SCHED_TWO_STREAM) PRR_TRY(stream_dep(spec_stream, stream, mem ? nullptr : events[3 * n_layers], mem, 5));
  return ok();
}

}  // extern "C"
