// Launch descriptors passed by value to the kernels, and the launchers the C ABI calls
// after it has validated every argument.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "prr.h"

#define PRR_MAX_PAGES_DEV PRR_MAX_PAGES
#define PRR_MAX_CAP_DEV PRR_MAX_CAP

namespace prr {

struct MetaLaunch {
  const void* k_cache;
  const int32_t* page_table;
  void* meta;
  int num_kv_heads, max_pages, page_size, num_tokens, page_begin, page_end;
  bool bf16, meta_mean;
};

struct ScoreLaunch {
  const void* q;
  const void* meta;
  float* scores;
  int32_t* selected;
  int32_t* selected_count;
  uint32_t* counters;  // [Hkv], zero between calls
  int num_kv_heads, group, max_pages, num_pages, kextra, cap, n_forced;
  bool bf16, meta_mean;
  int32_t forced[PRR_MAX_FORCED];
};

struct PredictLaunch {
  float* level;
  float* trend;
  uint32_t* init_bits;
  const float* scores;
  int32_t* predicted;
  int32_t* predicted_count;
  float alpha, beta, gamma;
  int num_kv_heads, max_pages, num_pages, kextra, cap, n_forced;
  int32_t forced[PRR_MAX_FORCED];
};

struct SpecLaunch {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const int32_t* page_table;
  const int32_t* pages;
  const int32_t* page_count;
  float* part_o;
  float* part_m;
  float* part_l;
  float* page_m;
  int num_kv_heads, group, max_pages, num_pages, num_tokens, page_size, cap, chunk, nchunks;
  bool bf16;
};

struct RepairLaunch {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const int32_t* page_table;
  const int32_t* selected;
  const int32_t* selected_count;
  const int32_t* predicted;
  const int32_t* predicted_count;
  const float* part_o;
  const float* part_m;
  const float* part_l;
  const float* page_m;
  float* out_o32;
  void* out_o;
  float* out_m;
  float* out_l;
  int32_t* missed_count;
  int32_t* wasted_count;
  float* ws_o;        // [Hkv][nwork][G][128]
  float* ws_ml;       // [Hkv][nwork][G][2]
  uint32_t* ws_cnt;   // [2*Hkv], zero between calls
  uint32_t* flags;    // sticky error bits
  int num_kv_heads, group, max_pages, num_pages, num_tokens, page_size, cap, chunk, nchunks, nwork, nmerge_per_kv, mode;
  bool bf16;
};

// One layer's whole decode step in one launch (the fused schedules of prr_decode_step).
struct FusedLaunch {
  const void* q;
  const void* meta;
  const void* k_cache;
  const void* v_cache;
  const int32_t* page_table;
  float* level;
  float* trend;
  uint32_t* init_bits;
  const int32_t* pred_cur;        // P^t [Hkv][cap] (PRR)
  const int32_t* pred_cur_count;
  int32_t* pred_nxt;              // P^{t+1} (PRR, prefill)
  int32_t* pred_nxt_count;
  float* scores;
  int32_t* selected;
  int32_t* selected_count;
  float* out_o32;
  void* out_o;
  float* out_m;
  float* out_l;
  int32_t* missed_count;
  int32_t* wasted_count;
  int32_t* covered_count;  // pages of A \ P attended by late speculation, or NULL
  uint64_t* t_score;  // [Hkv][max_pages] tagged score bits
  uint64_t* t_thr;    // [Hkv][8 copies][32] tagged threshold of A (words 0, 1 of each copy)
  uint64_t* t_mcnt;   // [Hkv][8][32] tagged count of the missed list (bit 31: attended by the select workgroup)
  uint64_t* t_mlist;  // [Hkv][cap] tagged missed pages
  uint64_t* t_part;   // [Hkv][nparts][G][2] tagged (m, l) of the partial states
  float* part_o;      // [Hkv][nparts][G][128] their outputs (complete before (m, l) are stored)
  uint64_t* t_candk;  // [3][Hkv][n_score][132] tagged candidate count, then keys (A, P^{t+1}) or
                      //   physical pages (late)
  uint64_t* t_candp;  // [3][Hkv][n_score][128] tagged candidate pages (bit 31: forced, bit 30: late)
  uint64_t* t_pkey;   // [Hkv][max_pages] tagged keys of the next prediction (EMA)
  uint64_t* t_lcnt;   // [Hkv][8][32] tagged number of late-speculated pages
  uint32_t* win;      // [Hkv][4] candidate bounds (ratios to |q-bar|_1) for A, P, late, kept across steps
  const uint32_t* pbits_cur;  // [Hkv][ceil(max_pages/32)] bitmap of P^t (a hint for the late filter)
  uint32_t* pbits_nxt;        // bitmap of P^{t+1}
  uint32_t* flags;
  unsigned long long* stamps;  // [kStampSlots][kStampMaxWorkgroups] phase timestamps (s_memrealtime), or NULL
  float alpha, beta, gamma;
  uint32_t epoch;
  const uint32_t* epoch_dev;  // if set, the epoch is read from here (graph replays)
  int schedule;  // 0 serial, 1 PRR, 2 prefill
  int mode;
  int num_kv_heads, group, max_pages, num_pages, num_tokens;
  int kextra_a, kextra_p, cap, chunk;
  int n_score, n_spec, n_miss, n_late, nparts;  // workgroups per KV head; partial slots per KV head
  int miss_wgs;  // workgroups per KV head for the missed list (n_miss chunks, taken in turn)
  int late;  // late speculation on (PRR schedule)
  int readahead;  // score workgroups read the first late pages ahead (allowed; decided at launch)
  int n_forced;
  bool meta_mean;
  int32_t forced[PRR_MAX_FORCED];
};

// Phase timestamps of a fused launch (prr_step_params.phase_stamps): entry
// [slot][workgroup] holds the device clock when that workgroup reached the phase.
enum StampSlot {
  kStampStart = 0,
  kStampScores,        // a score workgroup's scores computed
  kStampCandidates,    // a score workgroup's candidate lists stored (complete)
  kStampGathered,      // the select workgroup holds every candidate
  kStampThreshold,     // T published
  kStampMissed,        // missed count published
  kStampSpec,          // a speculation state published
  kStampLate,          // a late-speculation state published
  kStampMiss,          // a missed-page state published
  kStampMerge,         // a merge workgroup's output written
  kStampSelectDone,    // the select workgroup's last work (next step's bounds) done
  kStampPredictDone,   // P^{t+1} written
  kStampEnd,           // a workgroup ends
  kStampAttended,      // an attending workgroup's page states computed
  kStampLateList,      // a late workgroup holds its list
  kStampSlots = 16
};
constexpr int kStampMaxWorkgroups = 1024;

constexpr int kFusedMaxPages = 8192;   // 16 keys per thread of a 512-thread select
constexpr int kFusedScorePages = 128;   // pages per score workgroup of the fused step
constexpr int kFusedWaves = 8;          // waves of a fused-step workgroup
template <bool BF16, int PS, int NPW>
hipError_t launch_fused_inst(int grid, const FusedLaunch& a, hipStream_t stream);
hipError_t launch_fused(const FusedLaunch& a, bool bf16, int page_size, hipStream_t stream);
int fused_grid(const FusedLaunch& a);
// workgroups of the fused kernel resident at once on the current device (0: unknown)
int fused_resident(bool bf16, int page_size, int chunk);

// The argument checks of prr_score_topk (everything but the workspace), filling the launch
// descriptor; shared with the entry point that allocates nothing.  Errors are recorded
// for prr_last_error.
prr_status prepare_score(const prr_dims* dims, const void* q, const void* meta, int32_t num_pages, int32_t k_select,
                         const int32_t* forced, int32_t n_forced, int32_t forced_in_budget, float* scores,
                         int32_t* selected, int32_t* selected_count, int32_t cap, ScoreLaunch& a);
prr_status api_fail(prr_status st, const char* fmt, ...);
prr_status api_ok();

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t stream);
hipError_t launch_empty(int grid, int threads, hipStream_t stream);
hipError_t launch_read_stream(const void* p, size_t bytes, uint32_t* sink, int grid, hipStream_t stream);
hipError_t launch_epoch_advance(uint32_t* epoch_dev, hipStream_t stream);
void calibrate_grid(const float* scores, int n_traj, int n_rows, int n_blocks, const int32_t* form_row, int k_select,
                    int p_select, const float* grid, int n_grid, int n_threads, float* best_theta,
                    double* objective_out);
float pick_delta(const int32_t* context, const float* delta, const float* select_us, const float* spec_us, int n_rows,
                 int32_t query_context, int degree, float* select_est, float* spec_est);
hipError_t launch_meta(const MetaLaunch& a, hipStream_t stream);
hipError_t launch_score_topk(const ScoreLaunch& a, hipStream_t stream);
hipError_t launch_predict(const PredictLaunch& a, hipStream_t stream);
hipError_t launch_spec_attn(const SpecLaunch& a, hipStream_t stream);
hipError_t launch_repair(const RepairLaunch& a, hipStream_t stream);
hipError_t launch_merge_states(int n_states, int rows, int d, const float* o, const float* m, const float* l,
                               float* out_o, float* out_m, float* out_l, hipStream_t stream);

}  // namespace prr
