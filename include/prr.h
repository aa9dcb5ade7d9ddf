/*
 * prr.h -- C ABI of the speculate-reuse-repair decode path for dynamic sparse
 * attention on AMD Instinct MI355X (gfx950).
 *
 * One decode step of one layer, batch 1, is:
 *
 *   select   prr_score_topk   Quest page metadata -> GQA criticality -> top-K set A
 *   predict  prr_predict      EMA update with this step's scores -> predicted set P
 *   speculate prr_spec_attn   split-K flash-decode over P (may run while select runs)
 *   repair   prr_repair       attend the missed pages A \ P and merge, so the result
 *                             is attention over exactly A (or over P u A, on request)
 *
 * Citations name sections, equations and the appendix of "Predict, Reuse, and
 * Repair: Accelerating Dynamic Sparse Attention for Long-Context LLM Decoding".
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every call returns prr_status.  PRR_OK is 0.  Arguments are validated on the host
 *   before anything is launched; on an error nothing is launched, the outputs are
 *   untouched and prr_last_error() (thread-local) says why.
 * - Every call is asynchronous on the hipStream_t it is given (NULL = the legacy
 *   default stream).  Device faults surface at the caller's next synchronisation.
 * - All device memory is owned by the caller.  The library never allocates, frees or
 *   synchronises.  Inputs are read-only.  Pointers marked "device" must be device
 *   memory (or host memory the device can access); "host" pointers are read during
 *   the call only.
 * - Layouts are dense row-major in the order written, with no padding.  Per-page
 *   arrays of a KV head have a row stride of max_pages entries; page lists have a row
 *   stride of `cap` entries.
 * - Calls are re-entrant.  Calls on different streams may run concurrently if they
 *   write disjoint memory and do not share one workspace region (see
 *   prr_workspace_size).
 * - Query head j belongs to KV head j / G (G = num_q_heads / num_kv_heads).
 * - Attention statistics: m is the maximum of the scaled logits q.k/sqrt(head_dim)
 *   (natural-log units), l = sum exp(logit - m), o is normalised (divided by l).
 *   The empty state is o = 0, m = -inf, l = 0.
 * - Page ids in lists are logical pages.  The logical page p holds tokens
 *   [p*page_size, (p+1)*page_size); tokens at or beyond num_tokens are masked.
 *   A device-side list entry outside [0, num_pages) is skipped (never dereferenced);
 *   lists must be duplicate-free, otherwise results are unspecified (but no memory
 *   outside the arguments is touched).
 */
#ifndef PRR_H_
#define PRR_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t prr_status;

#define PRR_OK 0
#define PRR_ERR_INVALID_ARG 1 /* a size, pointer or flag is out of range */
#define PRR_ERR_UNSUPPORTED 2 /* shape or dtype without a compiled kernel instance */
#define PRR_ERR_WORKSPACE 3   /* workspace missing, too small or misaligned */
#define PRR_ERR_HIP 4         /* a HIP runtime call failed (launch error) */

#define PRR_F16 0  /* IEEE binary16 */
#define PRR_BF16 1 /* bfloat16 */

#define PRR_META_MINMAX 0 /* Quest: channel-wise min and max key per page (Appendix A.1) */
#define PRR_META_MEAN 1   /* mean-pooled block key (the InfLLM-v2 style compression, Section 2.1) */

#define PRR_EXACT_SELECTED 0 /* output = attention over exactly A */
#define PRR_KEEP_WASTED 1    /* output = attention over P u A (wasted pages kept as context, Section 1) */
#define PRR_RECOMPUTE_ON_MISS 2 /* fused schedules only: output = attention over exactly A, but when
                                   any page of A was not predicted the speculation is discarded and
                                   all of A is attended afresh (the ablation stage without repair,
                                   Section 5.3) */

/* Shape of one layer's paged KV cache.
 *   head_dim   128 (the only compiled value)
 *   page_size  16, 32, 64, 128 or 256 tokens (the fused schedules of prr_decode_step: 16
 *              or 64; other sizes give PRR_ERR_UNSUPPORTED there)
 *   max_pages  page slots per KV head in the cache; also the row stride of per-page arrays
 *   dtype      PRR_F16 or PRR_BF16, for q, keys, values, min/max metadata and out_o
 *   meta_kind  PRR_META_MINMAX or PRR_META_MEAN
 * Constraints: 1 <= num_kv_heads, num_q_heads = G * num_kv_heads with 1 <= G <= 16. */
typedef struct {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t page_size;
  int32_t max_pages;
  int32_t dtype;
  int32_t meta_kind;
} prr_dims;

/* Largest supported values. */
#define PRR_MAX_PAGES 16384 /* num_pages per KV head handled by one select */
#define PRR_MAX_CAP 1024    /* entries of a page list (|A|, |P|) */
#define PRR_MAX_FORCED 64   /* forced pages */

const char* prr_status_string(prr_status status);
const char* prr_last_error(void);

/* Bytes of workspace used by prr_score_topk, prr_repair and the fused schedules of
 * prr_decode_step for lists of at most `cap` pages and speculation chunks of
 * `chunk_pages` pages.  The workspace holds disjoint regions (selection counters,
 * repair counters, repair partial states, the fused step's tagged hand-off buffers);
 * one prr_score_topk and one prr_repair may use the same workspace at the same time,
 * two calls of the same entry point may not.  Returns 0 if the arguments are invalid. */
size_t prr_workspace_size(const prr_dims* dims, int32_t cap, int32_t chunk_pages);

/* Zero a workspace (device, `bytes` long, 256-byte aligned) with a fill kernel on
 * `stream`.  Required once before first use; every call leaves its counters at zero
 * again when it finishes. */
prr_status prr_workspace_init(void* workspace, size_t bytes, hipStream_t stream);

/* Size in floats of the speculation output of prr_spec_attn for lists of at most
 * `cap` pages: part_o [Hkv][ceil(cap/C)][G][128], part_m and part_l
 * [Hkv][ceil(cap/C)][G], page_m [Hkv][cap][G]. */
size_t prr_spec_state_floats(const prr_dims* dims, int32_t cap, int32_t chunk_pages,
                             size_t* part_o_floats, size_t* part_ml_floats, size_t* page_m_floats);

/* Page metadata (Appendix A.1; block means for PRR_META_MEAN, Section 2.1).
 *   k_cache     device [Hkv][max_pages][page_size][128] dtype (physical pages)
 *   page_table  device [max_pages] int32 logical -> physical page, or NULL = identity
 *   num_tokens  tokens in the cache; a partial last page uses its valid tokens only
 *   page_begin, page_end   logical pages [begin, end) to (re)build; end <= ceil(num_tokens/page_size)
 *   meta        device, MINMAX: [Hkv][max_pages][2][128] dtype (row 0 = min, row 1 = max),
 *               MEAN: [Hkv][max_pages][128] float32.  Only pages [begin, end) are written.
 * Min and max are exact; the mean is summed in float32. */
prr_status prr_build_page_meta(const prr_dims* dims, const void* k_cache, const int32_t* page_table,
                               int32_t num_tokens, int32_t page_begin, int32_t page_end, void* meta,
                               hipStream_t stream);

/* Criticality scores and top-K page selection (Appendix A.1; Section 1).
 *   q            device [Hq][128] dtype, this step's query
 *   meta         device, as written by prr_build_page_meta
 *   num_pages    logical pages in the cache, 1..PRR_MAX_PAGES
 *   k_select     budget K >= 0 in pages
 *   forced       host [n_forced] int32 distinct pages in [0, num_pages) always selected
 *                (copied into the launch), or NULL if n_forced = 0
 *   forced_in_budget  1: |A| = max(K, n_forced) (forced pages count against K);
 *                0: |A| = K + n_forced.  |A| is capped at num_pages.
 *   scores       device [Hkv][max_pages] float32 out: IS = sum_i max(qbar_i m_i, qbar_i M_i)
 *                (MEAN: qbar . kbar), unscaled, with qbar the mean of the group's queries
 *   selected     device [Hkv][cap] int32 out: A in ascending page order
 *   selected_count device [Hkv] int32 out: |A|
 *   cap          row stride of `selected`, >= |A|, <= PRR_MAX_CAP
 * Ranking key: (float32 score descending, page index ascending).
 * Uses the selection-counter region of the workspace. */
prr_status prr_score_topk(const prr_dims* dims, const void* q, const void* meta, int32_t num_pages,
                          int32_t k_select, const int32_t* forced, int32_t n_forced, int32_t forced_in_budget,
                          float* scores, int32_t* selected, int32_t* selected_count, int32_t cap,
                          void* workspace, size_t ws_bytes, hipStream_t stream);

/* prr_score_topk without a workspace, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid allocation).
 * The arguments and results are those of prr_score_topk.  Its only scratch, one arrival
 * counter per KV head, is a static device array of PRR_STATIC_MAX_KV_HEADS words that
 * each GPU holds until the process ends; the call uses the copy of the current device and
 * clears it on `stream` (with a fill kernel) before the selection.  Every call on one GPU
 * shares that array: calls that overlap on one GPU (on different streams, or from
 * different threads) race and give undefined results.  No allocation, no
 * synchronisation.  Errors: those of prr_score_topk; PRR_ERR_INVALID_ARG when
 * num_kv_heads > PRR_STATIC_MAX_KV_HEADS; PRR_ERR_HIP when the array's device address
 * cannot be looked up. */
#define PRR_STATIC_MAX_KV_HEADS 256
prr_status prr_score_topk_static(const prr_dims* dims, const void* q, const void* meta, int32_t num_pages,
                                 int32_t k_select, const int32_t* forced, int32_t n_forced, int32_t forced_in_budget,
                                 float* scores, int32_t* selected, int32_t* selected_count, int32_t cap,
                                 hipStream_t stream);

/* EMA predictor (Section 4.1, Eqs. (2)-(3)) and the predicted set P (Eq. (1)).
 *   ema_level, ema_trend  device [Hkv][max_pages] float32 in/out (level l and trend v)
 *   ema_init_bits         device [Hkv][ceil(max_pages/32)] uint32 in/out: bit p set once
 *                         page p has state; zero them when the cache is (re)filled
 *   scores       device [Hkv][max_pages] float32 this step's IS, or NULL = predict only.
 *                With scores: for a page without state, l = IS, v = 0 and the bit is set;
 *                otherwise v = beta (IS - l) + (1 - beta) v, then l = alpha IS + (1 - alpha) l.
 *   alpha in (0,1], beta in (0,1], gamma in [0,1]
 *   p_select, forced, n_forced, forced_in_budget  as k_select etc. of prr_score_topk
 *   predicted    device [Hkv][cap] int32 out: the p_select pages with the largest
 *                l + gamma v (pages without state are never predicted unless forced),
 *                ascending page order, ties to the lower page index
 *   predicted_count device [Hkv] int32 out
 * One workgroup per KV head; no workspace. */
prr_status prr_predict(const prr_dims* dims, float* ema_level, float* ema_trend, uint32_t* ema_init_bits,
                       const float* scores, int32_t num_pages, float alpha, float beta, float gamma,
                       int32_t p_select, const int32_t* forced, int32_t n_forced, int32_t forced_in_budget,
                       int32_t* predicted, int32_t* predicted_count, int32_t cap, hipStream_t stream);

/* Speculative split-K sparse flash-decode over a page list (Section 4.3,
 * "Instrumented speculative kernel").
 *   q, k_cache, v_cache  device, [Hq][128], [Hkv][max_pages][page_size][128] dtype
 *   page_table   device [max_pages] int32 or NULL (identity)
 *   num_tokens   tokens in the cache (masks a partial last page)
 *   pages        device [Hkv][cap] int32 list (normally P), page_count device [Hkv] int32
 *   chunk_pages  C, 1 <= C <= 256 / page_size (16 for 16-token pages, 4 for 64-token
 *                pages, 1 for 256-token pages): consecutive list entries [cC, cC+C)
 *                form chunk c
 *   part_o       device [Hkv][ceil(cap/C)][G][128] float32 out: normalised o of each chunk
 *   part_m, part_l device [Hkv][ceil(cap/C)][G] float32 out
 *   page_m       device [Hkv][cap][G] float32 out: max scaled logit of each listed page,
 *                or NULL (then prr_repair recomputes every chunk that holds a wasted page)
 * Only chunks with at least one listed page are written. */
prr_status prr_spec_attn(const prr_dims* dims, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* page_table, int32_t num_tokens, const int32_t* pages,
                         const int32_t* page_count, int32_t cap, int32_t chunk_pages, float* part_o,
                         float* part_m, float* part_l, float* page_m, hipStream_t stream);

/* Repair (Section 4.3, Eqs. (6)-(8)): fold the missed pages M = A \ P into the
 * speculative state and merge, in one kernel.
 *   selected, selected_count   A and |A| (device, as from prr_score_topk)
 *   predicted, predicted_count P and |P| (device, as given to prr_spec_attn), or both
 *                NULL: P is empty and every page of A is attended here (the serial
 *                select-then-attend path)
 *   part_o, part_m, part_l, page_m   the speculation output of prr_spec_attn over P
 *                with the same cap and chunk_pages (ignored when P is NULL)
 *   mode         PRR_EXACT_SELECTED: chunks of P that hold a wasted page (P \ A) have
 *                the wasted pages' contribution removed: re-attended and subtracted when
 *                they carry at most 7/8 of the chunk's softmax mass for every query head
 *                (the remaining part then holds at least 1/8 of it, so the subtraction
 *                amplifies float32 rounding at most 8-fold), otherwise the chunk's pages
 *                of A are re-attended; PRR_KEEP_WASTED: P u A is attended
 *   out_o32      device [Hq][128] float32 out, out_o device [Hq][128] dtype out or NULL
 *   out_m, out_l device [Hq] float32 out
 *   missed_count, wasted_count  device [Hkv] int32 out: |A \ P|, |P \ A|
 * Uses the repair regions of the workspace. */
prr_status prr_repair(const prr_dims* dims, const void* q, const void* k_cache, const void* v_cache,
                      const int32_t* page_table, int32_t num_tokens, int32_t num_pages,
                      const int32_t* selected, const int32_t* selected_count, const int32_t* predicted,
                      const int32_t* predicted_count, int32_t cap, int32_t chunk_pages,
                      const float* part_o, const float* part_m, const float* part_l, const float* page_m,
                      int32_t mode, float* out_o32, void* out_o, float* out_m, float* out_l,
                      int32_t* missed_count, int32_t* wasted_count, void* workspace, size_t ws_bytes,
                      hipStream_t stream);

/* ---------------------------------------------------------------------------------
 * Decode-step runtime: one token over a stack of layers, launched natively.
 * --------------------------------------------------------------------------------- */

/* Device buffers of one layer (all as described for the calls above). */
typedef struct {
  const void* q;           /* [Hq][128] this step's query of the layer */
  const void* k_cache;
  const void* v_cache;
  const int32_t* page_table; /* or NULL */
  const void* meta;
  float* scores;
  float* ema_level;
  float* ema_trend;
  uint32_t* ema_init_bits;
  int32_t* selected;
  int32_t* selected_count;
  int32_t* predicted[2];       /* double-buffered P: P^t in [parity], P^{t+1} goes to [1 - parity] */
  int32_t* predicted_count[2];
  float* part_o;
  float* part_m;
  float* part_l;
  float* page_m;
  float* out_o32;
  void* out_o;                 /* or NULL */
  float* out_m;
  float* out_l;
  int32_t* missed_count;       /* or NULL */
  int32_t* wasted_count;       /* or NULL */
  void* workspace;
  size_t ws_bytes;
  int32_t* covered_count;      /* or NULL: [Hkv] pages of A \ P attended by late speculation
                                  (fused PRR schedule; 0 otherwise) */
  const float* theta;          /* or NULL: HOST [3] (alpha, beta, gamma) of this layer's EMA
                                  predictor (Section 4.2 calibrates one per layer), in place of
                                  the step's; read when the call is made (a captured graph keeps
                                  the values of capture time); same ranges as the step's */
} prr_layer_io;

/* Per-step parameters shared by the layers. */
typedef struct {
  int32_t num_tokens;
  int32_t num_pages;
  int32_t k_select;
  int32_t p_select;            /* |P| budget (delta |A|) */
  int32_t cap;
  int32_t chunk_pages;
  int32_t mode;                /* PRR_EXACT_SELECTED | PRR_KEEP_WASTED | PRR_RECOMPUTE_ON_MISS (fused) */
  int32_t forced_in_budget;
  int32_t n_forced;
  const int32_t* forced;       /* host [n_forced] */
  float alpha, beta, gamma;
  uint32_t epoch;              /* fused schedules: >= 1 and different from every earlier call's
                                  value on the same workspaces (e.g. the token index + 1) */
  const uint32_t* epoch_dev;   /* fused schedules, or NULL: device word read by each launch
                                  instead of `epoch`, for launches captured once and replayed
                                  (HIP graphs); the caller advances it between replays with
                                  prr_epoch_advance, under the same uniqueness rule */
  int32_t late_spec;           /* PRR_SCHED_FUSED_PRR: 1 = also speculate, as soon as this step's
                                  scores exist, over the pages just above the selection threshold
                                  that P missed (the threshold is learned across steps); the result
                                  is still attention over exactly A (or P u A).  With 1 the score
                                  workgroups also read the first late pages ahead into the
                                  memory-side cache when the launch's grid is resident at once
                                  (those lines are then fetched twice); 2 = late speculation
                                  without the read-ahead; 0 = none; other values give
                                  PRR_ERR_INVALID_ARG */
  uint64_t* phase_stamps;      /* fused schedules, or NULL: device [n_layers][16][1024] zeroed by the
                                  caller; entry [l][k][w] receives the device real-time clock
                                  (100 MHz, s_memrealtime) when workgroup w of layer l's launch
                                  reached phase k (0 = never): 0 start; 1 scores computed; 2
                                  candidate lists stored; 3 candidates gathered (select and
                                  predict workgroups); 4 threshold published (predict: found);
                                  5 missed count published (predict: its middle path taken);
                                  6, 7, 8 a speculation, late or missed-page state published; 9
                                  an output row written; 10 select done (predict: its full
                                  gather taken); 11 next prediction written; 12 the workgroup's
                                  last wave ended; 13 an attending workgroup's page states
                                  computed; 14 a late workgroup holds its list.  One plain store
                                  per entry (12: an atomic maximum per wave).  Grids above 1024
                                  workgroups give PRR_ERR_UNSUPPORTED. */
} prr_step_params;

#define PRR_SCHED_SERIAL 0     /* per layer: select, then attend every page of A (one stream) */
#define PRR_SCHED_TWO_STREAM 1 /* per layer: select on `stream` while speculating over P on `spec_stream`,
                                  repair on `stream`, EMA update + next prediction on `spec_stream` */
#define PRR_SCHED_PREFILL 2    /* per layer: select, then initialise the EMA state and predict P (step 0) */
/* The same three steps, each layer as ONE launch on `stream` whose workgroups take the
 * roles of the separate kernels (score, select, predict, speculate, attend missed pages,
 * merge) and hand results to each other inside the launch, so selection and speculation
 * overlap without a second stream.  In the fused PRR step the speculation keeps one
 * softmax state per page of P and folds only the pages that turn out to be in A, so
 * PRR_EXACT_SELECTED needs no recomputation.  Fused schedules need page_size 16 or 64,
 * num_pages <= 8192, p_select <= cap, and use the fused region of the workspace
 * (prr_workspace_size). */
#define PRR_SCHED_FUSED_SERIAL 3
#define PRR_SCHED_FUSED_PRR 4
#define PRR_SCHED_FUSED_PREFILL 5

/* One decode step over n_layers layers in order (layer l+1 starts after layer l's output is
 * written on `stream`): the select / speculate / repair / predict steps of Fig. 1 and
 * Section 4 launched from native code with the fork/join of two streams.
 *   events      host [3 * n_layers + 1] hipEvent_t created by the caller (timing may be
 *               disabled) for the fork/join of PRR_SCHED_TWO_STREAM, else ignored; NULL
 *               with PRR_SCHED_TWO_STREAM orders the two streams with stream memory writes
 *               and waits instead (hipStreamWriteValue64 / hipStreamWaitValue64 on four
 *               64-bit words that the library allocates once per device and keeps until the
 *               process ends; the first such call on a device zeroes them and waits for
 *               `stream`; a dependency costs about half an event wait here).  Those
 *               words are shared: two-stream steps without events that run at the same time
 *               on one device (from several host threads) must not be enqueued; with events
 *               they may.  PRR_ERR_UNSUPPORTED when the device has no stream memory waits.
 *   parity      0 or 1: which predicted buffer holds P^t
 * When the call returns every launch is enqueued; all work of the step is ordered
 * before any later work on `stream` (the speculation stream is joined back).  The
 * arguments of every layer are validated as by the individual calls; on an error in
 * layer l, layers before l have been enqueued. */
prr_status prr_decode_step(const prr_dims* dims, const prr_step_params* params, const prr_layer_io* layers,
                           int32_t n_layers, int32_t parity, int32_t schedule, hipStream_t stream,
                           hipStream_t spec_stream, hipEvent_t* events);

/* Workgroups of one layer's launch of a fused schedule with these parameters (the
 * launch-floor measurement compares it with an empty launch of the same shape); 0 for
 * invalid arguments or a schedule that is not fused. */
int32_t prr_fused_grid(const prr_dims* dims, const prr_step_params* params, int32_t schedule);

/* Measurement helper: an empty kernel of `grid` workgroups of `threads` threads on
 * `stream` (the launch floor of a grid of that shape).  Errors: PRR_ERR_INVALID_ARG for a
 * grid outside [1, 2^20] or threads outside [1, 1024]. */
prr_status prr_empty_launch(int32_t grid, int32_t threads, hipStream_t stream);

/* Measurement helper: reads each 16-byte word of the device buffer `buf` (`bytes` long)
 * once, with `grid` workgroups of 256 threads on `stream`, and writes one word per
 * workgroup to the device array `sink` (grid words; their values are meaningless): the
 * chip's read-stream rate for a kernel of this library's access pattern.  Errors:
 * PRR_ERR_INVALID_ARG for a NULL or misaligned pointer (buf 16 bytes, sink 4), `bytes`
 * not a positive multiple of 16, or a grid outside [1, 2^20]. */
prr_status prr_read_stream(const void* buf, size_t bytes, uint32_t* sink, int32_t grid, hipStream_t stream);

/* Measurement helper: the cost of a dependency between two streams.  `n_hops` one-workgroup
 * empty launches alternate between streams `a` and `b`, each followed by a dependency of
 * the other stream on it: PRR_CHAIN_EVENTS records an event that the other stream waits
 * for (hipStreamWaitEvent); PRR_CHAIN_STREAM_MEMORY writes a 64-bit value that the other
 * stream waits for (hipStreamWriteValue64 / hipStreamWaitValue64, greater-or-equal);
 * PRR_CHAIN_ONE_STREAM launches all of them on `a` without dependencies (`b` unused).  The
 * chain ends on `a`, and all of it is enqueued here, so a timing on `a` around the call
 * measures the device's cost per hop, not the caller's.  The events and the two
 * stream-memory words are made on first use, once per device, and kept until the process
 * ends; values only grow, so calls made one after the other share them, but chains that run
 * at the same time on one device (from several host threads) must not be enqueued.  Errors:
 * PRR_ERR_INVALID_ARG for n_hops odd or outside [2, 256], an unknown mode, or a == b with a
 * dependency; PRR_ERR_UNSUPPORTED when the device has no stream memory waits; PRR_ERR_HIP. */
#define PRR_CHAIN_ONE_STREAM 0
#define PRR_CHAIN_EVENTS 1
#define PRR_CHAIN_STREAM_MEMORY 2
prr_status prr_stream_chain(int32_t n_hops, int32_t mode, hipStream_t a, hipStream_t b);

/* Advance the device epoch word of captured fused steps (prr_step_params.epoch_dev)
 * by one, skipping 0: one single-thread launch on `stream`, so it can be captured with
 * the steps it precedes.  Errors: PRR_ERR_INVALID_ARG for a NULL or misaligned pointer. */
prr_status prr_epoch_advance(uint32_t* epoch_dev, hipStream_t stream);

/* Online calibration of the EMA predictor (Section 4.2): for each candidate theta =
 * (alpha, beta, gamma) of `grid`, the score-weighted hit rate of Eq. (4) -- the EMA of
 * Eqs. (2)-(3) simulated over each prefill trajectory, P_phi = top-p_select of the
 * prediction, A_phi = top-k_select of row phi (ties: lower block index; keys rounded to
 * float32 as on the device) -- and the argmax of Eq. (5) (the first grid point on ties).
 * Blocks form as the prefill grows: block b exists from row form_row[b] on; its state
 * starts there as (level = its score, trend = 0), as Section 4.1 initialises a block when
 * it enters the cache.  A_phi ranks the blocks that exist at row phi, P_phi the blocks
 * that had a state before row phi.  The hit rates of rows 1..n_rows-1 (the rows with a
 * prediction) are averaged, then over the trajectories.  Host code, run on the CPU while
 * the device finishes the prefill; no device memory is touched.
 *   scores         host [n_traj][n_rows][n_blocks] float32 prefill score trajectories;
 *                  entries of blocks that do not exist yet at a row are never read
 *   form_row       host [n_blocks] int32 >= 0, the row at which each block forms (shared by
 *                  the trajectories), or NULL = every block exists from row 0
 *   k_select       |A_phi|; p_select: |P_phi| (0 = k_select)
 *   grid           host [n_grid][3] float32, alpha, beta in (0, 1], gamma in [0, 1]
 *   n_threads      host threads (0 = all hardware threads)
 *   best_theta     host [3] out: the argmax
 *   objective_out  host [n_grid] out (may be NULL): Eq. (4) per grid point
 * Errors: PRR_ERR_INVALID_ARG for NULL pointers, sizes < 1 (n_rows < 2), a negative
 * form_row entry, a grid point out of range. */
prr_status prr_calibrate(const float* scores, int32_t n_traj, int32_t n_rows, int32_t n_blocks,
                         const int32_t* form_row, int32_t k_select, int32_t p_select, const float* grid,
                         int32_t n_grid, int32_t n_threads, float* best_theta, double* objective_out);

/* Critical-path-aware speculation budget (Section 4.4): the largest delta = |P| / |A|
 * whose speculation latency fits within the selection window at `query_context`, from a
 * table profiled offline (one row per context length and delta).  At a profiled context
 * the row's latencies are used as measured; at any other context each delta's selection
 * and speculation latencies are estimated by least-squares polynomial regression in
 * log2(context) over that delta's rows (appendix "Profiling Overheads"), of degree
 * min(degree, distinct profiled contexts - 1).  Host code.
 *   context, delta, select_us, spec_us  host [n_rows] table columns (context >= 1,
 *                delta >= 1, latencies >= 0), or NULL when n_rows = 0
 *   degree       0..3
 *   delta_out    host out: the chosen delta; 1 when no delta fits or the table is empty
 *   select_est, spec_est  host out or NULL: the latencies of the chosen delta (estimated
 *                or measured) at query_context (of the smallest profiled delta when none
 *                fits; NaN when the table is empty)
 * Errors: PRR_ERR_INVALID_ARG for NULL pointers, n_rows < 0, query_context < 1, a
 * degree outside [0, 3], a table row out of range. */
prr_status prr_pick_delta(const int32_t* context, const float* delta, const float* select_us, const float* spec_us,
                          int32_t n_rows, int32_t query_context, int32_t degree, float* delta_out, float* select_est,
                          float* spec_est);

/* Merge n_states partial states per row (Eqs. (6)-(8) for arbitrary states).
 *   o  device [n_states][rows][d] float32, m, l device [n_states][rows] float32
 *   out_o device [rows][d], out_m, out_l device [rows]; d <= 1024; states with l = 0 are empty. */
prr_status prr_merge_states(int32_t n_states, int32_t rows, int32_t d, const float* o, const float* m,
                            const float* l, float* out_o, float* out_m, float* out_l, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PRR_H_ */
