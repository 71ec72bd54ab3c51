/*
 * mkv.h — C ABI of libmkv: decode attention over a KV cache held under one of
 * MetaKV's KV-cache compression configurations, on one AMD Instinct MI355X
 * (gfx950).
 *
 * The paper (MetaKV, arXiv 2609.07966) picks one compression configuration
 * per prompt (Section 2.3) from uncompressed FP16, KVQuant b-bit quantization,
 * H2O heavy-hitter eviction and RocketKV (SnapKV prefill eviction + hybrid
 * sparse attention) (Section 2.1, Table 1).  This library runs the decode step
 * of a batch in which every sequence carries its own configuration.
 *
 * Conventions that hold for every call:
 *   - fp16 tensors are uint16_t* holding IEEE binary16 bit patterns.
 *   - Every device pointer is owned by the caller; the library never
 *     allocates device memory.  The cache lives in a caller-provided arena.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Calls validate on the host, enqueue on `stream` and return without
 *     synchronising (mkv_export and mkv_fit_codebooks are synchronous).
 *     Inputs must stay live until the stream has consumed them.  Every
 *     kernel runs on `stream` itself (the library owns no streams or events
 *     outside profiling); use one stream for the decode calls of a step.
 *   - A call that fails validation returns an error, enqueues nothing and
 *     leaves the handle unchanged; mkv_last_error() then describes it.
 *   - One host thread at a time per handle; distinct handles are independent.
 *   - Tensor shapes: S = n_seqs, Hq = n_q_heads, Hkv = n_kv_heads,
 *     G = Hq / Hkv, d = head_dim.  Query head j belongs to kv head j / G.
 *   - Positions count from 0 over a sequence's prompt followed by its
 *     generated tokens.
 */
#ifndef MKV_H
#define MKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MKV_OK = 0,
  MKV_EINVAL = 1,        /* bad argument, shape or configuration */
  MKV_ENOMEM = 2,        /* arena smaller than mkv_cache_bytes() */
  MKV_ECAPACITY = 3,     /* more decode steps than max_new_tokens */
  MKV_ESTATE = 4,        /* call out of order (see the call order below) */
  MKV_EUNSUPPORTED = 5,  /* valid but not built (e.g. head_dim not 64/128) */
  MKV_EHIP = 6           /* a HIP runtime call failed */
} mkv_status;

/* Compression methods (Section 2.1). */
typedef enum {
  MKV_FP16 = 0,    /* uncompressed cache */
  MKV_UQ = 1,      /* uniform b-bit: keys per channel over `group`-token blocks,
                      values per token over `group`-channel groups; keys of an
                      incomplete final block stay fp16 */
  MKV_KVQ = 2,     /* KVQuant-style non-uniform b-bit: keys per channel with a
                      threshold frozen at prefill, values per token, values
                      above the threshold kept as fp16 outliers */
  MKV_H2O = 3,     /* heavy-hitter eviction at budget_pct % of the prompt */
  MKV_ROCKET = 4   /* SnapKV prefill eviction to keep_tokens, then top-k
                      sparse decode attention */
} mkv_method;

/* One sequence's configuration.  Unused fields are ignored. */
typedef struct {
  int32_t method;       /* mkv_method */
  int32_t bits;         /* UQ: 4.  KVQ: 2, 3 or 4 */
  int32_t group;        /* UQ: 64 */
  int32_t outlier_bp;   /* KVQ: outlier fraction in basis points (100 = 1 %),
                           0..5000; 0 disables outliers */
  int32_t budget_pct;   /* H2O: budget B = floor(budget_pct * prompt_len / 100)
                           tokens, of which floor(B/2) most recent; 1..10000 */
  int32_t keep_tokens;  /* ROCKET: tokens SnapKV keeps after prefill (>= window) */
  int32_t window;       /* ROCKET: observation window rows (32) */
  int32_t pool;         /* ROCKET: odd max-pool kernel over votes (7) */
  int32_t topk;         /* ROCKET: tokens attended per decode step; 0 = keep_tokens/2 */
  int32_t n_channels;   /* ROCKET: query channels used for approximate scores (32) */
  int32_t keep_ratio;   /* ROCKET: when > 0, SnapKV keeps max(floor(prompt_len / keep_ratio),
                           window) tokens instead of keep_tokens (the paper's r-times
                           compression settings, Section 2.1, RocketKV paragraph) */
} mkv_config;

typedef struct {
  int32_t n_seqs;          /* >= 1 */
  int32_t n_q_heads;       /* multiple of n_kv_heads; G = n_q_heads / n_kv_heads in {1,2,4,8} */
  int32_t n_kv_heads;      /* >= 1 */
  int32_t head_dim;        /* 64 or 128 */
  int32_t max_new_tokens;  /* decode steps the cache is sized for */
} mkv_shape;

typedef struct mkv_cache mkv_cache;  /* opaque host handle */

/* Static text for a status code. */
const char *mkv_status_str(mkv_status s);
/* Detail of the last failed call on this thread ("" if none). */
const char *mkv_last_error(void);

/*
 * Bytes of device arena a cache needs: all per-sequence cache regions,
 * prefill staging and the decode workspace.  cfg and prompt_len are host
 * arrays of n_seqs entries; prompt_len[s] >= 1.
 */
mkv_status mkv_cache_bytes(const mkv_shape *shape, const mkv_config *cfg,
                           const int32_t *prompt_len, size_t *arena_bytes);

/*
 * Lay out a cache in `arena` (device, >= arena_bytes, 256-byte aligned) and
 * initialise its device state on `stream` (this call waits for that
 * initialisation before returning).  codebooks: host float32, required when
 * any sequence uses MKV_KVQ, else may be NULL: for b = 2, 3, 4 in that order,
 * the key codebook (2^b ascending entries) then the value codebook (2^b
 * ascending entries): 56 floats in all, each exactly an fp16 value (the
 * codebook is stored in fp16, like the cache's other values; MKV_EINVAL
 * otherwise).  They are copied.
 * On success *out owns host metadata only; the arena stays the caller's.
 */
mkv_status mkv_cache_create(const mkv_shape *shape, const mkv_config *cfg,
                            const int32_t *prompt_len, const float *codebooks,
                            void *arena, size_t arena_bytes, void *stream,
                            mkv_cache **out);

/* Free the host handle (not the arena).  NULL is accepted. */
mkv_status mkv_cache_destroy(mkv_cache *cache);

/*
 * Append keys and values (Section 2.1: every method first writes the new
 * token's key and value into its cache; KVQuant and the uniform quantizer
 * quantize them on the way in).
 *   k, v   device fp16 [cu_new[S]][Hkv][d], sequence s owning rows
 *          cu_new[s] .. cu_new[s+1]-1
 *   cu_new host int32 [S+1] prefix offsets
 * First call (prefill): every sequence appends exactly prompt_len[s] rows;
 * KVQ calibrates its per-channel key thresholds here.  Later calls (decode):
 * one row per sequence.
 */
mkv_status mkv_append_quantize(mkv_cache *cache, const uint16_t *k, const uint16_t *v,
                               const int32_t *cu_new, void *stream);

/*
 * H2O (Section 2.1, H2O paragraph).
 * After the prefill append, with q_prompt = device fp16 [sum of prompt_len over
 * the H2O sequences][Hq][d] (those sequences' prompt queries, in sequence
 * order): score every prompt token by the causal attention it receives from
 * all prompt rows, summed over the kv head's query heads, and keep the
 * floor(B/2) most recent tokens plus the highest-scoring rest (newer wins a
 * tie).
 * After each decode mkv_decode_attention, with q_prompt = NULL: if a kv head
 * holds more than B tokens, evict the lowest-score token among those older
 * than the floor(B/2) most recent (older wins a tie).  The attention pass has
 * already chosen that token; this call removes it from the retained set
 * (mkv_export no longer reports it) and enqueues nothing: the next decode
 * append writes its token into the freed slot.
 * A no-op when no sequence uses H2O.
 */
mkv_status mkv_h2o_update_evict(mkv_cache *cache, const uint16_t *q_prompt, void *stream);

/*
 * RocketKV first stage, SnapKV (Section 2.1, RocketKV paragraph), once after
 * the prefill append.  q_window: device fp16 [sum over ROCKET sequences of
 * window][Hq][d]: each one's last `window` prompt query rows ending at its
 * last prompt token (when prompt_len < window only the last prompt_len of
 * them are read).  Per kv head, prompt tokens before the window are voted for
 * by the window rows' causal attention, summed over rows and the kv head's
 * query heads, max-pooled with kernel `pool`; the keep_tokens - window best
 * (lower position on ties) are kept together with the window.
 */
mkv_status mkv_snap_prefill_evict(mkv_cache *cache, const uint16_t *q_window, void *stream);

/*
 * RocketKV second stage, token selection (Section 2.1, RocketKV paragraph),
 * after each decode append.  q: device fp16 [S][Hq][d].  Per ROCKET kv head,
 * the n_channels largest sum_g |q_gc| channels (lower index on ties) give
 * approximate scores sum_c qbar_c k_jc (qbar = sum_g q_g), float32 in
 * ascending channel and head order without fused multiply-add, and the
 * min(topk, n) highest (lower position on ties) are selected.
 * pos_out: optional device int32 [S][Hkv][topk_max]; when non-NULL the
 * selected positions (ascending, -1 padded) are also written there; topk_max
 * is the largest effective topk over the ROCKET sequences.
 */
mkv_status mkv_topk_select(mkv_cache *cache, const uint16_t *q, int32_t *pos_out, void *stream);

/*
 * One decode step's attention for every sequence (Section 2.1: each method
 * ends in attention over what its cache keeps; Section 2.3: one configuration
 * per prompt, so a batch mixes methods): softmax(q k~ / sqrt(d)) v~ over the
 * tokens the sequence's method keeps (all tokens for FP16, UQ and KVQ with
 * k~, v~ their dequantized values; the retained set for H2O, whose
 * accumulated scores are updated here; the selected set for ROCKET).
 *   q   device fp16 [S][Hq][d]
 *   out device float32 [S][Hq][d]
 */
mkv_status mkv_decode_attention(mkv_cache *cache, const uint16_t *q, float *out, void *stream);

/*
 * mkv_decode_attention for callers that cannot allocate device memory, or
 * must not touch the cache arena's workspace, during a step (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation).
 * Same arguments, order rules and results as mkv_decode_attention; the
 * split-K partials of the attention tiles go to a static device workspace of
 * 8 MiB per GPU (held until the process ends) instead of the arena.  Calls no
 * allocating routine.  MKV_ENOMEM if the step's partials (attention tiles x
 * G x (d + 2) floats; see mkv_attention_tiles) exceed 8 MiB.  All calls on one
 * GPU share the workspace: calls that overlap on one GPU (other streams,
 * other handles, other threads) race and must be serialised by the caller.
 * The device that is current must be the cache's device.
 */
mkv_status mkv_decode_attention_noalloc(mkv_cache *cache, const uint16_t *q, float *out, void *stream);

/*
 * The four decode calls in their order (one decode step of Section 2.1's
 * methods, each sequence under its own configuration as Section 2.3 selects
 * per prompt): append (k, v: device fp16 [S][Hkv][d]), top-k select,
 * attention (q, out as for mkv_decode_attention), eviction.  Every argument
 * and the call order are checked before the first kernel is enqueued: a
 * rejected step (MKV_EINVAL for a NULL pointer, MKV_ESTATE, MKV_ECAPACITY)
 * enqueues nothing and leaves the handle unchanged.  Only MKV_EHIP can come
 * after a launch, and then the step may be partly enqueued.
 *
 * With RocketKV sequences in the batch the step's append launch also computes
 * their approximate scores, spread over several workgroups per kv head, and a
 * selection launch follows (the effect is that of the two calls in order).
 *
 * Graph capture: the step enqueues three or four kernels on `stream` (the
 * append, with the scores when RocketKV sequences are present; their
 * selection; attention partial; combine) and nothing else (no allocation,
 * copy, memset or synchronization; profiling events only when enabled), and
 * every per-step quantity (counts, positions, H2O eviction candidates,
 * outlier fills) lives in device state, so a captured step may be replayed
 * any number of times with new k, v, q written into the captured buffers.
 * The host-side step count then no longer follows the device: capacity is
 * also checked on the device, where an append into a full region drops the
 * token and leaves that (sequence, kv head) unchanged.
 */
mkv_status mkv_decode_step(mkv_cache *cache, const uint16_t *k, const uint16_t *v,
                           const uint16_t *q, float *out, void *stream);

/*
 * Copy one piece of state of (seq, kv_head) to host memory, synchronously
 * (waits for all work on the device).  `cap` is the capacity of host_dst in
 * bytes; *written receives the bytes written.  Arrays are in ascending
 * position order for FP16/UQ/KVQ/ROCKET token arrays and for H2O retained sets.
 */
typedef enum {
  MKV_EXPORT_COUNTS = 0,       /* int32[4]: tokens held, next position, attended count, kept-after-prefill */
  MKV_EXPORT_POSITIONS = 1,    /* int32[n]: positions held (H2O/ROCKET retained set; else 0..n-1) */
  MKV_EXPORT_CODES_K = 2,      /* uint8[n][d]: KVQ key codes; UQ: codes of the full 64-token blocks */
  MKV_EXPORT_CODES_V = 3,      /* uint8[n][d]: KVQ / UQ value codes */
  MKV_EXPORT_OUTLIERS_K = 4,   /* int32[n][d]: KVQ key outlier fp16 bits, -1 where none */
  MKV_EXPORT_OUTLIERS_V = 5,   /* int32[n][d]: KVQ value outlier fp16 bits, -1 where none */
  MKV_EXPORT_SCALES_K = 6,     /* KVQ: float32[d] thresholds tau_c.  UQ: float32[nblk][d][2] (min, step) */
  MKV_EXPORT_SCALES_V = 7,     /* KVQ: float32[n] per-token scales.  UQ: float32[n][d/64][2] (min, step) */
  MKV_EXPORT_SCORES = 8,       /* H2O: float32[n] accumulated scores, in POSITIONS order */
  MKV_EXPORT_TOPK = 9,         /* ROCKET: int32[m] positions selected by the last mkv_topk_select */
  MKV_EXPORT_CHANNELS = 10     /* ROCKET: int32[n_channels] channels used by the last mkv_topk_select */
} mkv_export_what;

mkv_status mkv_export(mkv_cache *cache, int32_t seq, int32_t kv_head, int32_t what,
                      void *host_dst, size_t cap, size_t *written);

/*
 * Fit one KVQ codebook pair on host data (synchronous, host only): the keys
 * are normalised per (kv head, channel) by their outlier threshold over the
 * n_tokens rows, the values per token by theirs (same rules as the cache),
 * and a 2^bits-entry codebook is fitted by 1-D Lloyd k-means (quantile
 * start, nearest entry with ties to the lower one, empty clusters keep their
 * centre, at most 100 iterations) to the non-outlier normalised values; the
 * centres are then rounded to fp16 (nearest even), the codebook's stored form.
 *   k, v     host fp16 [n_tokens][n_kv_heads][head_dim]
 *   cb_k, cb_v  host float32 [2^bits] holding fp16 values, ascending on return
 */
mkv_status mkv_fit_codebooks(const uint16_t *k, const uint16_t *v, int32_t n_tokens,
                             int32_t n_kv_heads, int32_t head_dim, int32_t bits,
                             int32_t outlier_bp, float *cb_k, float *cb_v);

/*
 * Kernel timing.  `enable` is a mask of kernel kinds (bit k = kind k; 0
 * turns timing off).  Every launch of a selected kind that the library makes
 * on behalf of `cache` is bracketed by HIP events on its stream (at most
 * `max_launches` per kind, pre-created here); each event costs a few
 * microseconds of device time, so time a step's rate with the fewest kinds
 * selected.  mkv_profile_read waits for them and returns, for kind `kind`,
 * the launch count and the summed device time in milliseconds.  Kinds:
 * 0 attention partial (one launch over every sequence's tiles), 1 attention
 * combine, 2 append, 3 top-k select, 4 the append of mkv_decode_step with
 * RocketKV sequences present (it also computes their approximate scores; the
 * step's selection then counts as kind 3).
 */
mkv_status mkv_profile_enable(mkv_cache *cache, int32_t enable, int32_t max_launches);
mkv_status mkv_profile_read(mkv_cache *cache, int32_t kind, int32_t *launches, double *total_ms);

/*
 * KV-cache memory of one sequence under one configuration (the paper's peak KV
 * memory metric, Table 1; Section 2.2 compares the methods by it), in this
 * library's storage format, host only: `resident` = bytes of the cache state
 * holding the tokens the method keeps after prompt_len prompt tokens and
 * n_generated decode steps (codes, fp16 rows, scales, outliers, per-slot
 * positions and scores; capacity reserved for later tokens and the per-step
 * attention workspace excluded); `peak` = the largest such state from prefill
 * to that step, where H2O and RocketKV hold the whole fp16 prompt before their
 * prefill eviction.  KVQ key outliers of decode tokens are counted at their
 * expected rate (outlier_bp), those of the prompt at their bound (the n_o-th
 * order statistic per channel).  shape->n_seqs and max_new_tokens are ignored.
 */
mkv_status mkv_kv_memory(const mkv_shape *shape, const mkv_config *cfg, int32_t prompt_len,
                         int32_t n_generated, size_t *resident, size_t *peak);

/*
 * MetaKV's per-prompt choice among candidate configurations (Section 2.3,
 * Steps 3-7, and the violation score v_c), host only.  Each candidate carries
 * its method, its compression level within the method (0 = least compressed,
 * e.g. KVQuant 4 bits, H2O 60 %, RocketKV 8x), and the predicted end-to-end
 * latency, peak memory and probability of a correct response for the prompt.
 *   1. Budget filter: keep the candidates with latency <= l_max and
 *      memory <= m_max.
 *   2. If FP16 (method MKV_FP16) is kept, choose it.
 *   3. Otherwise keep only the least compressed kept setting of each method;
 *      if one candidate remains choose it, else the highest p_correct.
 *   4. If no candidate passes the filter, choose the smallest
 *      v_c = latency / l_max + memory / m_max, the higher p_correct breaking
 *      a tie; *violated is then 1 (else 0).
 * Remaining ties go to the lower index.  *chosen is an index into cands.
 * MKV_EINVAL for n < 1, a NULL pointer or a non-positive budget.
 */
typedef struct {
  int32_t method;    /* mkv_method */
  int32_t level;     /* compression level within the method, 0 = least compressed */
  double latency;    /* predicted end-to-end latency (the unit of l_max) */
  double memory;     /* predicted peak memory (the unit of m_max) */
  double p_correct;  /* predicted probability of a correct response */
} mkv_candidate;

mkv_status mkv_select_config(const mkv_candidate *cands, int32_t n, double l_max, double m_max,
                             int32_t *chosen, int32_t *violated);

/*
 * Workgroups of the attention partial launch per decode step: `n_tiles` in
 * all, of which `n_tiles_uq` (may be NULL) belong to uniform 4-bit sequences
 * and `n_tiles_rocket` (may be NULL) to RocketKV sequences.
 */
mkv_status mkv_attention_tiles(mkv_cache *cache, int32_t *n_tiles, int32_t *n_tiles_uq,
                               int32_t *n_tiles_rocket);

/*
 * Measurement utility (no part of any method): the read bandwidth a plain
 * streaming kernel reaches on this GPU, for comparison with the attention
 * kernels' achieved bandwidth.  Reads the device buffer `buf` of `bytes`
 * bytes (a positive multiple of 256 KiB) once untimed and then `reps` times
 * between two HIP events on `stream`, waits, and stores the best single-pass
 * rate in GB/s (1e9 bytes/s) in *gbs.  `sink` is a device uint32 [256] that
 * the kernel may write (only to keep its loads from being optimised away).
 * Synchronous; allocates nothing on the device.
 */
mkv_status mkv_probe_read_bandwidth(const void *buf, size_t bytes, uint32_t *sink, int32_t reps,
                                    double *gbs, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* MKV_H */
