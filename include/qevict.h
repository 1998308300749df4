/*
 * qevict.h -- C ABI of the QEvict tiered decode-step library for MI355X (gfx950).
 *
 * QEvict (arXiv 2608.05326) keeps the historical KV cache of every layer as
 * contiguous windows of W tokens.  Outside a protected sink prefix and recent
 * region, each window is Full (bf16), Quantized (asymmetric low-bit codes that
 * attention still reads) or Evicted (Sec. 4.3, cache partition equation).
 * Every decode step attends over the accessible windows and adds each window's
 * attention mass, averaged over the query heads, to its cumulative score
 * (Sec. 4.2, cumulative window score equation).  A routing event ranks the
 * candidates by score and re-tiers them: top K_f -> Full, next K_q ->
 * Quantized, the rest deleted, with promotion from the low-bit ledger and
 * write-once quantization (Sec. 4.3 TopK equations; Algorithm 1).
 *
 * Conventions for every call:
 *  - Tensor arguments are HIP device pointers to contiguous row-major data
 *    unless a comment says "host".  bf16 values are passed as uint16_t bit
 *    patterns.  The caller owns every buffer; the library never allocates or
 *    frees device memory: all state lives in the caller's workspace (the one
 *    exception is the fixed per-device scratch array behind
 *    qevict_prefill_scores_noalloc, part of the library's code object).
 *  - Each buffer must hold the full extent its comment gives, with B, H_q,
 *    H_kv and d taken from the configuration: the kernels read and write
 *    whole extents and cannot check a buffer's size (null pointers and
 *    misalignment are rejected on the host).
 *  - Work is enqueued on the HIP stream given to qevict_cache_init and is
 *    asynchronous unless the comment says "synchronous".  Inputs must stay
 *    valid until the stream has passed the call.
 *  - Host-side validation runs before anything is enqueued; on error nothing
 *    is enqueued and the cache is unchanged.  Errors found on the device
 *    (non-finite score, exhausted slot pool) latch an error word that the next
 *    synchronous call reports; the cache then only accepts destroy.
 *  - qevict_last_error() returns a thread-local message for the last error.
 *  - A handle is not thread-safe; distinct handles are independent.
 *  - Per layer the call order is: prefill_assign, then per step
 *    decode_attend followed by retier at the routing cadence.
 */
#ifndef QEVICT_H_
#define QEVICT_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define QEVICT_ABI_VERSION 4

typedef struct qevict_cache qevict_cache;
typedef int32_t qevict_status;

enum {
  QEVICT_OK = 0,
  QEVICT_ERR_INVALID_ARG = -1,   /* null pointer, index out of range, bad shape        */
  QEVICT_ERR_UNSUPPORTED = -2,   /* shape or option the library does not implement     */
  QEVICT_ERR_WORKSPACE = -3,     /* workspace too small or misaligned                  */
  QEVICT_ERR_BAD_STATE = -4,     /* call out of protocol order, or cache poisoned       */
  QEVICT_ERR_NONFINITE = -5,     /* NaN/Inf in scores or quantizer input               */
  QEVICT_ERR_CAPACITY = -6,      /* a manual move would exceed K_f or K_q              */
  QEVICT_ERR_DEVICE = -7         /* a HIP runtime call failed                          */
};

/* Window tier codes returned by qevict_get_state. */
enum {
  QEVICT_TIER_UNUSED = 0,        /* window not reached yet                             */
  QEVICT_TIER_OPEN = 1,          /* in the recent region, or aged and not yet routed   */
  QEVICT_TIER_FULL = 2,
  QEVICT_TIER_QUANT = 3,
  QEVICT_TIER_EVICTED = 4
};

/* Ledger (persistent low-bit record) states (Algorithm 1). */
enum { QEVICT_LEDGER_NONE = 0, QEVICT_LEDGER_ACTIVE = 1, QEVICT_LEDGER_DORMANT = 2 };

#define QEVICT_BITS_MIXED_4_2 42       /* int4 for new ledgers ranked in the upper half of Q, int2 below */
#define QEVICT_OUT_F32 0
#define QEVICT_OUT_BF16 1
#define QEVICT_FLAG_NO_PROMOTION 0x1u  /* one-way Full -> Quantized -> Evicted policy (App. K)      */
#define QEVICT_FLAG_DEBUG_MASSES 0x2u  /* keep per-head window masses of the last step              */
/* Routing work (re-rank, quantize, promote) of qevict_retier runs on a stream
 * the library owns, so the routing of one layer overlaps the attention of the
 * layers after it.  Requests are launched in batches (up to num_layers / 2,
 * at most 8, layers per batch; one re-rank launch and one migration launch
 * serve all layers of a batch): a batch runs after everything enqueued on the
 * cache's stream before it was launched, which includes each of its layers'
 * latest decode_attend.  That order is kept either on the device (a
 * one-thread kernel on the cache's stream publishes a sequence number in the
 * workspace header and a one-wave kernel on the routing stream waits for it)
 * or by a queue-level wait (hipStreamWaitEvent on the routing stream), which
 * stalls the cache's stream by about 12 us a batch on this hardware.  The
 * cache takes the device-side wait when a migration workgroup fits on a
 * compute unit beside two attention workgroups (registers and LDS of the
 * kernels its configuration launches), so that routing proceeds beside
 * attention, and the queue-level wait otherwise, whose stall then gives the
 * routing work room (qevict_routing_order reports the choice).  A batch whose
 * device-side wait exceeds 10 s is skipped and its layers' next synchronous
 * call returns QEVICT_ERR_BAD_STATE; for the same reason the cache's stream
 * must not be under HIP graph capture while routing is requested.  Every later call that touches a layer
 * (decode_attend, prefill, retier, manual moves, state queries) launches that
 * layer's queued request if needed and orders the cache's stream after its
 * routing; qevict_join_routing does so for every layer. */
#define QEVICT_FLAG_ASYNC_ROUTING 0x4u
/* With QEVICT_FLAG_ASYNC_ROUTING only, at most one of the two: always order
 * routing batches with the queue-level wait, or always with the device-side
 * wait, instead of the choice by kernel footprints. */
#define QEVICT_FLAG_ROUTING_QUEUE_WAIT 0x8u
#define QEVICT_FLAG_ROUTING_DEVICE_WAIT 0x10u

/* Window ranking functions (the hierarchy needs only an order over windows:
 * Sec. 4.2 and the appendix on alternative ranking functions).
 * CUMULATIVE: S(w) += (1/H_q) sum_h (mass of w under head h), every decode step
 *   (Sec. 4.2, cumulative window score equation).
 * DECAY: the exponentially decayed score S_t = lambda S_{t-R} + u_t, u_t the
 *   attention w received since the previous routing event (appendix, decayed
 *   score equation): the library multiplies every live window's score by
 *   lambda in the first decode step after each routing event (and after
 *   prefill), before adding that step's mass. */
#define QEVICT_SCORE_CUMULATIVE 0
#define QEVICT_SCORE_DECAY 1
/* KEY_NORM: the attention-free key-norm score S(w) = -(1/W) sum_{i in w} |k_i|,
 *   |k_i| the L2 norm of token i's key over all KV heads of the layer (appendix,
 *   key-norm equation): prefill computes it for the prompt windows (init_scores
 *   is ignored and may be NULL) and every decode step adds the new token's
 *   share -|k_new| / W to its window; attention masses are not accumulated. */
#define QEVICT_SCORE_KEY_NORM 2
/* PNORM: the attention p-norm S_t = (sum_r u_r^p)^(1/p) over the routing
 *   periods r <= t, u_r the attention w received in period r (appendix,
 *   p-norm equation; the prompt's init_scores are the first period's u).
 *   Scores hold S^p, which orders windows exactly as S does: the sum over
 *   completed periods plus u^p of the period in progress, so that a routing
 *   event at any step ranks by the norm as it stands.  Uses 8 more bytes of
 *   workspace per window (completed-period sum and running u). */
#define QEVICT_SCORE_PNORM 3

/* RoPE-aware Quantized tier (Sec. 4.3: keys are quantized in the pre-RoPE
 * domain and RoPE is reapplied after dequantization).  With rope_base > 0 the
 * keys the caller passes (prompt and decode) are taken as attention consumes
 * them, rotated by half-split RoPE at their absolute positions (channel
 * i < d/2 pairs with i + d/2, angle p * rope_base^(-2i/d)); Full, recent and
 * sink tokens keep them as given.  A window's first quantization un-rotates its
 * keys (float32, each product and sum rounded) and rounds them to bf16: the
 * codes describe pre-RoPE keys.  Attention rotates dequantized keys back to
 * their positions; promotion stores RNE_bf16 of the rotation, taken in float64
 * from the exact z + s c.  cos and sin come from a float32 table of
 * max_context x d/2 pairs in the workspace, filled at init from the C
 * library's double-precision cos / sin. */
typedef struct {
  int32_t abi_version;       /* QEVICT_ABI_VERSION                                          */
  int32_t batch;             /* B sequences, all with the same length                       */
  int32_t num_layers;
  int32_t num_q_heads;       /* H_q                                                          */
  int32_t num_kv_heads;      /* H_kv; H_q % H_kv == 0 and H_q / H_kv <= 16                  */
  int32_t head_dim;          /* d; the library supports 128                                  */
  int32_t window_tokens;     /* W; 8, 32 or 64                                               */
  int32_t group_size;        /* G, the value group: values are quantized per token in groups  */
                             /* of G channels, keys per channel across the window's W tokens;  */
                             /* G == W for W = 32 or 64, G == 32 for W = 8 (no RoPE then)     */
  int32_t quant_bits;        /* 4, 2 or QEVICT_BITS_MIXED_4_2                                */
  int32_t sink_tokens;       /* protected sink prefix |S| (at most 64 windows)               */
  int32_t recent_tokens;     /* protected recent region: a window is routed only once it is  */
                             /* complete and older than this many latest tokens              */
  int32_t max_context;       /* largest sequence length the cache will hold                  */
  int32_t capacity_full;     /* K_f windows                                                  */
  int32_t capacity_quant;    /* K_q windows                                                  */
  int32_t retier_interval;   /* R: decode steps between routing events (sizes the ring)      */
  int32_t out_dtype;         /* QEVICT_OUT_F32 or QEVICT_OUT_BF16                            */
  uint32_t flags;            /* QEVICT_FLAG_*                                                */
  float softmax_scale;       /* 0 selects 1/sqrt(head_dim)                                    */
  int32_t num_splits;        /* split-K factor of the attention pass; 0 = automatic          */
  int32_t score_mode;        /* QEVICT_SCORE_CUMULATIVE (0), _DECAY, _KEY_NORM or _PNORM     */
  float score_decay;         /* lambda of QEVICT_SCORE_DECAY, in (0, 1]                       */
  float score_p;             /* p of QEVICT_SCORE_PNORM, in [1, 16]                           */
  float rope_base;           /* > 0: RoPE-aware Quantized tier (see below); 0: keys as given  */
} qevict_config;

typedef struct {
  int32_t promotions;          /* Quantized -> Full (ledger becomes dormant)   */
  int32_t admissions_full;     /* aged -> Full                                  */
  int32_t first_quantizations; /* ledger created (Full or aged -> Quantized)    */
  int32_t reactivations;       /* Full -> Quantized reusing a dormant ledger    */
  int32_t evictions;           /* any -> Evicted                                 */
  int32_t n_full, n_quant_int4, n_quant_int2;  /* tier sizes after the event */
} qevict_retier_stats;

/* Tier capacities from a byte budget (Sec. 4.3, byte-constrained tier
 * allocation): after the protected sink and recent regions (bf16 keys and
 * values: 4 * H_kv * d bytes per token), a share q of the remaining historical
 * budget B_hist goes to the Quantized tier and 1 - q to the Full tier:
 *   K_f = floor((1 - q) B_hist / M_f),  K_q = floor(q B_hist / M_q).
 * Per-window costs (one layer, one sequence):
 *   M_f = 4 H_kv W d (bf16 keys and values) + 4 (slot index) + 4 (position)
 *   M_q = 2 H_kv W d b / 8 (codes, b = 4 for QEVICT_BITS_MIXED_4_2: the slot
 *         size) + 4 H_kv d (key scale and zero point per channel, fp16)
 *         + 4 H_kv W d / G (value scale and zero point) + 4 + 4 (slot index,
 *         position) + 2 (ledger state and bit width)
 * budget_bytes is per layer and sequence; q is given in thousandths
 * (0 .. 1000) and the arithmetic is exact in integers.  The capacity fields
 * of cfg are ignored; every other field is validated as by
 * qevict_workspace_size.  Fails with QEVICT_ERR_INVALID_ARG when the budget
 * does not cover the protected regions (host only). */
qevict_status qevict_capacities_for_budget(const qevict_config *cfg, int64_t budget_bytes,
                                           int32_t q_permille, int32_t *k_full, int32_t *k_quant);

/* Persistent cache bytes of one (layer, sequence) in the current state, split
 * as the memory accounting appendix lists them (M_sink + M_recent + M_FP + M_Q
 * + M_quant-meta + M_position + M_ledger); the per-window costs are those of
 * qevict_capacities_for_budget, so a state with n_f Full and n_q Quantized
 * windows (no dormant ledger) totals sink + recent + n_f M_f + n_q M_q.
 *   sink        bf16 keys and values of the sink tokens held
 *   recent      bf16 keys and values of the tokens after the routed windows
 *   full        bf16 keys and values of the Full windows
 *   quant_codes packed codes of the Quantized windows (each at its bit width)
 *   quant_meta  their fp16 scales and zero points
 *   position    slot index and position, 8 bytes per Full or Quantized window
 *   ledger      codes and parameters kept by dormant ledger entries (promoted
 *               windows), plus 2 bytes per ledger entry (active or dormant)
 * Workspace beyond these (live lists, split statistics, spare slots) is not
 * counted.  Synchronous, like qevict_get_state. */
typedef struct {
  int64_t sink, recent, full, quant_codes, quant_meta, position, ledger, total;
} qevict_memory;
qevict_status qevict_memory_report(qevict_cache *c, int32_t layer, int32_t seq, qevict_memory *out);

/* Bytes of device workspace a cache with this config needs (host only). */
qevict_status qevict_workspace_size(const qevict_config *cfg, size_t *bytes);

/* Create a cache in the caller's workspace (device pointer, 256-byte aligned,
 * at least qevict_workspace_size bytes; it must outlive the handle).
 * hip_stream is a hipStream_t (NULL = default stream).  Enqueues the state
 * initialisation; *out receives a host handle owned by the library. */
qevict_status qevict_cache_init(const qevict_config *cfg, void *workspace, size_t bytes,
                                void *hip_stream, qevict_cache **out);

/* Release the host handle (the workspace is the caller's). */
qevict_status qevict_cache_destroy(qevict_cache *c);

/* Prefill of one layer (Sec. 4.2: prompt attention initialises the window
 * scores and the first tier assignment).
 *   k, v        [B, H_kv, prompt_len, d] bf16 prompt keys / values
 *   init_scores [B, n_w] fp32, n_w = ceil((prompt_len - sink)/W): initial
 *               cumulative score of every prompt window (also partial ones);
 *               unused (may be NULL) with QEVICT_SCORE_KEY_NORM or when the
 *               prompt has no window (prompt_len <= sink)
 * The complete windows outside the sink and recent regions are routed at once
 * (TopK on init_scores; Quantized windows are quantized from k, v).  The
 * prompt buffers are only read by work enqueued here. */
qevict_status qevict_prefill_assign(qevict_cache *c, int32_t layer, const uint16_t *k,
                                    const uint16_t *v, int32_t prompt_len,
                                    const float *init_scores);

/* Initial window scores from prompt attention (Sec. 4.2: prompt attention
 * initialises the window scores).  The observation queries are those of the
 * last n_obs prompt positions; each attends causally (keys 0 .. its own
 * position, softmax(q k^T * scale), query head h on KV head h / (H_q/H_kv)),
 * and the score of window w (tokens sink + w W .. sink + (w + 1) W - 1, the
 * last one possibly partial) is the attention mass its tokens receive, summed
 * over the observation queries and averaged over the H_q heads.  Sink tokens
 * take part in the softmax and belong to no window.  The result is the
 * init_scores argument of qevict_prefill_assign (any score mode that takes
 * initial scores); the cache's state is neither read nor written.
 *   q_obs   [B, H_q, n_obs, d] bf16, 16-byte aligned
 *   n_obs   1 .. min(prompt_len, 4096)
 *   k       [B, H_kv, prompt_len, d] bf16 prompt keys, 16-byte aligned
 *   scratch device memory of qevict_prefill_scores_scratch_size bytes,
 *           256-byte aligned, owned by the caller, overwritten
 *   scores  [B, n_w] fp32 out, n_w = ceil((prompt_len - sink) / W) (0 when
 *           prompt_len <= sink; scores may then be NULL), 16-byte aligned
 * Work is enqueued on the cache's stream; the buffers must stay valid until
 * it completes.  Reductions run in a fixed order: the result is bitwise
 * repeatable. */
qevict_status qevict_prefill_scores_scratch_size(const qevict_config *cfg, int32_t prompt_len,
                                                 int32_t n_obs, size_t *bytes);
qevict_status qevict_prefill_scores(qevict_cache *c, const uint16_t *q_obs, int32_t n_obs,
                                    const uint16_t *k, int32_t prompt_len, void *scratch,
                                    size_t scratch_bytes, float *scores);

/* The same initial window scores without a caller scratch buffer, for callers
 * that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation).  The three kernels of
 * qevict_prefill_scores run on a fixed scratch array that the library keeps
 * in device memory, one per device, for the life of the process
 * (QEVICT_STATIC_SCRATCH_BYTES = 16 MiB, enough for a batch-1 32K-token prompt
 * with 32 observation queries at 8 KV heads and GQA 4); its address on the
 * device current at qevict_cache_init is looked up then.  This call allocates
 * nothing.  Arguments and results are those of qevict_prefill_scores (bitwise
 * the same scores).  Fails with QEVICT_ERR_WORKSPACE, enqueuing nothing, when
 * the prompt needs more scratch than the array holds
 * (qevict_prefill_scores_scratch_size tells).  Every call on one device shares
 * that device's array, which keeps the last call's contents (every entry a
 * call reads is written by the same call first): calls that overlap on one
 * device, on different streams or from different threads, race. */
#define QEVICT_STATIC_SCRATCH_BYTES (16u << 20)
qevict_status qevict_prefill_scores_noalloc(qevict_cache *c, const uint16_t *q_obs, int32_t n_obs,
                                            const uint16_t *k, int32_t prompt_len, float *scores);

/* One decode step of one layer (Sec. 4.1 decode attention; Sec. 4.2 score).
 *   q      [B, H_q, d]  bf16 queries
 *   k_new, v_new [B, H_kv, d] bf16 key / value of the new token
 *   out    [B, H_q, d]  out_dtype attention output
 * Appends the token to the recent region, attends over sink, recent, Full and
 * Quantized windows (codes dequantized in registers), and adds every live
 * window's head-averaged attention mass to its cumulative score. */
qevict_status qevict_decode_attend(qevict_cache *c, int32_t layer, const uint16_t *q,
                                   const uint16_t *k_new, const uint16_t *v_new, void *out);

/* Routing event of one layer (Sec. 4.3 candidate pool / TopK; Algorithm 1).
 * Candidates are the Full and Quantized windows plus the windows that left
 * the recent region; ranking is by score, ties to the lower window index.
 * Runs the promote / quantize-once / reactivate / evict moves on the device.
 * stats (host, nullable): when given, the call is synchronous and fills the
 * batch totals. */
qevict_status qevict_retier(qevict_cache *c, int32_t layer, qevict_retier_stats *stats);

/* Manual single-window moves (synchronous), with the ledger rules of a routing
 * event (Sec. 4.3, migration-stable quantization and the state-transition
 * equation; Algorithm 1): quantize_window moves a Full window to Quantized,
 * quantizing it once (its first demotion: asymmetric codes, keys per channel
 * across the window's tokens, values per token in groups of G channels, fp16
 * scale and zero point) or reactivating its dormant ledger without
 * requantizing; QEVICT_ERR_CAPACITY if Q already holds K_q windows.
 * promote_window moves a Quantized window to Full: bf16 reconstruction of the
 * low-bit values z + s c (rounded once), the ledger kept dormant;
 * QEVICT_ERR_CAPACITY if F already holds K_f windows, QEVICT_ERR_BAD_STATE
 * under QEVICT_FLAG_NO_PROMOTION.  QEVICT_ERR_BAD_STATE if the window is not
 * in the source tier; QEVICT_ERR_INVALID_ARG for a sequence or window index
 * out of range.  The cache's stream is synchronised. */
qevict_status qevict_quantize_window(qevict_cache *c, int32_t layer, int32_t seq, int32_t window);
qevict_status qevict_promote_window(qevict_cache *c, int32_t layer, int32_t seq, int32_t window);

/* Inspection (synchronous; host output buffers, each of length >= cap,
 * any may be NULL).  *n_windows receives the number of windows reached so far. */
qevict_status qevict_get_state(qevict_cache *c, int32_t layer, int32_t seq, int8_t *tiers,
                               float *scores, int8_t *ledger, int8_t *bits, int32_t cap,
                               int32_t *n_windows);

/* Copy one window out in natural layouts (synchronous; host buffers, NULL to skip).
 *   codes_k, codes_v [H_kv, W, d] uint8 codes of the window's ledger
 *   meta_k  [H_kv, 2, d] fp16 bits: scale then zero point per key group (channel)
 *   meta_v  [H_kv, 2, W, d/G] fp16 bits: scale then zero point per value group
 *   full_k, full_v [H_kv, W, d] bf16 bits of the Full-tier copy
 * Returns QEVICT_ERR_BAD_STATE when a requested part does not exist. */
qevict_status qevict_export_window(qevict_cache *c, int32_t layer, int32_t seq, int32_t window,
                                   uint8_t *codes_k, uint8_t *codes_v, uint16_t *meta_k,
                                   uint16_t *meta_v, uint16_t *full_k, uint16_t *full_v);

/* Test workload support (synchronous): add delta [H_kv, d] (host fp32) to the
 * key zero points of a window's ledger, z <- RNE_fp16(z + delta) with the sum
 * formed in double, which shifts every dequantized key of the window. */
qevict_status qevict_debug_shift_keys(qevict_cache *c, int32_t layer, int32_t seq, int32_t window,
                                      const float *delta);

/* Per-head window masses of the last decode step of a layer (synchronous;
 * needs QEVICT_FLAG_DEBUG_MASSES).  masses: host [B, H_q, n_cap + 1] fp32,
 * the last column is the sink mass; n_cap from qevict_get_state's capacity. */
qevict_status qevict_debug_masses(qevict_cache *c, int32_t layer, float *masses, int32_t n_cap);
/* The same for the cache's full window capacity: masses host [B, H_q, N_w + 1]
 * fp32, N_w = ceil((max_context - sink_tokens) / window_tokens). */
qevict_status qevict_debug_last_masses(qevict_cache *c, int32_t layer, float *masses);

/* Test support for the routing stream's device-side wait (a cache whose
 * qevict_routing_order is QEVICT_ROUTING_GATE, else QEVICT_ERR_INVALID_ARG):
 * launches queued routing, then sets the wait's time
 * limit to timeout_us microseconds (> 0) and, with release = 0, stops the
 * cache's stream from releasing later routing batches, so that each of them
 * times out, leaves its layers unchanged and makes their next synchronous
 * call return QEVICT_ERR_BAD_STATE (such a cache is for destruction only). */
qevict_status qevict_debug_routing_gate(qevict_cache *c, int64_t timeout_us, int32_t release);

/* How the cache orders routing batches after its stream: QEVICT_ROUTING_SYNC
 * (no routing stream), QEVICT_ROUTING_GATE (device-side wait) or
 * QEVICT_ROUTING_QUEUE_WAIT (see QEVICT_FLAG_ASYNC_ROUTING). */
enum { QEVICT_ROUTING_SYNC = 0, QEVICT_ROUTING_GATE = 1, QEVICT_ROUTING_QUEUE_WAIT = 2 };
qevict_status qevict_routing_order(qevict_cache *c, int32_t *order);

/* Kernel timing with HIP events on the cache's stream (off by default).
 * kernel: 0 attention pass, 1 split merge + score accumulation, 2 re-rank,
 * 3 migrations (quantize and promote / admit, one launch), 4 initial window
 * scores (qevict_prefill_scores, its three launches together).  read
 * returns the summed milliseconds and the number of timed launches since
 * enable (for 2 and 3: the number of layer routing events, since with
 * QEVICT_FLAG_ASYNC_ROUTING one launch serves the queued events of up to
 * eight layers), and is synchronous. */
qevict_status qevict_profile_enable(qevict_cache *c, int32_t on);
qevict_status qevict_profile_read(qevict_cache *c, int32_t kernel, double *total_ms, int64_t *count);

/* Algorithmic bytes the last decode_attend of a layer had to read/write in
 * the attention pass (live windows' codes/values, recent and sink tokens,
 * queries, outputs, scores; synchronous). */
qevict_status qevict_last_attend_bytes(qevict_cache *c, int32_t layer, int64_t *bytes);

/* Launch every queued routing request and make the cache's stream wait (on
 * the device, no host synchronisation) for all routing work requested so far.
 * A no-op without QEVICT_FLAG_ASYNC_ROUTING.
 * After it, synchronising the cache's stream also covers every retier call. */
qevict_status qevict_join_routing(qevict_cache *c);

const char *qevict_status_string(qevict_status s);
const char *qevict_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* QEVICT_H_ */
