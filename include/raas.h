/*
 * raas.h -- C ABI of the MI355X (gfx950) decode path of page-based RaaS,
 * Reasoning-Aware Attention Sparsity (Hu et al., arXiv 2502.11147).
 *
 * The library keeps, per (sequence, layer, KV head) -- a "unit" -- a fixed
 * pool of S = budget_tokens / page_size pages in HBM (O(L) memory, Section
 * 4.3). Prefill pages are stored and marked non-evictable (Algorithm 1,
 * Section 3.1). Every decode step (Algorithm 1, Sections 3.2-3.3):
 *   1. stores the new token's K/V in the unit's tail page, opening a fresh
 *      page in the lowest free slot when the tail is full;
 *   2. computes exact softmax attention of the G query heads of the unit
 *      over every resident token (scale 1/sqrt(head_dim));
 *   3. scores every evictable page once against the step's queries with a
 *      representative key: per-channel key min/max of the page, score =
 *      max over the G heads of sum_c max(q_c*kmax_c, q_c*kmin_c), in fp64
 *      (Section 3.3 adopts Quest's representative-key strategy);
 *   4. gives the latest timestamp (the token's absolute position) to the
 *      evictable pages strictly above the (n-k)-th smallest score, where n
 *      is the number of evictable pages and k = floor(r*n) ("top-r", r =
 *      0.5 = above the median, Section 3.2);
 *   5. when the next token has no room (tail page full, no free slot),
 *      evicts the evictable page with the oldest timestamp, ties to the
 *      smallest logical page id (Algorithm 1, eviction in the decode-stage
 *      store).
 *
 * Conventions for every call:
 *  - Tensor arguments are DEVICE pointers owned by the caller, contiguous,
 *    in the pool's dtype (fp32 or bf16) unless stated otherwise. Head-major
 *    layouts: q and out [batch][n_q_heads][head_dim]; k_new, v_new
 *    [batch][n_kv_heads][head_dim]; prefill k, v
 *    [batch][n_kv_heads][prefill_len][head_dim]. Query head h belongs to KV
 *    head h / (n_q_heads / n_kv_heads). Q and K are post-positional-encoding.
 *  - `stream` is a hipStream_t passed as void* (NULL = default stream).
 *    Calls enqueue work on it and return without waiting, except
 *    raas_destroy and raas_export_state, which synchronise it. Inputs must
 *    stay valid until the enqueued work has run.
 *  - A call that returns an error has changed no state; raas_last_error()
 *    gives a message (thread-local). RAAS_E_HIP reports a failed HIP call,
 *    possibly of earlier asynchronous work.
 *  - Inputs must be finite. Calls on one pool are not thread-safe and must
 *    be ordered (one stream, or synchronised between streams): they share
 *    the pool's state and per-step scratch buffers.
 */
#ifndef RAAS_H
#define RAAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RAAS_ABI_VERSION 3

typedef enum {
    RAAS_OK = 0,
    RAAS_E_INVALID = -1, /* bad argument or configuration */
    RAAS_E_BUDGET = -2,  /* prefill does not fit and the policy is RAAS_PREFILL_ERROR */
    RAAS_E_STATE = -3,   /* call out of order: decode before prefill, prefill twice */
    RAAS_E_HIP = -4,     /* a HIP runtime call failed */
    RAAS_E_OOM = -5      /* device allocation failed */
} raas_status;

typedef enum { RAAS_F32 = 0, RAAS_BF16 = 1 } raas_dtype;

/* What to do when the prefill needs more than S-1 pages (Limitations: the
 * budget then goes to prefill tokens and decode tokens are discarded). */
typedef enum {
    RAAS_PREFILL_PIN_HEAD = 0, /* pin the first S-1 prefill pages, drop the rest;
                                  one slot is left for decode pages */
    RAAS_PREFILL_ERROR = 1     /* refuse with RAAS_E_BUDGET */
} raas_prefill_policy;

/* How the G query heads of a unit combine into one page score. The paper
 * does not say (it keeps one decision per page); both are readings. */
typedef enum {
    RAAS_SCORE_MAX = 0,        /* max over the heads of the representative bound (default) */
    RAAS_SCORE_SOFTMAX_SUM = 1 /* sum over the heads of each head's softmax, over the ranked
                                  pages, of the bounds scaled by 1/sqrt(head_dim): scores
                                  then sum to G */
} raas_score_aggregation;

/* What one retention decision covers. The paper does not say; both are
 * readings. */
typedef enum {
    RAAS_SCOPE_KV_HEAD = 0, /* one page table per unit (sequence, layer, KV head) (default) */
    RAAS_SCOPE_SEQUENCE = 1 /* one page table per (sequence, layer), shared by its KV heads:
                               every KV head keeps its own keys and values in the same slots,
                               and a page's score aggregates all n_q_heads (<= 1024) query heads,
                               each against its own KV head's representative key */
} raas_decision_scope;

typedef struct {
    int32_t batch;          /* sequences, >= 1; all advance together */
    int32_t n_layers;       /* >= 1; each layer has its own pool and clock */
    int32_t n_q_heads;      /* multiple of n_kv_heads, group G = n_q_heads/n_kv_heads <= 16 */
    int32_t n_kv_heads;     /* >= 1 */
    int32_t head_dim;       /* 64 or 128 */
    int32_t page_size;      /* tokens per page: 8, 16, 32, 64 or 128 (the paper uses 16) */
    int32_t budget_tokens;  /* L: multiple of page_size, 2 <= L/page_size <= 2048 */
    int32_t dtype;          /* raas_dtype of q, k, v and out */
    double r;               /* fraction of evictable pages refreshed per step, in [0, 1] (0.5);
                               k = floor(r * n) is taken in double precision, so that r = 0.7 at
                               n = 10 refreshes 7 pages (a float 0.7 lies below 0.7) */
    int32_t prefill_policy; /* raas_prefill_policy */
    /* Variants of step 3-4 (0, 0 = the behaviour described above): */
    int32_t score_aggregation; /* raas_score_aggregation */
    int32_t rank_pinned;       /* 1: the pinned prefill pages are scored and ranked with the
                                  evictable ones (n counts them) but never take timestamps;
                                  0: only evictable pages are ranked */
    int32_t decision_scope;    /* raas_decision_scope */
    /* Quest on the prompt, RaaS on the decode tokens (recommended for long
     * prompts or small budgets, Section 4.2 and Limitations): with
     * prompt_tokens > 0 the pool keeps a prompt region of prompt_tokens
     * tokens (a multiple of page_size and of 32) in front of the decode
     * budget; prefill pages go there (a longer prompt: the first pages are
     * kept under RAAS_PREFILL_PIN_HEAD, RAAS_E_BUDGET under
     * RAAS_PREFILL_ERROR), budget_tokens then counts decode tokens only, and
     * each step attends to the prompt_topk (>= 1) prompt pages of largest
     * representative bound (max over the group's heads; ties to the lower
     * page), every decode page and the new token. Not with rank_pinned.
     * 0, 0 = off. */
    int32_t prompt_tokens;
    int32_t prompt_topk;
    /* 1: bitwise-reproducible outputs. The attention of a unit is spread
     * over the wavefronts of a workgroup; by default they claim its blocks
     * as they become free, so which wavefront sums which blocks, and with it
     * the rounding of the output, can change from run to run (retention
     * never does). With 1 each wavefront takes a fixed interleave of the
     * blocks: identical inputs give identical outputs, at about 2% of the
     * step time. 0: the dynamic claims. */
    int32_t deterministic;
} raas_config;

typedef struct raas_pool raas_pool; /* opaque */

/* Validates cfg, allocates the pool for every layer in device memory
 * (hipMalloc) and clears it on `stream`. *out receives the pool; the caller
 * releases it with raas_destroy. Errors: RAAS_E_INVALID, RAAS_E_OOM,
 * RAAS_E_HIP. */
raas_status raas_create_pool(const raas_config* cfg, void* stream, raas_pool** out);

/* The prefill stage of Algorithm 1's cache store, for one layer: stores
 * the prefill_len (>= 0) tokens of every unit in pages 0, 1, ... and marks
 * them non-evictable; sets the clock to prefill_len. A partial last page is
 * not topped up by decode tokens. k, v: [batch][n_kv_heads][prefill_len]
 * [head_dim] (NULL allowed when prefill_len == 0). Must come exactly once
 * per layer, before its first decode step (else RAAS_E_STATE). Errors:
 * RAAS_E_INVALID, RAAS_E_STATE, RAAS_E_BUDGET, RAAS_E_HIP. */
raas_status raas_prefill(raas_pool* pool, int32_t layer, const void* k, const void* v,
                         int32_t prefill_len, void* stream);

/* Ragged prefill of one layer: sequence b stores its first prefill_lens[b]
 * tokens, as raas_prefill does for all (per-sequence clocks, pinned pages
 * and budget rule). k, v: [batch][n_kv_heads][max_len][head_dim], rows past
 * a sequence's length ignored (NULL allowed when no selected sequence keeps
 * a token). prefill_lens: HOST int32 [batch], each in [0, max_len].
 * seq_mask: optional HOST int32 [batch]; only sequences with a nonzero entry
 * are (re)initialised, the others keep their state (NULL = all). Unlike
 * raas_prefill it may be called again at any time: a selected sequence
 * starts over with the new prompt (its pages freed, its clock reset), which
 * is how a finished request's place in the batch is reused. The first
 * prefill of a layer must cover every sequence (else RAAS_E_STATE). The
 * lengths reach the device through a pinned buffer of the pool; a call first
 * waits for the previous ragged prefill's copy out of it. Errors:
 * RAAS_E_INVALID, RAAS_E_STATE, RAAS_E_BUDGET (policy RAAS_PREFILL_ERROR and
 * a selected prompt over S-1 pages), RAAS_E_HIP. */
raas_status raas_prefill_ragged(raas_pool* pool, int32_t layer, const void* k, const void* v,
                                const int32_t* prefill_lens, const int32_t* seq_mask, int32_t max_len,
                                void* stream);

/* One decode step of one layer for every unit (steps 1-5 above). q
 * [batch][n_q_heads][head_dim]; k_new, v_new [batch][n_kv_heads][head_dim];
 * out [batch][n_q_heads][head_dim] receives the attention output, rounded
 * to the pool dtype (nearest-even). Optional outputs (NULL = not written),
 * per unit u = seq * n_kv_heads + kv_head and slot s, after the step:
 *   page_table_out [u][S]: logical page id held by the slot (prefill pages
 *                          0.. in prefill order, then decode pages), or -1;
 *   timestamps_out [u][S]: timestamp of an evictable page, -1 otherwise;
 *   evicted_out    [u]   : logical page id evicted by this step, or -1.
 * Errors: RAAS_E_INVALID, RAAS_E_STATE (layer not prefilled), RAAS_E_HIP. */
raas_status raas_decode_step(raas_pool* pool, int32_t layer, const void* q, const void* k_new,
                             const void* v_new, void* out, int32_t* page_table_out,
                             int32_t* timestamps_out, int32_t* evicted_out, void* stream);

/* raas_decode_step for the sequences whose entry of `active` (DEVICE int32
 * [batch], read when the step runs) is nonzero: the others take no token
 * this step; their state, clock, outputs (out, page_table_out,
 * timestamps_out, evicted_out rows) are left untouched. active = NULL is
 * raas_decode_step. Sequences thereby advance at their own pace (ragged
 * batches). Errors as raas_decode_step. */
raas_status raas_decode_step_masked(raas_pool* pool, int32_t layer, const void* q, const void* k_new,
                                    const void* v_new, void* out, int32_t* page_table_out,
                                    int32_t* timestamps_out, int32_t* evicted_out, const int32_t* active,
                                    void* stream);

/* raas_decode_step for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops or harnesses that forbid
 * hipMalloc): the same kernels and results, but the step's scratch memory
 * -- the partial attention of split units, the page scores handed to the
 * epilogue kernel, and the prompt selection's fills and block lists -- lies
 * in a fixed array of RAAS_STATIC_SCRATCH_BYTES in the library's device
 * code instead of the pool's own buffers. The call allocates nothing and
 * records no profiling events. Steps whose plan needs no scratch (one
 * workgroup per unit without a separate prompt selection, the default for
 * bf16 pools of up to 48 blocks per unit or batches that fill the GPU)
 * never touch the array. A step needing more than the array holds is
 * refused with RAAS_E_INVALID, before anything is enqueued. Each GPU holds
 * one copy of the array until the process ends, shared by every call on it:
 * its contents are the last call's (no step relies on it starting at zero),
 * and calls that overlap on one GPU (other streams, other threads) race on
 * it, so they must be ordered. Errors as raas_decode_step. */
#define RAAS_STATIC_SCRATCH_BYTES (16u << 20)
raas_status raas_decode_step_static(raas_pool* pool, int32_t layer, const void* q, const void* k_new,
                                    const void* v_new, void* out, int32_t* page_table_out,
                                    int32_t* timestamps_out, int32_t* evicted_out, void* stream);

/* Synchronises the pool's last stream, frees all device memory and the
 * pool. NULL is ignored. */
void raas_destroy(raas_pool* pool);

/* Message of the last error on this thread ("" if none). */
const char* raas_last_error(void);

/* RAAS_ABI_VERSION of the library. */
int32_t raas_abi_version(void);

/* Device bytes the pool holds; fixed from creation on. */
size_t raas_pool_bytes(const raas_pool* pool);

/* Copies one layer's retention state to host memory (synchronises
 * `stream`). host_buf holds n_ints int32 = units * (4*S + 4), in order:
 * lid [units][S], ts [units][S], state [units][S] (0 free, 1 pinned,
 * 2 evictable), fill [units][S], then per unit {tail slot or -1,
 * next logical page id, clock, last evicted id or -1}. Errors:
 * RAAS_E_INVALID (wrong n_ints), RAAS_E_HIP. */
raas_status raas_export_state(raas_pool* pool, int32_t layer, int32_t* host_buf, size_t n_ints,
                              void* stream);

/* Checkpoint and resume of one layer: its whole state (keys, values,
 * representative keys, slot and unit records, the clock, and the host-side
 * step bookkeeping) to or from a host buffer of raas_layer_checkpoint_bytes
 * bytes. A pool of the same configuration that loads the buffer continues
 * exactly as the saved one would have: the same retention decisions, and
 * with `deterministic` set the same outputs bit for bit. raas_save_layer
 * synchronises `stream`; raas_load_layer returns once the copies are
 * enqueued (the buffer must stay valid until they have run) and replaces
 * the layer's state, prefilled or not. The buffer starts with a header
 * (magic, ABI version, the configuration) that raas_load_layer checks.
 * Errors: RAAS_E_INVALID (NULL, wrong size, a header that does not match
 * this pool or holds out-of-range step bookkeeping; nothing is copied
 * then), RAAS_E_HIP. */
size_t raas_layer_checkpoint_bytes(const raas_pool* pool);
raas_status raas_save_layer(raas_pool* pool, int32_t layer, void* host_buf, size_t bytes, void* stream);
raas_status raas_load_layer(raas_pool* pool, int32_t layer, const void* host_buf, size_t bytes, void* stream);

/* Tuning: number of slices each unit's pages are split into for the
 * attention step (split-K). 0 restores the automatic choice. Results do not
 * depend on it beyond floating-point rounding. Errors: RAAS_E_INVALID. */
raas_status raas_set_attention_splits(raas_pool* pool, int32_t splits);

/* Kernel timing with HIP events recorded on the call's stream around each
 * enabled kernel of raas_decode_step. mask bit i enables kernel i:
 * 0 the step kernel (attention, append, page scores, and the epilogue when a
 * single workgroup covers a unit), 1 the epilogue kernel (split merge,
 * refresh, eviction; launched when a unit is split over several
 * workgroups, for fp32 pools and for the sequence scope), 2 the prompt
 * selection kernel (with a prompt region, when the step kernel does not
 * select the prompt pages itself: split plans, the softmax aggregation and
 * fp32 pools). mask 0 turns timing off.
 * raas_profile_read returns, for kernel i, the summed duration in ms and the
 * number of timed launches since the last read (synchronising on the
 * recorded events), then resets them. Errors: RAAS_E_INVALID, RAAS_E_HIP. */
raas_status raas_profile(raas_pool* pool, int32_t mask);
raas_status raas_profile_read(raas_pool* pool, int32_t kernel, double* total_ms, int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* RAAS_H */
