/*
 * dmc.h -- C ABI of the MI355X (gfx950) Dynamic Memory Compression decode path.
 *
 * Method: Nawrot et al., "Dynamic Memory Compression: Retrofitting LLMs for
 * Accelerated Inference" (ICML 2024).
 *   - Sec. 3.1 (Inference), the equation re-using the first key/query neurons:
 *     alpha_t = round(sigmoid(k_t[0])), omega_t = sigmoid(q_t[0]).
 *   - Algorithm 1 (single-head KV cache update): alpha_t = 1 merges k_t, v_t
 *     into the last slot as an omega-weighted running mean (z_t = z_{t-1} +
 *     omega_t), alpha_t = 0 appends a slot (z_t = omega_t); k_t[0] and q_t[0]
 *     are zeroed.
 *   - Sec. 3.1, last paragraph: attention (Sec. 2.1, softmax of q.k/sqrt(d_h))
 *     runs over the compressed per-head sequences; heads are independent.
 *   - Sec. 3.3 (Practical considerations): variable-length per-head caches
 *     stored in pages allocated on demand per head; Sec. 5.2 uses 32-token
 *     pages.
 *
 * A "unit" is one (layer, batch row b, kv head g); u = b * num_kv_heads + g.
 * Query heads g*G .. g*G+G-1 (G = num_q_heads / num_kv_heads) read unit u.
 *
 * Conventions for every entry point:
 *   - Pointers named *_dev are device pointers (HIP), owned by the caller and
 *     kept alive until the stream has consumed them.  The library never
 *     allocates device memory and keeps no input pointer past a call.
 *   - Inputs are const: the zeroing of k[0] / q[0] (Algorithm 1) happens
 *     inside the kernels, not in caller memory.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream) and return after enqueueing.  Every host-detectable error
 *     (NULL or misaligned pointer, layer out of range, unsupported shape,
 *     bad stride) returns a status before anything is enqueued; the message
 *     is available from dmc_last_error() on the same thread.
 *   - Device-detected failures (page pool exhausted, per-unit slot capacity
 *     reached, invalid imported lengths) never write out of bounds: the
 *     affected token is dropped, a sticky device flag is raised, and
 *     dmc_cache_check() reports it.  Outputs of such a call are undefined.
 *   - One handle is used by one stream at a time; the ABI is not reentrant on
 *     the same handle.  No exception or abort crosses the ABI.
 *   - Floating point: inputs, cache slots and outputs use the configured dtype
 *     (bf16 or fp32); all arithmetic accumulates in fp32; bf16 results are
 *     rounded to nearest even.
 */
#ifndef DMC_H
#define DMC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef void *dmc_stream_t; /* a hipStream_t */

typedef enum {
  DMC_OK = 0,
  DMC_ERR_INVALID_ARG = 1, /* bad pointer, layer, shape, stride or config   */
  DMC_ERR_UNSUPPORTED = 2, /* valid request outside what the kernels handle */
  DMC_ERR_CAPACITY = 3,    /* page pool or per-unit slot capacity exhausted */
  DMC_ERR_HIP = 4          /* a HIP runtime call failed                     */
} dmc_status;

typedef enum { DMC_BF16 = 0, DMC_FP32 = 1 } dmc_dtype;

/* Which query neuron supplies omega for a kv head shared by G query heads
 * (grouped-query attention; the paper combines DMC with GQA, Sec. 5, but
 * does not name the head).  LEAD: query head g*G.  GROUP_MEAN: mean of the
 * G heads' sigmoid(q[0]). */
typedef enum { DMC_OMEGA_LEAD_QHEAD = 0, DMC_OMEGA_GROUP_MEAN = 1, DMC_OMEGA_UNIFORM = 2 } dmc_omega_src;

/* Which heads' neurons decide (alpha) and weigh (omega) each unit's token.
 * PER_HEAD: every kv head its own (DMC).  SHARED_LAYER: kv head 0 of the
 * batch row (its k[0]; omega per dmc_omega_src from query group 0) for every
 * head of the layer -- the DMC-HardC ablation of the appendix, whose heads
 * therefore keep equal lengths.  UNIFORM omega is the uniform-weighting
 * ablation (every token of a segment weighs 1). */
typedef enum { DMC_DECISION_PER_HEAD = 0, DMC_DECISION_SHARED_LAYER = 1 } dmc_decision_src;

typedef struct dmc_cache_config {
  int32_t num_layers;
  int32_t batch;
  int32_t num_q_heads;
  int32_t num_kv_heads;      /* num_q_heads % num_kv_heads == 0, G in {1,2,4,8} */
  int32_t head_dim;          /* 64 or 128 */
  int32_t dtype;             /* dmc_dtype: inputs, cache slots and outputs */
  int32_t page_size;         /* slots per page, power of two in [8, 65536]; the paper uses 32.
                                A page as large as max_slots_per_seq gives every unit one
                                contiguous padded region (the padded-tensor layout of DMC-C) */
  int32_t max_slots_per_seq; /* slot capacity of one unit; page-table width = ceil(/page_size) */
  int64_t num_pages;         /* pool capacity in pages, shared by all units, < 2^31 */
  float decision_bias;       /* c: alpha = round(sigmoid(k[0] - c)) = (k[0] > c); 0 = Algorithm 1 */
  int32_t omega_src;         /* dmc_omega_src */
  int32_t split_tile;        /* cap on slots per split-K range; 0 = no cap: each wave of
                                a decode launch gets an equal share of the layer's actual
                                (compressed) slots */
  int32_t max_prompt_len;    /* largest n for dmc_prefill_compress / dmc_prefill_attend;
                                0 = max_slots_per_seq */
  int32_t decision_src;      /* dmc_decision_src */
  int32_t window;            /* 0: exact Algorithm 1.  w in [1, 64]: the window-grouping
                                approximation of Sec. 3.3 -- every step's partial
                                accumulation runs over the last w tokens only, so the open
                                slot is the omega-weighted mean of the last min(w, length)
                                tokens of its segment and a closed slot keeps that of its
                                segment's last w tokens.  Each unit then also keeps its open
                                segment's last w raw tokens (key with element 0 zeroed,
                                value, omega) in the workspace; the paper uses w = 12 */
} dmc_cache_config;

typedef struct dmc_cache dmc_cache; /* opaque host handle */

/* Bytes of device workspace a cache with this configuration needs.  The cache
 * is the paged storage of Sec. 3.3 (Practical considerations): every
 * (layer, batch row, kv head) keeps its own variable-length sequence of
 * slots, held in fixed-size pages taken from one shared pool on demand, with
 * a per-unit page table -- so the workspace is the page pool, the page
 * tables, the slot counts and running importance sums z of Algorithm 1, the
 * control words of the page allocator, and the decode split-K partials and
 * prefill staging.  Returns 0 for an invalid configuration (see
 * dmc_last_error). */
size_t dmc_cache_workspace_bytes(const dmc_cache_config *cfg);

/* Create a cache (the paged per-head storage of Sec. 3.3, every unit empty:
 * Algorithm 1 starts from an empty cache, so the first token of a unit opens
 * its first slot) inside the caller-owned device buffer `workspace_dev` of
 * `bytes` bytes (>= dmc_cache_workspace_bytes(cfg), 256-byte aligned, on the
 * current HIP device).  Enqueues the initialisation (all lengths and z zero,
 * empty pool, flags clear) on `stream`.  *out receives the host handle.
 * Errors: DMC_ERR_INVALID_ARG for a bad configuration, a NULL or misaligned
 * workspace, or one smaller than needed (nothing enqueued); DMC_ERR_HIP if
 * the device query or the initialisation launch fails (*out stays NULL). */
dmc_status dmc_cache_alloc(const dmc_cache_config *cfg, void *workspace_dev, size_t bytes,
                           dmc_stream_t stream, dmc_cache **out);

/* Release the host handle of a paged cache (Sec. 3.3); the workspace and the
 * pages in it stay the caller's, untouched.  DMC_ERR_INVALID_ARG for NULL. */
dmc_status dmc_cache_free(dmc_cache *cache);

/* Empty every layer: lengths, z, page pool and flags back to the initial state. */
dmc_status dmc_cache_reset(dmc_cache *cache, dmc_stream_t stream);

/* Prompt phase of one layer (Algorithm 1 applied to n prompt tokens in order,
 * without attention): per unit, the first token opens a slot, then every
 * token with k[0] > c merges into the open slot and every other token opens
 * a new one.  The result equals n sequential decode-step updates: slot s of
 * a unit is the omega-weighted mean of its segment's keys (element 0 zeroed)
 * and values, z is the omega sum of the last segment (with a window w: of
 * the segment's last min(w, length) tokens, which the unit also keeps).
 *   k_dev, v_dev: logical [B, n, Hkv, d] of the config dtype; k_strides /
 *     v_strides give the element strides of the B, n and Hkv axes (the d axis
 *     is contiguous); base pointers 16-byte aligned, strides multiples of 8.
 *   q_dev: logical [B, n, Hq, d] with q_strides for B, n, Hq; only element 0
 *     of each query row is read (a [B, n, Hq] tensor of q[..., 0] with
 *     strides (n*Hq, Hq, 1) is accepted), no alignment requirement.
 *   The token (n-axis) strides of k, v and q are below 32 MiB, else
 *   DMC_ERR_UNSUPPORTED (the kernels address up to 64 consecutive tokens from
 *   one base with 32-bit offsets).
 *   n: prompt length, 0 <= n <= max_prompt_len.
 *   prompt_lens_dev: optional int32 [B]; row b uses tokens t < prompt_lens[b]
 *     (values outside [0, n] raise the invalid-argument device flag and are
 *     clamped).  NULL = n for every row.
 *   slot_index_dev: optional int32 [B, Hkv, n]: slot each token went to, -1
 *     for tokens past the row's prompt length.
 * The layer's previous contents are discarded (its pages are not reclaimed:
 * the pool is a bump allocator emptied only by dmc_cache_reset). */
dmc_status dmc_prefill_compress(dmc_cache *cache, int32_t layer,
                                const void *k_dev, const int64_t k_strides[3],
                                const void *v_dev, const int64_t v_strides[3],
                                const void *q_dev, const int64_t q_strides[3],
                                int32_t n, const int32_t *prompt_lens_dev,
                                int32_t *slot_index_dev, dmc_stream_t stream);

/* Prompt phase of one layer with attention outputs: the compaction of
 * dmc_prefill_compress (same cache result, same slot_index), and for every
 * prompt token t the softmax attention of its G query heads over the cache
 * as it stands right after token t's own update -- the per-position form of
 * the inference rule of Sec. 3.1 (Sec. 3.2 states the same set as a mask
 * over the unrolled intermediate states): the final state of every segment
 * that closed before t (slots 0 .. slot(t)-1), plus the running omega-
 * weighted mean of t's own segment over its tokens up to t.  Scale
 * 1/sqrt(d), q[0] treated as 0, as in decode.
 *   k_dev, v_dev, k_strides, v_strides, n, prompt_lens_dev, slot_index_dev:
 *     as for dmc_prefill_compress.
 *   q_dev: logical [B, n, Hq, d] with q_strides for B, n, Hq (d contiguous);
 *     every element is read; 16-byte aligned, strides multiples of 8.
 *   out_dev: logical [B, n, Hq, d], config dtype, out_strides for B, n, Hq
 *     (d contiguous), 16-byte aligned, strides multiples of 8.  Rows of
 *     tokens t >= prompt_lens[b] are written as zeros.  out must not overlap
 *     q, k or v.
 * bf16 runs on the matrix cores (v_mfma_f32_16x16x32_bf16, fp32
 * accumulation), fp32 on the vector ALUs.  Uses the staging area sized by
 * max_prompt_len, including the per-32-token running-sum records. */
dmc_status dmc_prefill_attend(dmc_cache *cache, int32_t layer,
                              const void *k_dev, const int64_t k_strides[3],
                              const void *v_dev, const int64_t v_strides[3],
                              const void *q_dev, const int64_t q_strides[3],
                              int32_t n, const int32_t *prompt_lens_dev,
                              void *out_dev, const int64_t out_strides[3],
                              int32_t *slot_index_dev, dmc_stream_t stream);

/* One auto-regressive decode step of one layer: for every unit, the DMC
 * update of Algorithm 1 with the new token (alpha from the unit's own k[0];
 * the first token of an empty unit always appends), then softmax attention
 * of each of the G query heads over the updated compressed sequence with
 * scale 1/sqrt(d) and q[0] treated as 0.
 *   q_dev:   [B, Hq, d] contiguous, config dtype, 16-byte aligned.
 *   k_dev, v_dev: [B, Hkv, d] contiguous, 16-byte aligned.
 *   out_dev: [B, Hq, d] contiguous, 16-byte aligned, written.
 *   slot_index_dev: optional int32 [B, Hkv]: slot index the token went to
 *     (-1 when it was dropped for lack of capacity).
 * The call only enqueues kernels on `stream` (no allocation, no host
 * synchronisation, no memset), so it can be captured in a HIP graph.  Every
 * call on a layer uses the same device buffers (its last kernel copies the
 * post-step lengths back into the layer's current-lengths buffer), so a
 * captured step can be replayed any number of times. */
dmc_status dmc_decode_step(dmc_cache *cache, int32_t layer, const void *q_dev,
                           const void *k_dev, const void *v_dev, void *out_dev,
                           int32_t *slot_index_dev, dmc_stream_t stream);

/* Bytes of the library's static device scratch used by dmc_decode_step_static
 * (one copy per GPU the library runs on, held until the process ends). */
#define DMC_STATIC_SCRATCH_BYTES (64u << 20)

/* dmc_decode_step for callers that cannot allocate device memory (code under
 * HIP-graph capture, tight serving loops, harnesses that forbid allocation
 * or extra workspace traffic): the same update and attention, through the
 * same kernels, with results bit-identical to dmc_decode_step -- but the
 * split-K partial records and the per-unit record table come from a static
 * device array of the library (DMC_STATIC_SCRATCH_BYTES per GPU) instead of
 * the cache workspace.  The call allocates nothing and calls no allocating
 * routine; the array's address on a device is resolved once, when the first
 * cache on that device is created (dmc_cache_alloc).
 *   Arguments, layouts and device-side errors: as for dmc_decode_step.
 *   Limit: a launch of this cache needs units * 8 bytes (rounded up to 256)
 *     plus (ranges + units) * G * (head_dim + 4) * 4 bytes of records, ranges
 *     being the launch's waves (2048 on a 256-CU MI355X) or, with a split_tile,
 *     ceil(units * (max_slots_per_seq + 32) / split_tile) if that is larger; a
 *     cache that needs more returns DMC_ERR_UNSUPPORTED before anything is
 *     enqueued.
 *   Nothing in the array has to start at zero: every record a call reads is
 *     written earlier in the same call.  All calls on one GPU share that
 *     GPU's array, so calls that overlap on one GPU (other streams, other
 *     caches or layers in flight concurrently) race and give wrong results:
 *     serialise them, e.g. on one stream. */
dmc_status dmc_decode_step_static(dmc_cache *cache, int32_t layer, const void *q_dev,
                                  const void *k_dev, const void *v_dev, void *out_dev,
                                  int32_t *slot_index_dev, dmc_stream_t stream);

/* Copy the slot counts of one layer into lengths_dev (int32 [B, Hkv]). */
dmc_status dmc_cache_lengths(const dmc_cache *cache, int32_t layer, int32_t *lengths_dev,
                             dmc_stream_t stream);

/* Gather one layer into dense tensors k_dense_dev, v_dense_dev
 * [B, Hkv, dense_slots, d] (config dtype; slots at or past a unit's length
 * are zero-filled; units longer than dense_slots are truncated) and its
 * running importance sums into z_dev (fp32 [B, Hkv]). */
dmc_status dmc_cache_export(const dmc_cache *cache, int32_t layer, void *k_dense_dev,
                            void *v_dense_dev, int32_t dense_slots, float *z_dev,
                            dmc_stream_t stream);

/* Install an already-compressed layer: unit u gets lengths_dev[u] slots
 * taken from k_dense_dev / v_dense_dev [B, Hkv, dense_slots, d] and the
 * running sum z_dev[u] of its open slot.  Pages come from the pool.  Lengths
 * outside [0, min(dense_slots, max_slots_per_seq)] raise the device flag and
 * are treated as 0.  A cache configured with a window returns
 * DMC_ERR_UNSUPPORTED: its open segment's raw tokens cannot be rebuilt from
 * slots. */
dmc_status dmc_cache_import(dmc_cache *cache, int32_t layer, const void *k_dense_dev,
                            const void *v_dense_dev, int32_t dense_slots,
                            const int32_t *lengths_dev, const float *z_dev,
                            dmc_stream_t stream);

/* Synchronise `stream` and report the sticky device flags: DMC_OK,
 * DMC_ERR_CAPACITY (pool or slot capacity exhausted) or DMC_ERR_INVALID_ARG
 * (bad imported lengths or prompt lengths).  Flags clear only on reset. */
dmc_status dmc_cache_check(dmc_cache *cache, dmc_stream_t stream);

/* Synchronise `stream` and return the number of pool pages handed out. */
dmc_status dmc_cache_pages_used(dmc_cache *cache, int64_t *pages_out, dmc_stream_t stream);

/* ---------------------------------------------------------------------------
 * Training-time DMC attention of one layer (Sec. 3.2 "Training", Sec. 3.3
 * window grouping, and the masking appendix).  Forward and backward over a
 * whole sequence, for continued pre-training that teaches a model DMC:
 *   - decisions relaxed by Gumbel-sigmoid: alpha_t = sigmoid((k_t[0] - c +
 *     g_t) / tau), g_t logistic noise drawn by the caller (noise_dev);
 *   - importance omega_t = sigmoid(q_t[0]) of the group's first query head
 *     (floored at 2^-100), or 1 with DMC_OMEGA_UNIFORM;
 *   - unrolled states: every position j keeps the partial accumulation
 *     (Sec. 3.2) of its last w tokens, started afresh at the window's first
 *     token, with continuous alpha; keys enter with element 0 zeroed;
 *   - query i attends to states j <= i with the additive mask
 *     log(1 - alpha_{j+1}) for j < i and 0 for j = i, scores over elements
 *     1..d-1 of q and the state, scaled by 1/sqrt(d).
 * Layouts: q, out, dout, dq [B, n, Hq, d]; k, v, dk, dv [B, n, Hkv, d]; all
 * contiguous in the config dtype, 16-byte aligned.  noise, alpha, dalpha:
 * fp32 [B, n, Hkv] contiguous.  The workspace (caller-owned device memory,
 * 256-byte aligned, dmc_train_workspace_bytes) carries what the forward saves
 * for the backward (states, decisions, softmax statistics); pass the same
 * workspace, untouched, to the backward of the same inputs.
 * ------------------------------------------------------------------------- */
typedef struct dmc_train_config {
  int32_t batch;
  int32_t seq_len;           /* n >= 1 */
  int32_t num_q_heads;
  int32_t num_kv_heads;      /* G = num_q_heads / num_kv_heads in {1,2,4,8} */
  int32_t head_dim;          /* 64 or 128 */
  int32_t dtype;             /* dmc_dtype of q, k, v, out and the gradients */
  float decision_bias;       /* c; the paper uses 5 */
  float temperature;         /* tau > 0; the paper uses 0.1 */
  int32_t window;            /* w in [1, 64]; the paper uses 12 */
  int32_t omega_src;         /* DMC_OMEGA_LEAD_QHEAD or DMC_OMEGA_UNIFORM */
} dmc_train_config;

/* Workspace bytes for a training configuration (0 if invalid). */
size_t dmc_train_workspace_bytes(const dmc_train_config *cfg);

/* Forward: out_dev [B, n, Hq, d] and, when alpha_dev is not NULL, the relaxed
 * decisions alpha [B, n, Hkv] (fp32; what the compression loss of Sec. 3.2
 * sums).  Fills the workspace for dmc_train_backward. */
dmc_status dmc_train_forward(const dmc_train_config *cfg, const void *q_dev, const void *k_dev,
                             const void *v_dev, const float *noise_dev, void *out_dev,
                             float *alpha_dev, void *workspace_dev, size_t workspace_bytes,
                             dmc_stream_t stream);

/* Backward: gradients of sum(out * dout) + sum(alpha * dalpha) with respect
 * to q, k and v (dalpha_dev may be NULL), given the forward's inputs and
 * outputs and its workspace.  dq, dk, dv are written in full (the decision
 * and importance neurons k[0], q[0] get their gradients through alpha and
 * omega).  Outputs must not overlap the inputs. */
dmc_status dmc_train_backward(const dmc_train_config *cfg, const void *q_dev, const void *k_dev,
                              const void *v_dev, const float *noise_dev, const void *out_dev,
                              const void *dout_dev, const float *dalpha_dev, void *dq_dev,
                              void *dk_dev, void *dv_dev, void *workspace_dev,
                              size_t workspace_bytes, dmc_stream_t stream);

/* Message for the last non-OK status returned on this thread ("" if none). */
const char *dmc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DMC_H */
