/*
 * wici.h — C ABI of the offloaded decoder forward on one MI355X (gfx950).
 *
 * The paper moves an LLM application's GPU work to a remote GPU at the driver
 * boundary: model tensors are uploaded tensor by tensor (Sec. "Model Caching"),
 * and each generated token then runs one fixed group of GPU calls whose inputs
 * follow from the token index (Sec. "Batching and Trace Replay", trace replay).
 * Time to first token and the token rate are what the user sees (Sec.
 * "Evaluation").  This header exposes exactly that work as four calls —
 * wici_load_weights, wici_prefill, wici_decode_step, wici_reset_kv — plus the
 * plumbing to create a model, size and bind its device memory, and read errors.
 *
 * What is computed: a dense pre-norm decoder-only transformer (RMSNorm, Q/K/V/O
 * projections, rotate-half RoPE, causal grouped-query attention over a paged KV
 * cache, SwiGLU MLP, final RMSNorm, LM head) and greedy argmax (lowest index
 * among exactly equal maxima).
 *
 * Conventions for every call:
 *  - Return codes only; nothing throws or aborts across this boundary.
 *  - Arguments and state are checked before any GPU work is issued; a call that
 *    fails a check changes nothing.
 *  - A HIP runtime error returns WICI_E_HIP and puts the model in a sticky
 *    failed state in which every call except wici_destroy / wici_last_error
 *    returns WICI_E_STATE.
 *  - A model is not thread-safe; use one model per thread (one client per
 *    server thread, as in the paper's context management, Sec. "WiCi Library").
 *  - Device memory is owned by the caller (see wici_bind_memory); the library
 *    owns only host state, captured decode graphs (the per-token step, and the
 *    batched step per batch size it led) and a 16-byte pinned, device-mapped
 *    host buffer into which each step's last kernel writes the step state (read
 *    by the host after the stream drains), all released by wici_destroy.
 */
#ifndef WICI_H
#define WICI_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct wici_model wici_model; /* opaque host-side model state */

typedef enum {
  WICI_OK = 0,
  WICI_E_ARG = -1,      /* bad argument: pointer, size, token id, tensor name/shape/dtype */
  WICI_E_STATE = -2,    /* call not allowed in the current state (or model failed) */
  WICI_E_CAPACITY = -3, /* position + new tokens would exceed max_seq */
  WICI_E_HIP = -4,      /* HIP runtime error; model is now failed */
  WICI_E_NUMERIC = -5   /* a logit was NaN or infinite; no token is returned */
} wici_status;

/* Element types.  WICI_Q8 is a weight storage format only (wici_config's
 * weight_dtype): block-scaled 8-bit codes, see wici_quantize_q8; its weight
 * tensors are given as WICI_BF16 or WICI_F32 and quantised at load. */
typedef enum { WICI_F32 = 0, WICI_BF16 = 1, WICI_Q8 = 2 } wici_dtype;

/* Arithmetic of the prefill projections (decode always multiplies bf16/fp32
 * weights by fp32 activations with fp32 accumulation). */
typedef enum {
  WICI_PREFILL_BF16X2 = 0, /* matrix cores, bf16; each fp32 activation stored as two
                              bf16 terms (two products per tile), ~2^-16 relative */
  WICI_PREFILL_BF16 = 1,   /* matrix cores, bf16; activations rounded to bf16 once */
  WICI_PREFILL_F32 = 2,    /* vector fp32 (required for fp32 weights) */
  WICI_PREFILL_BF16X3 = 3, /* matrix cores, bf16; three bf16 terms per activation
                              (three products per tile), fp32-accurate */
  WICI_PREFILL_BF16X3Q = 4 /* matrix cores, bf16; three bf16 terms stored, the Q/K/V
                              projection and the attention read all three and the
                              O, gate/up and down projections the first two (the
                              cached keys and values carry the prompt's precision
                              into every decode step; the other products' ~2^-16
                              leaves the workloads' greedy ids unchanged, measured) */
} wici_prefill_mode;

enum {
  WICI_FLAG_NO_GRAPH = 1,   /* run decode steps eagerly instead of replaying a graph */
  WICI_FLAG_FAULT_DRILL = 2 /* for tests of the error path: every in-launch merge (the decode
                               attention's, the batched products' split-K sums) reports its
                               splits as run on different XCDs, so decode steps fail with
                               WICI_E_HIP as they would on a real misplacement */
};

typedef struct {
  int32_t n_layers;
  int32_t d_model;        /* multiple of 64 */
  int32_t n_heads;        /* query heads, a multiple of n_kv_heads, n_heads/n_kv_heads <= 8 */
  int32_t n_kv_heads;
  int32_t head_dim;       /* 64 or 128 */
  int32_t ffn_dim;        /* multiple of 64 */
  int32_t vocab;          /* >= 1 */
  float rms_eps;          /* > 0 */
  double rope_base;       /* > 1 */
  int32_t tied_embeddings;/* 1: the LM head is the embedding matrix */
  int32_t weight_dtype;   /* wici_dtype of every matrix (norm gains are always F32) */
  int32_t kv_dtype;       /* wici_dtype of the KV cache storage */
  int32_t max_seq;        /* capacity in positions (prompt + generated); 1..16384 */
  int32_t prefill_chunk;  /* prompt rows processed per pass; 1..8192 */
  int32_t kv_page;        /* positions per KV page: 16, 32, 64 or 128 */
  int32_t prefill_mode;   /* wici_prefill_mode; F32 is required when weight_dtype is F32 */
  int32_t flags;          /* WICI_FLAG_* */
  int32_t prefill_planes; /* 0: every prefill product reads the activation terms
                             prefill_mode says.  Else (WICI_PREFILL_BF16X3 only)
                             the number of the three bf16 terms each product reads,
                             two bits each (1..3): bits 0-1 the Q/K/V projection,
                             2-3 the O projection, 4-5 gate/up, 6-7 down, and bits
                             8-9 the terms of the attention's query and
                             probabilities (0: three); a product reading fewer
                             terms does less matrix work and carries its
                             activations to ~2^-16 (two) or ~2^-8 (one) */
} wici_config;

/* One named weight tensor in logical [out, in] row-major layout.  Names:
 *   tok_embeddings [vocab, d_model]
 *   layers.<l>.attn_norm [d_model]           (F32)
 *   layers.<l>.wq [n_heads*head_dim, d_model]
 *   layers.<l>.wk, layers.<l>.wv [n_kv_heads*head_dim, d_model]
 *   layers.<l>.wo [d_model, n_heads*head_dim]
 *   layers.<l>.ffn_norm [d_model]            (F32)
 *   layers.<l>.w_gate, layers.<l>.w_up [ffn_dim, d_model]
 *   layers.<l>.w_down [d_model, ffn_dim]
 *   norm [d_model]                           (F32)
 *   lm_head [vocab, d_model]                 (absent when tied_embeddings)
 * bf16 data is given as raw bf16 bit patterns (uint16). */
typedef struct {
  const char* name;
  int32_t dtype;      /* wici_dtype */
  int32_t ndim;       /* 1 or 2 */
  int64_t shape[2];
  const void* data;   /* host or device pointer (see on_device); borrowed for the call */
  int32_t on_device;  /* 1: data is device memory on the model's GPU */
} wici_tensor;

/* Validate cfg and create host state.  hip_stream (hipStream_t, may be NULL for
 * the null stream) is where every kernel of this model is launched; decode-step
 * graph replay needs a non-NULL stream and is disabled on the null stream.
 * Performs no GPU call.  Errors: WICI_E_ARG for a NULL pointer or an invalid or
 * unsupported configuration. */
wici_status wici_create(const wici_config* cfg, void* hip_stream, wici_model** out);

/* Bytes of device memory the caller must provide for cfg (each region must be
 * 256-byte aligned): packed weights, the paged KV cache, and scratch
 * (activations, logits, reduction partials, device-side position and token).
 * Performs no GPU call.  Errors: WICI_E_ARG. */
wici_status wici_memory_requirements(const wici_config* cfg, size_t* weight_bytes,
                                     size_t* kv_bytes, size_t* scratch_bytes);

/* Bind caller-owned device memory (non-owning; it must outlive the model).
 * Sizes must be at least those of wici_memory_requirements.  Allowed once, in
 * the created state.  Also resets the KV cache state (position 0). */
wici_status wici_bind_memory(wici_model* m, void* d_weights, size_t weight_bytes,
                             void* d_kv, size_t kv_bytes, void* d_scratch,
                             size_t scratch_bytes);

/* Upload weight tensors (any subset, any order, any number of calls; a tensor
 * given again overwrites the earlier copy).  The library repacks them into its
 * fused device layout.  The model becomes ready once every required tensor has
 * been given.  Synchronous.  Errors: WICI_E_ARG for an unknown, duplicate (within
 * one call), mis-shaped or mis-typed tensor (nothing of that call is uploaded),
 * WICI_E_STATE before wici_bind_memory. */
wici_status wici_load_weights(wici_model* m, const wici_tensor* tensors, int32_t n_tensors);

/* Append n_tokens prompt ids (host array) at the current position, processing
 * them in chunks of prefill_chunk rows, and return the greedy next token (and,
 * if logits is not NULL, the fp32 logits [vocab] of the last position into host
 * memory).  Synchronous: the result is final when the call returns (without
 * logits the call returns as soon as the step's final kernel has published it to
 * host memory, which may be before the model's stream has retired that kernel;
 * any later work on the stream is ordered after it).  Errors: WICI_E_ARG (NULL tokens/first_token,
 * n_tokens < 1, an id outside [0, vocab)), WICI_E_STATE (weights incomplete),
 * WICI_E_CAPACITY (position + n_tokens > max_seq), WICI_E_NUMERIC (the
 * positions were still appended; no token is returned, so a following decode
 * step needs an explicit token_in). */
wici_status wici_prefill(wici_model* m, const int32_t* tokens, int32_t n_tokens,
                         int32_t* first_token, float* logits);

/* One greedy decode step: feed token_in (or, when token_in < 0, the token the
 * previous prefill/decode call returned) at the current position and return the
 * next token (and optionally the logits, as for wici_prefill).  Synchronous, as
 * wici_prefill is.
 * Errors: WICI_E_ARG (NULL next_token, token_in >= vocab), WICI_E_STATE (no
 * prefill since the last reset), WICI_E_CAPACITY, WICI_E_NUMERIC, WICI_E_HIP
 * (also when the attention kernel finds that the blocks of one KV head, which
 * exchange their partial results through one XCD's L2 cache, did not all run
 * on the same XCD: the step's results are then not trusted; sticky). */
wici_status wici_decode_step(wici_model* m, int32_t token_in, int32_t* next_token,
                             float* logits);

/* n greedy decode steps without a host round trip per token: the on-GPU form of
 * the paper's function batching, several calls answered in one round trip
 * (Sec. "Batching and Trace Replay"), applied to the per-token call group that
 * the paper replays as a trace.  Each step's argmax stays on the device and is
 * the next step's input; the captured step graph is replayed n times back to
 * back and the host waits once.  token_in as for wici_decode_step (< 0: the
 * last returned token).  tokens_out (host array, n entries) receives the n
 * generated tokens in order; *n_done the number that are valid.  logits (host,
 * [vocab], may be NULL) receives the last step's fp32 logits.  Results are
 * bit-identical to n calls of wici_decode_step.  Synchronous.
 * Errors: WICI_E_ARG (NULL tokens_out/n_done, n < 1, token_in >= vocab),
 * WICI_E_STATE (no prefill since the last reset, or no token to feed),
 * WICI_E_CAPACITY (position + n > max_seq; nothing is run), WICI_E_NUMERIC (a
 * step's logits were not finite: the steps before it are returned in
 * tokens_out[0 .. *n_done), the failed step's position was appended, the rest
 * are -1 and ran as no-ops; the next decode call needs an explicit token_in). */
wici_status wici_decode_n(wici_model* m, int32_t token_in, int32_t n, int32_t* tokens_out,
                          int32_t* n_done, float* logits);

/* Bind a second client to the weights of `src` (the paper's multi-client
 * setting, Sec. "WiCi Library", context management: one model per client, all
 * on the same GPU): m uses src's weight memory read-only (non-owning; src must
 * stay alive and must not reload weights while m is used) and its own KV cache
 * and scratch (sizes from wici_memory_requirements of m's configuration).  The
 * configurations must agree on everything the weight region depends on (shapes,
 * weight dtype, rms_eps, rope_base, tied_embeddings, max_seq).  m becomes ready
 * at once; wici_load_weights on m is refused (WICI_E_STATE).  Allowed once, in
 * the created state; resets the KV state.  Errors: WICI_E_ARG (NULL or identical
 * models, a differing configuration, NULL/small/misaligned regions),
 * WICI_E_STATE (m already bound, src without complete weights). */
wici_status wici_bind_memory_shared(wici_model* m, const wici_model* src, void* d_kv,
                                    size_t kv_bytes, void* d_scratch, size_t scratch_bytes);

/* One greedy decode step for n clients at once: models[0..n) must share one
 * weight copy (wici_bind_memory_shared) and configuration (also kv_dtype and
 * kv_page), be distinct, prefilled and below capacity.  The weights are read
 * once for all n sequences: row b of every activation matrix is sequence b, the
 * projections run as matrix products (on the matrix cores in models[0]'s
 * prefill mode), and each sequence's RoPE, KV append, attention and argmax use
 * its own cache and position.  tokens_in (host, n entries, or NULL for all -1)
 * as token_in of wici_decode_step; next_tokens (host, n) receives each next
 * token; logits (host, n * vocab, may be NULL) each sequence's fp32 logits,
 * row b for sequence b.  Runs on models[0]'s stream and scratch (n <= its prefill_chunk and
 * <= 256); n == 1 runs models[0]'s own decode step (wici_decode_step), whose
 * weight-streaming products are faster for a single row.  Synchronous.  Errors: WICI_E_ARG (bad pointers or counts, models
 * that do not share weights and configuration, duplicates, a token id >= vocab,
 * n beyond the scratch), WICI_E_STATE (a model not ready, not prefilled or
 * without a token to feed), WICI_E_CAPACITY (a model at max_seq),
 * WICI_E_NUMERIC (a sequence's logits were not finite: its next token is -1,
 * the other sequences advanced normally), WICI_E_HIP (a HIP error, or the
 * workgroups of a product split along K, which add their partial sums through
 * one XCD's L2 cache, did not all run on the same XCD: the step's results are
 * then not trusted and models[0] is failed).  Errors are reported on models[0]. */
wici_status wici_decode_batch(wici_model* const* models, int32_t n, const int32_t* tokens_in,
                              int32_t* next_tokens, float* logits);

/* Forget the sequence: position 0, KV pages returned to the pool.  Weights stay. */
wici_status wici_reset_kv(wici_model* m);

/* Current position (number of cached positions).  Host state only. */
wici_status wici_position(const wici_model* m, int32_t* pos);

/* Diagnostic: copy the cached keys and values of one layer for positions
 * [begin, end) into host arrays in logical layout [end-begin, n_kv_heads,
 * head_dim] of the KV storage type (bf16 as uint16 bit patterns).  Synchronous.
 * Errors: WICI_E_ARG for a bad layer or range (end must not exceed the current
 * position), WICI_E_STATE before bind. */
wici_status wici_read_kv(wici_model* m, int32_t layer, int32_t begin, int32_t end,
                         void* host_k, void* host_v);

/* Diagnostic: one decode step exactly as wici_decode_step (same arguments, checks
 * and state effects) but launched eagerly, each launch timed by HIP events that
 * its kernels' dispatches record as the first kernel starts and the last one
 * ends (kernel execution time, without the gaps between launches).  Writes the
 * duration in ms of each launch, in launch order, to durations_ms (capacity
 * entries) and their number (3 + 5 * n_layers) to *n_written.  Order: embedding
 * (0 with bf16 weights, whose first QKV GEMV gathers the embedding row itself);
 * per layer: QKV GEMV (with RoPE and the KV append), attention (with a bf16
 * cache and up to 4 query heads of 128 or 8 of 64 per KV head, one launch that
 * also merges the splits; otherwise split pass start to merge end), O GEMV,
 * gate/up GEMV, down GEMV; then the LM
 * head GEMV and the final argmax.  Errors as wici_decode_step, plus WICI_E_ARG
 * for NULL outputs or a capacity below 3 + 5 * n_layers. */
wici_status wici_profile_decode_step(wici_model* m, int32_t token_in, int32_t* next_token,
                                     float* durations_ms, int32_t capacity, int32_t* n_written);

/* Block-scaled 8-bit quantisation of a row-major matrix [rows, cols] (host
 * memory; cols a multiple of 32), the storage of WICI_Q8 weights.  The paper's
 * models are stored at about 8.5 bits per weight (Sec. "Experiment Setup", Tab.
 * "model_conf"); this format spends exactly that: each row is cut into blocks of
 * 32 weights along cols, and a block keeps one half-precision scale
 *   d = fp16(max_i |w_i| / 127)             (float32 division, ties to even)
 * and 32 codes
 *   q_i = clamp(rint(w_i / d), -127, 127)   (float32 division, ties to even;
 *                                            q_i = 0 when d == 0),
 * so the model computes with w'_i = q_i * d.  Output: codes[rows*cols] holds
 * q_i + 128 as unsigned bytes, scales[rows*(cols/32)] the half-precision bit
 * patterns, both row-major.  src_dtype is WICI_F32 or WICI_BF16 (bit patterns).
 * Host only (no GPU call; multi-threaded for large matrices).  Errors:
 * WICI_E_ARG for NULL pointers, bad sizes or dtype, a non-finite weight or a
 * block scale that overflows half precision (outputs then partly written). */
wici_status wici_quantize_q8(const void* src, int32_t src_dtype, int64_t rows, int64_t cols,
                             uint8_t* codes, uint16_t* scales);

/* MD5 (RFC 1321) of `bytes` bytes of host memory into out16: the name of a
 * tensor in the content store of wici_load_weights_cached.  Host only. */
wici_status wici_md5(const void* data, size_t bytes, uint8_t* out16);

/* What wici_load_weights_cached did with each tensor. */
enum {
  WICI_CACHE_SENT = 0,   /* below the threshold: uploaded from the given data */
  WICI_CACHE_HIT = 1,    /* found in the store: uploaded from the store's file */
  WICI_CACHE_SAVED = 2,  /* not in the store: uploaded from the data, then saved */
  WICI_CACHE_NEEDED = 3  /* not in the store and no data given: not uploaded */
};

/* Weight upload through a content-addressed store, the paper's model caching
 * (Sec. "Model Caching"): a tensor of at least threshold_bytes is named by the
 * MD5 of its bytes (hashes[16*i], or computed from its data when hashes is
 * NULL); if store_dir holds a file of that name (and of the tensor's size) the
 * tensor is loaded from it and its data pointer is not read, else it is uploaded
 * from its data and written to the store (written to a temporary name, then
 * renamed).  A tensor below the threshold is always uploaded from its data.  A
 * caller that has sent only hashes (data NULL) gets WICI_CACHE_NEEDED for the
 * misses and sends those tensors again with data, as in the paper's exchange.
 * outcome[i] receives one WICI_CACHE_* value per tensor.  Uploading follows
 * wici_load_weights (same names, shapes, dtypes, errors).  Errors: WICI_E_ARG
 * (NULL model/store_dir/outcome, a negative threshold, a bad shape, data NULL
 * where it is needed, a tensor given with both a hash and data that misses the
 * store and whose data does not have that hash: it would be saved under the
 * wrong name; checked before anything is uploaded), anything wici_load_weights
 * returns; a store file that cannot be written is not an error. */
wici_status wici_load_weights_cached(wici_model* m, const wici_tensor* tensors,
                                     const uint8_t* hashes, int32_t n_tensors,
                                     const char* store_dir, int64_t threshold_bytes,
                                     int32_t* outcome);

/* Diagnostic, no model: the plain streaming-read rate of device memory, the
 * ceiling a weight-streaming decode step is held to (the paper's per-token work
 * is bound by reading the model's weights, Sec. "Batching and Trace Replay").
 * d_buf: device buffer of `bytes` bytes (a multiple of 16384), read whole `reps`
 * times by `grid` 256-thread workgroups, workgroup b reading the 16 KiB blocks
 * b, b + grid, ... with four non-temporal 16-byte loads per lane in flight.
 * d_sink: device workspace of 256 * grid + 1 32-bit words: word 256 b + t
 * receives the XOR of the words thread t of workgroup b read, word 256 * grid
 * their XOR when a checksum is asked for.  Both buffers stay with the caller.
 * Runs on hip_stream (NULL: the null stream) and waits for it; *ms_per_read
 * receives the average time of one read (events around the reads only).
 * checksum (host, may be NULL) receives the XOR of every 32-bit word of the
 * buffer (each word is read by exactly one thread, so the result does not
 * depend on the grid).  Errors: WICI_E_ARG (NULL pointers, sizes), WICI_E_HIP (a
 * HIP call failed). */
wici_status wici_stream_read(const void* d_buf, size_t bytes, int32_t grid, int32_t reps,
                             void* d_sink, void* hip_stream, float* ms_per_read,
                             uint32_t* checksum);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops that must not allocate, harnesses that forbid it): one read of
 * d_buf exactly as wici_stream_read with grid workgroups, but its workspace is
 * the library's own file-scope device array, so the call allocates nothing
 * (no hipMalloc, hipFree or allocating library routine).  The array holds the
 * partial results of at most 4096 workgroups (4 MiB + 256 bytes per GPU, held
 * until the process ends).  Its device address is looked up once per device on
 * the first call there.  Every call on a GPU shares that GPU's array, so calls
 * that overlap on one GPU race.  Each call writes every partial it reads, so
 * nothing needs clearing.  checksum (host) receives the XOR of every 32-bit word
 * of the buffer; no time is taken.  Synchronous on hip_stream (NULL: the null
 * stream).  Errors: WICI_E_ARG (NULL pointers, bytes not a positive multiple of
 * 16384, grid outside [1, 4096]), WICI_E_HIP (a HIP call failed). */
wici_status wici_stream_read_noalloc(const void* d_buf, size_t bytes, int32_t grid,
                                     void* hip_stream, uint32_t* checksum);

/* Message of the last failed call on this model ("" if none).  Valid until the
 * next call on the model. */
const char* wici_last_error(const wici_model* m);

/* Free host state and the captured graph; NULL is allowed.  Device memory stays
 * with the caller. */
void wici_destroy(wici_model* m);

#ifdef __cplusplus
}
#endif

#endif /* WICI_H */
