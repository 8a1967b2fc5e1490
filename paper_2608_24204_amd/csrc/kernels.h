// Host-side launchers of the libwici HIP kernels.  All pointers are device
// pointers; every launcher enqueues on `st` and returns hipGetLastError().
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wici {

enum GemvEpi { GEMV_STORE = 0, GEMV_RESID = 1, GEMV_SWIGLU = 2, GEMV_ARGMAX = 3, GEMV_QKV = 4 };

// Weight storage (the values of the C ABI's wici_dtype).  A W_Q8 matrix [N, K]
// is N*K code bytes (q + 128, row-major) followed, at the next 256-byte
// boundary, by N*K/32 half-precision block scales (row-major, one per 32
// consecutive weights of a row); the weight is (code - 128) * scale.
enum WType { W_F32 = 0, W_BF16 = 1, W_Q8 = 2 };
__host__ __device__ inline size_t q8_scale_offset(size_t n, size_t k) {
  return (n * k + 255) / 256 * 256;
}
__host__ __device__ inline size_t weight_bytes(int wt, size_t n, size_t k) {
  if (wt == W_Q8) return q8_scale_offset(n, k) + n * (k / 32) * 2;
  return n * k * (wt == W_BF16 ? 2 : 4);
}

struct ArgmaxPart { float v; int32_t i; };

// Timing of the decode launchers (used by the profiling entry point): while set
// on the calling thread, a launcher's first kernel records `start` when it begins
// and its last kernel records `stop` when it ends.
struct LaunchTimer { hipEvent_t start; hipEvent_t stop; };
void set_launch_timer(const LaunchTimer* t);
const LaunchTimer* launch_timer();

struct KvLayout {
  void* base;            // this layer's pool
  const int32_t* table;  // logical page -> physical page
  int page;              // positions per page
  int n_kv;              // KV heads
  int hd;                // head dim
  int max_pos;           // capacity (positions); the table covers ceil(max_pos / page) pages
  // element offset of (phys page, kv 0/1, head h, slot s, dim d):
  //   ((phys * 2 + kv) * n_kv + h) * page * hd + s * hd + d
};

// The merge of a batch-1 decode attention done by the last split block of each
// KV head (one launch, no merge kernel), for bf16 caches of up to 32 splits.
// cnt and xcc each hold 64 ints per KV head (attn_fuse_ints(n_kv) ints in all,
// cnt first); the counters must be zero before the first launch and are zero
// again after every launch.  state is the step's DecodeState: its `fault` field
// is set if the splits of one head did not all run on one XCD (their partials
// then cannot be trusted).  The launcher fills in the other fields.
struct AttnFuse {
  int* cnt;
  int* xcc;
  void* state;
  float* out;
  int nsplit, n_heads, n_kv;
  int drill;  // nonzero: report the splits as misplaced (tests of the error path)
};
int attn_fuse_ints(int n_kv);

// The decode QKV projection's epilogue (GEMV_QKV): RoPE at the current position
// and the KV-cache append.  W is [(n_q + 2 n_kv) * hd, K] (query heads, then key
// heads, then value heads); the GEMV walks it in RoPE pairs (rows j and j + hd/2
// of a head), so each finished pair is rotated in registers:
//   query heads: y[h*hd + j], y[h*hd + j + hd/2] = rotated values * q_scale;
//   key heads:   rotated values, rounded to the cache type, stored at the position;
//   value heads: values rounded to the cache type, stored at the position.
struct QkvRope {
  const float* cos_t;  // [max_pos][hd/2]
  const float* sin_t;
  const void* state;   // DecodeState: the position being appended
  KvLayout kv;         // this layer's cache (kv.hd = head dim, kv.n_kv = KV heads)
  int kv_bf16;         // cache element type: 1 bf16, 0 fp32
  int n_q;             // query heads
  float q_scale;       // 1/sqrt(hd)
  // bf16 embedding [V, K] or nullptr.  Set: the projection's input is the
  // embedding row of the state's token (a negative token gives a zero row)
  // instead of x, and that row is also stored into x (the residual stream), so
  // no separate gather runs before the first layer.
  const void* embed;
};

// y = W x for W [N, K] row-major (bf16 bits or fp32), x fp32 [K].
// norm_gain != nullptr: x is first RMS-normalised (eps) and scaled by the gain.
// RESID: y[n] += acc (norm_gain must be nullptr).  The others take a
// normalised x (norm_gain required): SWIGLU: rows (2i, 2i+1) hold (gate_i,
// up_i) and y[i] = silu(gate_i) * up_i.  ARGMAX: y[n] = acc and one ArgmaxPart
// per workgroup into `part` (at most 1024; the count is returned through
// *nblocks).  QKV: as described for QkvRope (`rope` required,
// N = (n_q + 2 n_kv) * hd).  (STORE is a GEMM epilogue only.)
hipError_t launch_gemv(int wt, int epi, const void* W, int N, int K, const float* x,
                       const float* norm_gain, float eps, float* y, ArgmaxPart* part,
                       int* nblocks, hipStream_t st, const QkvRope* rope = nullptr);

// Final argmax over `n` partials -> st->token; st->pos += advance (or = set_pos
// when set_pos >= 0); st->bad set when a partial carries index -1 (a logit was
// not finite), in which case st->token = -1.  The chosen token is also stored
// at hist[new pos - 1] (the token that follows that position).  A decode step
// (advance > 0) that finds st->bad already set changes nothing: once a step of
// a device-resident run has failed, the steps queued after it are no-ops.  With
// host_mirror != nullptr (pinned host memory holding a DecodeState) the new
// state is also written there, for the host to read after synchronising.
hipError_t launch_argmax_final(const ArgmaxPart* part, int n, void* state, int32_t* hist,
                               int advance, int set_pos, void* host_mirror, hipStream_t st);

// x[t, :] = E[tokens[t], :] for t < T (tokens == nullptr: the state's token, T = 1;
// a negative state token, left by a failed step, gives a zero row).
hipError_t launch_embed(int wt, const void* E, int V, int d, const int32_t* tokens, int T,
                        const void* state, float* x, hipStream_t st);
// st->token = token and clear st->bad (a host-given token restarts decoding).
hipError_t launch_set_token(void* state, int token, hipStream_t st);
hipError_t launch_reset_state(void* state, hipStream_t st);
hipError_t launch_init_block_table(int32_t* table, int n_pages, hipStream_t st);
// One plain streaming read of `bytes` (a multiple of 16 KiB) of device memory by
// `grid` workgroups; sink[256 b + t] receives the XOR of the 32-bit words thread t
// of workgroup b read (every word of the buffer is read by exactly one thread).
hipError_t launch_stream_read(const void* buf, size_t bytes, int grid, unsigned* sink,
                              hipStream_t st);
// out[0] = XOR of in[0 .. n) (one workgroup).
hipError_t launch_xor_reduce(const unsigned* in, int n, unsigned* out, hipStream_t st);
// p[i] = v for i < n (a fill kernel, so it can sit in captured work).
hipError_t launch_fill_i32(int32_t* p, int n, int v, hipStream_t st);

// y[t, :] = RMSNorm(x[t, :]) * gain for T rows of width d (row stride d).
hipError_t launch_rmsnorm_rows(const float* x, const float* gain, float eps, int T, int d,
                               const ActBuf& y, hipStream_t st);


// One sequence of a batched decode step (a device array of B of them).
struct SeqDesc {
  void* kv;                  // the sequence's KV pool (layer 0; layer l at + l * kv_layer_stride)
  size_t kv_layer_stride;    // bytes per layer
  const int32_t* table;      // its page table
  void* state;               // its DecodeState
  int32_t* hist;             // its token history [max_seq]
};

// Batched decode helpers (row b = sequence b).
hipError_t launch_gather_tokens(const SeqDesc* seqs, int B, int32_t* tokens, hipStream_t st);
// Rotate row b's queries in place (times q_scale) and keys at sequence b's position,
// append keys and values to its cache (layer `layer`; kv gives page, heads, hd).
hipError_t launch_rope_append_batch(bool kv_bf16, float* qkv, int B, int Hq, const float* cos_t,
                                    const float* sin_t, const SeqDesc* seqs, int layer,
                                    KvLayout kv, float q_scale, hipStream_t st);
// Greedy token per row of logits [B, V]; advances each sequence's state and history
// (a row with a non-finite logit gets token -1 and the failed flag).
hipError_t launch_argmax_rows(const float* logits, int B, int V, const SeqDesc* seqs,
                              hipStream_t st);
// RoPE tables and the query scale, for a decode attention that applies RoPE and
// appends the new key and value itself.
struct RopeIn {
  const float* cos;  // [max_seq][hd / 2]
  const float* sin;
  float q_scale;
};
// Batched decode attention: row b's queries (q + b * q_stride, rotated and scaled)
// over sequence b's cache [0, pos_b]; partials [B][Hq][nsplit]; out is the
// activation buffer of the O projection, row b at b * Hq * hd.  With rope (bf16
// caches only) row b is instead the raw projection row (query, key, value
// heads): the launch rotates and scales the queries and rotates and appends the
// position's key and value itself, in place of launch_rope_append_batch.
hipError_t launch_attn_decode_batch(bool kv_bf16, const float* q, int q_stride, int B, int Hq,
                                    KvLayout kv, const SeqDesc* seqs, int layer, int nsplit,
                                    float* part_o, float* part_ml, const ActBuf& out,
                                    hipStream_t st, const RopeIn* rope = nullptr);

// Prefill: rotate q (in place) and k of T rows at positions p0..p0+T-1 and
// append k, v to the cache.  qkv rows are [Hq*hd | Hkv*hd | Hkv*hd] fp32.
// nsplit > 1: the projection was split along K and its rows are the sums, in
// range order, of the nsplit partial products part[s * p_split + ...] (same row
// layout); the rotated queries are then written to qkv.
hipError_t launch_rope_append(bool kv_bf16, float* qkv, int T, int p0, int Hq,
                              const float* cos_t, const float* sin_t, KvLayout kv,
                              hipStream_t st, const float* part = nullptr, int nsplit = 1,
                              size_t p_split = 0);

// Prefill attention: queries = rotated q rows of qkv (T rows at p0..), keys =
// cache positions [0, p0+T), causal; out [T, Hq*hd] (row stride Hq*hd).  With a
// bf16 cache and split output, the scores and probabilities go through the matrix
// cores with the query and the probabilities as `terms` bf16 terms (1-3; 0: as
// many as `out` stores).
hipError_t launch_attn_prefill(bool kv_bf16, const float* qkv, int T, int p0, int Hq,
                               KvLayout kv, const ActBuf& out, hipStream_t st, int terms = 0);


// Decode attention at position state->pos: q = the rotated, pre-scaled queries
// [Hq*hd] (the QKV GEMV's GEMV_QKV output), keys and values = cache positions
// [0, pos] (the new position already appended by that GEMV); splits of 64
// positions (grid nsplit x Hkv, nsplit = attn_decode_splits(max_seq)) merged
// into out [Hq*hd] fp32.
// fuse != nullptr merges in the last split block where the launch allows it.
hipError_t launch_attn_decode(bool kv_bf16, const float* q, int Hq, KvLayout kv,
                              const void* state, int nsplit, float* part_o, float* part_ml,
                              float* out, const AttnFuse* fuse, hipStream_t st);
int attn_decode_splits(int max_seq);
bool attn_group_supported(int G);

// C[M, N] (ldc) = A[M, K] (lda) x W[N, K]^T with epilogue STORE / RESID (into C,
// fp32) or SWIGLU (H[M, N/2] (ldh) = silu(gate) * up of the packed column pairs,
// written as an activation buffer).  A.nt == 0: vector fp32 product (W bf16 or
// fp32); A.nt = 1..3: matrix-core product of the nt bf16 planes with bf16 W.
// K must be a multiple of 32.
hipError_t launch_gemm(int wt, int epi, const ActBuf& A, int lda, const void* W, int M,
                       int N, int K, float* C, int ldc, const ActBuf& H, int ldh,
                       hipStream_t st);
// The same product (matrix cores, nt >= 1, M > 32) over nsplit K ranges of equal
// depth (K a multiple of 32 nsplit): range s writes P + s * p_split ([M, N], row
// stride N, fp32).  gemm_split_count picks nsplit (1: do not split).
hipError_t launch_gemm_split(int wt, const ActBuf& A, int lda, const void* W, int M, int N, int K,
                             int nsplit, float* P, size_t p_split, hipStream_t st);
int gemm_split_count(int wt, int nt, int M, int N, int K, int max_split);
// The product for at most 32 rows (a batched decode step), bf16 weights, nt >= 1,
// K a multiple of 128, staged through LDS in whole lines; otherwise, or for other
// weight types, launch_gemm.  With part (part_floats floats), sync
// (kGemmRowsSyncInts ints, zero before the first launch and zero again after
// every launch) and fault all non-null, products with few weight rows are split
// along K and summed in the launch by the last split of each 64-row tile, all
// splits of a tile on one XCD; *fault is set to 1 if they were not (the result
// cannot be trusted then; with drill, every split-K sum reports so, for tests of
// the error path).  Launches that share sync must not overlap.
constexpr int kGemmRowsSyncInts = 512 * 64;
int gemm_rows_splits(int M, int N, int K, size_t part_floats);
hipError_t launch_gemm_rows(int wt, int epi, const ActBuf& A, int lda, const void* W, int M,
                            int N, int K, float* C, int ldc, const ActBuf& H, int ldh,
                            float* part, size_t part_floats, int* sync, int* fault,
                            hipStream_t st, bool drill = false);
// x[t] += sum over s < nsplit of P[s * p_split + t * d] (in that order) for T rows
// of width d; then, with gain != nullptr, y[t] = RMSNorm(x[t]) * gain (as
// launch_rmsnorm_rows).
hipError_t launch_resid_sum_rmsnorm(float* x, const float* P, int nsplit, size_t p_split,
                                    const float* gain, float eps, int T, int d, const ActBuf& y,
                                    hipStream_t st);

}  // namespace wici
