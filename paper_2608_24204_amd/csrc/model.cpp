// libwici runtime and C ABI: configuration checks, device memory layout, weight
// packing, the chunked-prefill loop, and the per-token decode step, captured
// once as a HIP graph and replayed for every token (the fixed per-token call
// group the paper replays as a trace, Sec. "Batching and Trace Replay").
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <algorithm>
#include <atomic>
#include <cstring>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/wici.h"
#include "common.h"
#include "kernels.h"

using wici::ArgmaxPart;
using wici::DecodeState;
static_assert((int)wici::W_F32 == WICI_F32 && (int)wici::W_BF16 == WICI_BF16 &&
                  (int)wici::W_Q8 == WICI_Q8,
              "kernel weight types follow wici_dtype");

namespace {

constexpr size_t kAlign = 256;
constexpr int kMaxGemvBlocks = 1024;
constexpr int kMaxBatch = 256;  // sequences per batched decode step
constexpr size_t kFuseRopeMaxBlocks = 3 * 4 * 256;  // see enqueue_decode_batch
constexpr int kMaxKSplit = 4;   // K ranges of a prefill residual product (partials kept)

size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }
size_t dsize(int32_t dt) { return dt == WICI_BF16 ? 2 : 4; }

// bf16 activation terms stored for the prefill products, read by each of them,
// and carried by the prefill attention's query and probabilities
struct Planes {
  int store, qkv, o, gu, down, attn;
};
Planes prefill_planes(const wici_config& c) {
  const int nt = c.prefill_mode == WICI_PREFILL_F32 ? 0
                 : c.prefill_mode == WICI_PREFILL_BF16 ? 1
                 : c.prefill_mode == WICI_PREFILL_BF16X2 ? 2 : 3;
  Planes p{nt, nt, nt, nt, nt, nt};
  // (two attention terms flip the 8B shape's 8-bit run at a near tie: three stay)
  if (c.prefill_mode == WICI_PREFILL_BF16X3Q) p = Planes{3, 3, 2, 2, 2, 3};
  if (c.prefill_planes) {
    p.qkv = c.prefill_planes & 3;
    p.o = (c.prefill_planes >> 2) & 3;
    p.gu = (c.prefill_planes >> 4) & 3;
    p.down = (c.prefill_planes >> 6) & 3;
    const int at = (c.prefill_planes >> 8) & 3;
    p.attn = at ? at : nt;
  }
  return p;
}

struct Layout {
  // weights
  size_t l_wqkv, l_wo, l_wgu, l_wdown, l_anorm, l_fnorm, layer_stride;
  size_t embed, final_norm, lm_head, rope_cos, rope_sin, weight_bytes;
  // kv
  int n_pages;
  size_t kv_layer_stride, kv_bytes;
  // scratch
  size_t x, a, qkv, att, h, kpart, logits, parts, part_o, part_ml, tokens, table, state, hist,
      seqs, attn_sync, gemm_sync;
  size_t scratch_bytes;
  int nsplit;
};

bool config_ok(const wici_config* c, std::string* why) {
  auto bad = [&](const char* m) { if (why) *why = m; return false; };
  if (!c) return bad("config is NULL");
  if (c->n_layers < 1 || c->n_layers > 4096) return bad("n_layers out of range");
  if (c->d_model < 64 || c->d_model % 64) return bad("d_model must be a positive multiple of 64");
  if (c->ffn_dim < 64 || c->ffn_dim % 64) return bad("ffn_dim must be a positive multiple of 64");
  if (c->head_dim != 64 && c->head_dim != 128) return bad("head_dim must be 64 or 128");
  if (c->n_kv_heads < 1 || c->n_heads < 1 || c->n_heads % c->n_kv_heads)
    return bad("n_heads must be a positive multiple of n_kv_heads");
  if (!wici::attn_group_supported(c->n_heads / c->n_kv_heads))
    return bad("query heads per KV head must be 1, 2, 4, 5 or 8");
  if (c->max_seq > 16384) return bad("max_seq above 16384");
  if (c->n_heads > 128) return bad("at most 128 query heads");
  // the decode GEMV stages its whole input vector in LDS
  if (c->d_model > 32768 || c->ffn_dim > 32768 || c->n_heads * c->head_dim > 32768)
    return bad("d_model, ffn_dim and n_heads*head_dim must be at most 32768");
  if (c->vocab < 1) return bad("vocab must be >= 1");
  if (!(c->rms_eps > 0.f) || !std::isfinite(c->rms_eps)) return bad("rms_eps must be > 0");
  if (!(c->rope_base > 1.0) || !std::isfinite(c->rope_base)) return bad("rope_base must be > 1");
  if (c->weight_dtype != WICI_F32 && c->weight_dtype != WICI_BF16 && c->weight_dtype != WICI_Q8)
    return bad("bad weight_dtype");
  if (c->kv_dtype != WICI_F32 && c->kv_dtype != WICI_BF16) return bad("bad kv_dtype");
  if (c->max_seq < 1 || c->max_seq > (1 << 20)) return bad("max_seq out of range");
  if (c->prefill_chunk < 1 || c->prefill_chunk > 8192) return bad("prefill_chunk out of range");
  if (c->kv_page != 16 && c->kv_page != 32 && c->kv_page != 64 && c->kv_page != 128)
    return bad("kv_page must be 16, 32, 64 or 128");
  if (c->prefill_mode < WICI_PREFILL_BF16X2 || c->prefill_mode > WICI_PREFILL_BF16X3Q)
    return bad("bad prefill_mode");
  if (c->weight_dtype == WICI_F32 && c->prefill_mode != WICI_PREFILL_F32)
    return bad("fp32 weights need prefill_mode WICI_PREFILL_F32");
  // the decode GEMV keeps each lane's slices of x in registers
  if (c->weight_dtype == WICI_F32 &&
      (c->d_model > 16384 || c->ffn_dim > 16384 || c->n_heads * c->head_dim > 16384))
    return bad("fp32 weights need d_model, ffn_dim and n_heads*head_dim of at most 16384");
  if (c->flags & ~(WICI_FLAG_NO_GRAPH | WICI_FLAG_FAULT_DRILL)) return bad("unknown flags");
  if (c->prefill_planes != 0) {
    if (c->prefill_mode != WICI_PREFILL_BF16X3)
      return bad("prefill_planes needs prefill_mode WICI_PREFILL_BF16X3");
    if (c->prefill_planes & ~0x3ff) return bad("prefill_planes has bits above 9");
    for (int i = 0; i < 4; ++i)
      if (((c->prefill_planes >> (2 * i)) & 3) == 0) return bad("prefill_planes: a field of 0");
  }
  if (c->tied_embeddings != 0 && c->tied_embeddings != 1) return bad("tied_embeddings must be 0 or 1");
  return true;
}

Layout make_layout(const wici_config& c) {
  Layout L{};
  const int wt = c.weight_dtype;
  const size_t d = c.d_model, F = c.ffn_dim, V = c.vocab;
  const size_t qd = (size_t)c.n_heads * c.head_dim, kvd = (size_t)c.n_kv_heads * c.head_dim;
  const size_t nqkv = qd + 2 * kvd;
  auto mat = [&](size_t n, size_t k) { return wici::weight_bytes(wt, n, k); };
  size_t o = 0;
  L.l_wqkv = o; o = align_up(o + mat(nqkv, d));
  L.l_wo = o; o = align_up(o + mat(d, qd));
  L.l_wgu = o; o = align_up(o + mat(2 * F, d));
  L.l_wdown = o; o = align_up(o + mat(d, F));
  L.l_anorm = o; o = align_up(o + d * 4);
  L.l_fnorm = o; o = align_up(o + d * 4);
  L.layer_stride = o;
  o = L.layer_stride * c.n_layers;
  L.embed = o; o = align_up(o + mat(V, d));
  L.final_norm = o; o = align_up(o + d * 4);
  if (c.tied_embeddings) {
    L.lm_head = L.embed;
  } else {
    L.lm_head = o; o = align_up(o + mat(V, d));
  }
  const size_t half = c.head_dim / 2;
  L.rope_cos = o; o = align_up(o + (size_t)c.max_seq * half * 4);
  L.rope_sin = o; o = align_up(o + (size_t)c.max_seq * half * 4);
  L.weight_bytes = o;

  L.n_pages = (c.max_seq + c.kv_page - 1) / c.kv_page;
  L.kv_layer_stride = align_up((size_t)L.n_pages * 2 * c.n_kv_heads * c.kv_page * c.head_dim *
                               dsize(c.kv_dtype));
  L.kv_bytes = L.kv_layer_stride * c.n_layers;

  L.nsplit = wici::attn_decode_splits(c.max_seq);
  const size_t C = c.prefill_chunk;
  o = 0;
  // activation buffers hold fp32 rows or up to three bf16 planes (6 bytes/value)
  L.x = o; o = align_up(o + C * d * 4);
  L.a = o; o = align_up(o + C * d * 6);
  L.qkv = o; o = align_up(o + C * nqkv * 4);
  L.att = o; o = align_up(o + C * qd * 6);
  L.h = o; o = align_up(o + C * F * 6);
  L.kpart = o; o = align_up(o + (size_t)kMaxKSplit * C * d * 4);  // split-K partials
  L.logits = o; o = align_up(o + V * 4);
  L.parts = o; o = align_up(o + kMaxGemvBlocks * sizeof(ArgmaxPart));
  L.part_o = o; o = align_up(o + (size_t)c.n_heads * L.nsplit * c.head_dim * 4);
  L.part_ml = o; o = align_up(o + (size_t)c.n_heads * L.nsplit * 2 * 4);
  // token ids: a whole prompt (copied once per prefill call), or a batch's tokens
  L.tokens = o; o = align_up(o + (size_t)std::max<int64_t>(C, std::max(c.max_seq, kMaxBatch)) * 4);
  L.table = o; o = align_up(o + (size_t)L.n_pages * 4);
  L.state = o; o = align_up(o + sizeof(DecodeState));
  L.hist = o; o = align_up(o + (size_t)c.max_seq * 4);  // token emitted after each position
  L.seqs = o; o = align_up(o + (size_t)kMaxBatch * sizeof(wici::SeqDesc));  // batched decode
  // counters and XCD records of the decode attention's in-launch merge
  L.attn_sync = o; o = align_up(o + (size_t)wici::attn_fuse_ints(c.n_kv_heads) * 4);
  // counters and XCD records of the batched products' split-K sums
  L.gemm_sync = o; o = align_up(o + (size_t)wici::kGemmRowsSyncInts * 4);
  L.scratch_bytes = o;
  return L;
}

enum TensorKind { T_EMBED, T_FINAL_NORM, T_LM_HEAD, T_ANORM, T_WQ, T_WK, T_WV, T_WO, T_FNORM,
                  T_GATE, T_UP, T_DOWN };

struct TensorSpec {
  TensorKind kind;
  int layer;
  int32_t dtype;
  int ndim;
  int64_t rows, cols;
};

}  // namespace

struct wici_model {
  wici_config cfg{};
  Layout L{};
  hipStream_t stream = nullptr;
  bool bound = false, failed = false;
  char* dw = nullptr;
  char* dkv = nullptr;
  char* ds = nullptr;
  std::string err;
  std::unordered_map<std::string, int> spec_index;
  std::vector<TensorSpec> specs;
  std::vector<uint8_t> loaded;
  int n_loaded = 0;
  int32_t pos = 0;
  bool have_token = false;
  bool shared_weights = false;  // weights bound from another model (read-only here)
  DecodeState* h_state = nullptr;         // pinned, device-mapped state mirror (host view)
  DecodeState* d_state_mirror = nullptr;  // the same memory as the kernels address it
  hipGraph_t graph = nullptr;
  hipGraphExec_t gexec = nullptr;
  // batched decode steps led by this model, captured per batch size (the
  // sequences' descriptors are read from device memory, so a graph serves any
  // group of that size)
  std::unordered_map<int, std::pair<hipGraph_t, hipGraphExec_t>> batch_graphs;
  int gemv_lm_blocks = 0;

  bool ready() const { return bound && n_loaded == (int)specs.size(); }
  template <typename T> T* W(size_t off) const { return reinterpret_cast<T*>(dw + off); }
  template <typename T> T* S(size_t off) const { return reinterpret_cast<T*>(ds + off); }
  size_t layer(int l, size_t off) const { return (size_t)l * L.layer_stride + off; }
  wici::KvLayout kv(int l) const {
    wici::KvLayout k;
    k.base = dkv + (size_t)l * L.kv_layer_stride;
    k.table = S<int32_t>(L.table);
    k.page = cfg.kv_page;
    k.n_kv = cfg.n_kv_heads;
    k.hd = cfg.head_dim;
    k.max_pos = cfg.max_seq;
    return k;
  }
};

namespace {

wici_status fail(wici_model* m, wici_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  m->err = buf;
  return s;
}

#define HIP_TRY(m, expr)                                                                   \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess) {                                                                \
      (m)->failed = true;                                                                  \
      return fail((m), WICI_E_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));         \
    }                                                                                      \
  } while (0)

void build_specs(wici_model* m) {
  const wici_config& c = m->cfg;
  const int64_t d = c.d_model, F = c.ffn_dim, V = c.vocab;
  const int64_t qd = (int64_t)c.n_heads * c.head_dim, kvd = (int64_t)c.n_kv_heads * c.head_dim;
  auto add = [&](const std::string& name, TensorKind k, int l, int32_t dt, int nd, int64_t r,
                 int64_t cc) {
    m->spec_index[name] = (int)m->specs.size();
    m->specs.push_back({k, l, dt, nd, r, cc});
  };
  const int32_t wd = c.weight_dtype;
  add("tok_embeddings", T_EMBED, -1, wd, 2, V, d);
  for (int l = 0; l < c.n_layers; ++l) {
    const std::string p = "layers." + std::to_string(l) + ".";
    add(p + "attn_norm", T_ANORM, l, WICI_F32, 1, d, 1);
    add(p + "wq", T_WQ, l, wd, 2, qd, d);
    add(p + "wk", T_WK, l, wd, 2, kvd, d);
    add(p + "wv", T_WV, l, wd, 2, kvd, d);
    add(p + "wo", T_WO, l, wd, 2, d, qd);
    add(p + "ffn_norm", T_FNORM, l, WICI_F32, 1, d, 1);
    add(p + "w_gate", T_GATE, l, wd, 2, F, d);
    add(p + "w_up", T_UP, l, wd, 2, F, d);
    add(p + "w_down", T_DOWN, l, wd, 2, d, F);
  }
  add("norm", T_FINAL_NORM, -1, WICI_F32, 1, d, 1);
  if (!c.tied_embeddings) add("lm_head", T_LM_HEAD, -1, wd, 2, V, d);
  m->loaded.assign(m->specs.size(), 0);
}

bool usable(const wici_model* m) { return m && !m->failed; }

// Enqueue one decode step (position and input token read from device state).
// With `timers`, every launcher call is timed: a start/stop event pair recorded
// by the dispatches of its first and last kernel (the profiling entry point uses
// this; graph capture never does).
hipError_t enqueue_decode(wici_model* m, std::vector<wici::LaunchTimer>* timers = nullptr) {
  const wici_config& c = m->cfg;
  const Layout& L = m->L;
  const int wb = c.weight_dtype;
  const bool kb = c.kv_dtype == WICI_BF16;
  const int d = c.d_model, F = c.ffn_dim, qd = c.n_heads * c.head_dim;
  const int nqkv = qd + 2 * c.n_kv_heads * c.head_dim;
  float* x = m->S<float>(L.x);
  float* qkv = m->S<float>(L.qkv);
  float* att = m->S<float>(L.att);
  float* h = m->S<float>(L.h);
  void* st = m->ds + L.state;
  hipStream_t s = m->stream;
  hipError_t e;
  wici::LaunchTimer cur{};
  auto arm = [&]() -> hipError_t {
    if (!timers) return hipSuccess;
    hipError_t r = hipEventCreate(&cur.start);
    if (r == hipSuccess) r = hipEventCreate(&cur.stop);
    if (r == hipSuccess) wici::set_launch_timer(&cur);
    return r;
  };
  auto disarm = [&]() {
    if (!timers) return;
    wici::set_launch_timer(nullptr);
    timers->push_back(cur);
  };
#define WICI_STEP(call)         \
  do {                          \
    if ((e = arm())) return e;  \
    e = (call);                 \
    disarm();                   \
    if (e) return e;            \
  } while (0)
  wici::AttnFuse fuse{};
  fuse.cnt = m->S<int>(L.attn_sync);
  fuse.xcc = fuse.cnt + c.n_kv_heads * 64;
  fuse.state = st;
  fuse.drill = (c.flags & WICI_FLAG_FAULT_DRILL) != 0;
  // bf16 weights: the first QKV projection gathers the embedding row itself (its
  // profiling slot stays, at zero time)
  const bool fold_embed = wb == WICI_BF16;
  if (fold_embed) {
    if (timers) timers->push_back(wici::LaunchTimer{nullptr, nullptr});
  } else {
    WICI_STEP(wici::launch_embed(wb, m->dw + L.embed, c.vocab, d, nullptr, 1, st, x, s));
  }
  for (int l = 0; l < c.n_layers; ++l) {
    wici::QkvRope rope{};
    rope.cos_t = m->W<float>(L.rope_cos);
    rope.sin_t = m->W<float>(L.rope_sin);
    rope.state = st;
    rope.kv = m->kv(l);
    rope.kv_bf16 = kb ? 1 : 0;
    rope.n_q = c.n_heads;
    rope.q_scale = 1.0f / std::sqrt((float)c.head_dim);
    rope.embed = fold_embed && l == 0 ? m->dw + L.embed : nullptr;
    WICI_STEP(wici::launch_gemv(wb, wici::GEMV_QKV, m->dw + m->layer(l, L.l_wqkv), nqkv, d, x,
                                m->W<float>(m->layer(l, L.l_anorm)), c.rms_eps, qkv, nullptr,
                                nullptr, s, &rope));
    WICI_STEP(wici::launch_attn_decode(kb, qkv, c.n_heads, m->kv(l), st, L.nsplit,
                                       m->S<float>(L.part_o), m->S<float>(L.part_ml), att,
                                       kb ? &fuse : nullptr, s));
    WICI_STEP(wici::launch_gemv(wb, wici::GEMV_RESID, m->dw + m->layer(l, L.l_wo), d, qd, att,
                                nullptr, 0.f, x, nullptr, nullptr, s));
    WICI_STEP(wici::launch_gemv(wb, wici::GEMV_SWIGLU, m->dw + m->layer(l, L.l_wgu), 2 * F, d, x,
                                m->W<float>(m->layer(l, L.l_fnorm)), c.rms_eps, h, nullptr,
                                nullptr, s));
    WICI_STEP(wici::launch_gemv(wb, wici::GEMV_RESID, m->dw + m->layer(l, L.l_wdown), d, F, h,
                                nullptr, 0.f, x, nullptr, nullptr, s));
  }
  int nb = 0;
  WICI_STEP(wici::launch_gemv(wb, wici::GEMV_ARGMAX, m->dw + L.lm_head, c.vocab, d, x,
                              m->W<float>(L.final_norm), c.rms_eps, m->S<float>(L.logits),
                              m->S<ArgmaxPart>(L.parts), &nb, s));
  WICI_STEP(wici::launch_argmax_final(m->S<ArgmaxPart>(L.parts), nb, st, m->S<int32_t>(L.hist), 1,
                                      -1, m->d_state_mirror, s));
#undef WICI_STEP
  return hipSuccess;
}

// Enqueue one prefill chunk of T rows at positions p0.. (token ids already on
// the device); x[T-1] holds the last row's residual stream afterwards.
hipError_t enqueue_prefill_chunk(wici_model* m, int p0, int T, int tok_off) {
  const wici_config& c = m->cfg;
  const Layout& L = m->L;
  const int wb = c.weight_dtype;
  const bool kb = c.kv_dtype == WICI_BF16;
  const int d = c.d_model, F = c.ffn_dim, qd = c.n_heads * c.head_dim;
  const int nqkv = qd + 2 * c.n_kv_heads * c.head_dim;
  float* x = m->S<float>(L.x);
  float* qkv = m->S<float>(L.qkv);
  const size_t C = c.prefill_chunk;
  const Planes pl = prefill_planes(c);
  const int nt = pl.store;
  auto act = [&](size_t off, size_t width) {
    wici::ActBuf b;
    b.f32 = m->S<float>(off);
    b.planes = m->S<wici::bf16_t>(off);
    b.plane_stride = C * width;
    b.nt = nt;
    return b;
  };
  // the same buffer as a product reads it: its first n terms
  auto rd = [](wici::ActBuf b, int n) {
    b.nt = b.nt == 0 ? 0 : n;
    return b;
  };
  const wici::ActBuf a = act(L.a, d), att = act(L.att, qd), h = act(L.h, F);
  const wici::ActBuf none{};
  hipStream_t s = m->stream;
  hipError_t e;
  if ((e = wici::launch_embed(wb, m->dw + L.embed, c.vocab, d, m->S<int32_t>(L.tokens) + tok_off,
                              T, nullptr, x, s)))
    return e;
  // The residual products (O, down) have only d output columns: with few rows
  // they are split along K into partials that the next row RMSNorm adds to x
  // (in split order, so the result does not depend on scheduling).
  float* P = m->S<float>(L.kpart);
  const size_t p_split = C * d;
  const int s_o = wici::gemm_split_count(wb, rd(att, pl.o).nt, T, d, qd, kMaxKSplit);
  const int s_d = wici::gemm_split_count(wb, rd(h, pl.down).nt, T, d, F, kMaxKSplit);
  // the QKV projection too, as far as its partials fit the split buffer; they are
  // added (in range order) by the RoPE + append kernel.  Measured at 1024 rows
  // (8B): 185 -> 164 us; at 512 rows (1B): 56 -> 33 us.
  const int s_q = wici::gemm_split_count(wb, rd(a, pl.qkv).nt, T, nqkv, d,
                                         std::min(kMaxKSplit, kMaxKSplit * d / nqkv));
  const size_t q_split = C * nqkv;
  int pending = 0;  // splits of the previous down product not yet added to x
  // (the normalised rows are written with as many terms as their product reads)
  auto norm = [&](const float* gain, int nsplit, int terms) {
    const wici::ActBuf y = rd(a, terms);
    return nsplit > 1 ? wici::launch_resid_sum_rmsnorm(x, P, nsplit, p_split, gain, c.rms_eps, T,
                                                       d, y, s)
                      : wici::launch_rmsnorm_rows(x, gain, c.rms_eps, T, d, y, s);
  };
  auto resid = [&](const wici::ActBuf& in, int K, size_t w, int nsplit) {
    return nsplit > 1 ? wici::launch_gemm_split(wb, in, K, m->dw + w, T, d, K, nsplit, P, p_split,
                                                s)
                      : wici::launch_gemm(wb, wici::GEMV_RESID, in, K, m->dw + w, T, d, K, x, d,
                                          none, 0, s);
  };
  for (int l = 0; l < c.n_layers; ++l) {
    if ((e = norm(m->W<float>(m->layer(l, L.l_anorm)), pending, pl.qkv))) return e;
    if (s_q > 1) {
      if ((e = wici::launch_gemm_split(wb, rd(a, pl.qkv), d, m->dw + m->layer(l, L.l_wqkv), T,
                                       nqkv, d, s_q, P, q_split, s)))
        return e;
    } else if ((e = wici::launch_gemm(wb, wici::GEMV_STORE, rd(a, pl.qkv), d,
                                      m->dw + m->layer(l, L.l_wqkv), T, nqkv, d, qkv, nqkv, none,
                                      0, s))) {
      return e;
    }
    if ((e = wici::launch_rope_append(kb, qkv, T, p0, c.n_heads, m->W<float>(L.rope_cos),
                                      m->W<float>(L.rope_sin), m->kv(l), s, s_q > 1 ? P : nullptr,
                                      s_q, q_split)))
      return e;
    if ((e = wici::launch_attn_prefill(kb, qkv, T, p0, c.n_heads, m->kv(l), att, s, pl.attn)))
      return e;
    if ((e = resid(rd(att, pl.o), qd, m->layer(l, L.l_wo), s_o))) return e;
    if ((e = norm(m->W<float>(m->layer(l, L.l_fnorm)), s_o, pl.gu))) return e;
    if ((e = wici::launch_gemm(wb, wici::GEMV_SWIGLU, rd(a, pl.gu), d,
                               m->dw + m->layer(l, L.l_wgu), T, 2 * F, d, nullptr, 0, h, F, s)))
      return e;
    if ((e = resid(rd(h, pl.down), F, m->layer(l, L.l_wdown), s_d))) return e;
    pending = s_d;
  }
  if (pending > 1)
    return wici::launch_resid_sum_rmsnorm(x, P, pending, p_split, nullptr, 0.f, T, d, a, s);
  return hipSuccess;
}

// Enqueue one batched decode step of B sequences (descriptors already in the
// lead model's scratch) on the lead's stream, in its scratch: row b of every
// activation matrix is sequence b.  The projections are the prefill products
// (matrix cores with the lead's prefill mode, or the vector product), the
// per-sequence parts (RoPE and append, attention, argmax) read the descriptors.
hipError_t enqueue_decode_batch(wici_model* m, int B) {
  const wici_config& c = m->cfg;
  const Layout& L = m->L;
  const int wb = c.weight_dtype;
  const bool kb = c.kv_dtype == WICI_BF16;
  const int d = c.d_model, F = c.ffn_dim, qd = c.n_heads * c.head_dim;
  const int nqkv = qd + 2 * c.n_kv_heads * c.head_dim;
  const size_t C = c.prefill_chunk;
  const Planes pl = prefill_planes(c);
  const int nt = pl.store;
  auto act = [&](size_t off, size_t width) {
    wici::ActBuf b;
    b.f32 = m->S<float>(off);
    b.planes = m->S<wici::bf16_t>(off);
    b.plane_stride = C * width;
    b.nt = nt;
    return b;
  };
  auto rd = [](wici::ActBuf b, int n) {
    b.nt = b.nt == 0 ? 0 : n;
    return b;
  };
  const wici::ActBuf a = act(L.a, d), att = act(L.att, qd), h = act(L.h, F);
  const wici::ActBuf none{};
  const wici::SeqDesc* seqs = m->S<wici::SeqDesc>(L.seqs);
  float* x = m->S<float>(L.x);
  float* qkv = m->S<float>(L.qkv);
  // attention partials and the logits live in the FFN buffer, free at those times
  float* part_o = m->S<float>(L.h);
  float* part_ml = part_o + (size_t)B * c.n_heads * L.nsplit * c.head_dim;
  float* logits = m->S<float>(L.h);
  wici::KvLayout kv = m->kv(0);  // geometry; pool and table come per sequence
  const float q_scale = 1.0f / std::sqrt((float)c.head_dim);
  const wici::RopeIn rope{m->W<float>(L.rope_cos), m->W<float>(L.rope_sin), q_scale};
  // A bf16 cache: the attention can apply RoPE and append the position itself
  // (one launch fewer per layer), but its registers then allow four workgroups
  // per CU instead of five.  Measured (8B, 21 splits): B = 2, 4, 8 +4%, +4%,
  // +2%, B = 16 even, B = 32 -2%; so only while its grid is at most about three
  // rounds of the chip at that occupancy.
  const bool fuse_rope = kb && (size_t)L.nsplit * c.n_kv_heads * B <= kFuseRopeMaxBlocks;
  hipStream_t s = m->stream;
  hipError_t e;
  // the products: split-K partials in the prefill's split buffer, a misplaced
  // split reported through the lead sequence's state
  float* gpart = m->S<float>(L.kpart);
  const size_t gpart_floats = (size_t)kMaxKSplit * C * d;
  int* gsync = m->S<int>(L.gemm_sync);
  int* gfault = &reinterpret_cast<DecodeState*>(m->ds + L.state)->fault;
  auto prod = [&](int epi, const wici::ActBuf& in, int K, size_t w, int N, float* out, int ldo,
                  const wici::ActBuf& hout, int ldh) {
    return wici::launch_gemm_rows(wb, epi, in, K, m->dw + w, B, N, K, out, ldo, hout, ldh,
                                  gpart, gpart_floats, gsync, gfault, s,
                                  (c.flags & WICI_FLAG_FAULT_DRILL) != 0);
  };
#define WICI_TRY(call) \
  do {                 \
    if ((e = (call))) return e; \
  } while (0)
  WICI_TRY(wici::launch_gather_tokens(seqs, B, m->S<int32_t>(L.tokens), s));
  WICI_TRY(wici::launch_embed(wb, m->dw + L.embed, c.vocab, d, m->S<int32_t>(L.tokens), B,
                              nullptr, x, s));
  for (int l = 0; l < c.n_layers; ++l) {
    WICI_TRY(wici::launch_rmsnorm_rows(x, m->W<float>(m->layer(l, L.l_anorm)), c.rms_eps, B, d,
                                       a, s));
    WICI_TRY(prod(wici::GEMV_STORE, rd(a, pl.qkv), d, m->layer(l, L.l_wqkv), nqkv, qkv, nqkv,
                  none, 0));
    if (!fuse_rope)
      WICI_TRY(wici::launch_rope_append_batch(kb, qkv, B, c.n_heads, m->W<float>(L.rope_cos),
                                              m->W<float>(L.rope_sin), seqs, l, kv, q_scale, s));
    WICI_TRY(wici::launch_attn_decode_batch(kb, qkv, nqkv, B, c.n_heads, kv, seqs, l, L.nsplit,
                                            part_o, part_ml, att, s, fuse_rope ? &rope : nullptr));
    WICI_TRY(prod(wici::GEMV_RESID, rd(att, pl.o), qd, m->layer(l, L.l_wo), d, x, d, none, 0));
    WICI_TRY(wici::launch_rmsnorm_rows(x, m->W<float>(m->layer(l, L.l_fnorm)), c.rms_eps, B, d,
                                       a, s));
    WICI_TRY(prod(wici::GEMV_SWIGLU, rd(a, pl.gu), d, m->layer(l, L.l_wgu), 2 * F, nullptr, 0, h,
                  F));
    WICI_TRY(prod(wici::GEMV_RESID, rd(h, pl.down), F, m->layer(l, L.l_wdown), d, x, d, none, 0));
  }
  WICI_TRY(wici::launch_rmsnorm_rows(x, m->W<float>(L.final_norm), c.rms_eps, B, d, a, s));
  WICI_TRY(prod(wici::GEMV_STORE, a, d, L.lm_head, c.vocab, logits, c.vocab, none, 0));
  WICI_TRY(wici::launch_argmax_rows(logits, B, c.vocab, seqs, s));
#undef WICI_TRY
  return hipSuccess;
}

// Configurations whose weight regions are interchangeable (shapes, storage,
// norm eps, RoPE tables, capacity).
bool same_weights_geometry(const wici_config& a, const wici_config& b) {
  return a.n_layers == b.n_layers && a.d_model == b.d_model && a.n_heads == b.n_heads &&
         a.n_kv_heads == b.n_kv_heads && a.head_dim == b.head_dim && a.ffn_dim == b.ffn_dim &&
         a.vocab == b.vocab && a.rms_eps == b.rms_eps && a.rope_base == b.rope_base &&
         a.tied_embeddings == b.tied_embeddings && a.weight_dtype == b.weight_dtype &&
         a.max_seq == b.max_seq;
}

// Pinned host memory that the final argmax kernel writes the step state into
// (coherent, so the kernel's stores reach it directly), replacing a
// device-to-host copy per step.
hipError_t alloc_state_mirror(wici_model* m) {
  if (m->h_state) return hipSuccess;
  if (hipError_t e = hipHostMalloc((void**)&m->h_state, sizeof(DecodeState),
                                   hipHostMallocMapped | hipHostMallocCoherent))
    return e;
  *m->h_state = DecodeState{};
  return hipHostGetDevicePointer((void**)&m->d_state_mirror, m->h_state, 0);
}

// An in-launch merge (the decode attention's, or a batched product's split-K
// sum) found its split blocks on different XCDs, so partials may have been read
// before they were visible: the results of the step cannot be trusted and the
// model stops here.
wici_status placement_fault(wici_model* m) {
  m->failed = true;
  m->have_token = false;
  return fail(m, WICI_E_HIP, "decode step: the split blocks of an attention head or of a "
                             "product tile did not all run on one XCD (workgroups not dealt to "
                             "the XCDs in turn)");
}

// Clear the mirror's `done` before queueing work whose final argmax writes it.
void arm_mirror(wici_model* m) {
  *static_cast<volatile int32_t*>(&m->h_state->done) = 0;
}

// Wait for the final argmax kernel's `done` in the pinned mirror: a spin on host
// memory, so the step's result is taken as soon as it lands rather than after
// the stream's completion has been signalled (on this runtime a wait of a few
// milliseconds ends in an interrupt-driven sleep, which costs ~15 us per step).
// The stream is polled as well: if it finishes or fails without `done`, returns
// false (the caller then synchronises and reports what the stream says).
bool wait_mirror(wici_model* m) {
  const volatile int32_t* done = &m->h_state->done;
  for (uint32_t i = 1;; ++i) {
    if (*done) {
      std::atomic_thread_fence(std::memory_order_acquire);
      return true;
    }
    if ((i & 1023) == 0 && hipStreamQuery(m->stream) != hipErrorNotReady) return *done != 0;
    __builtin_ia32_pause();
  }
}

// The step's final argmax kernel has written the new state into the pinned
// mirror m->h_state as well.  Without logits to copy, the call returns once the
// mirror's `done` is set (the stream may still be retiring that kernel; later
// work on it is ordered after it); otherwise once the stream has drained.
wici_status finish_step(wici_model* m, int32_t* tok, float* logits) {
  if (logits) {
    HIP_TRY(m, hipMemcpyAsync(logits, m->ds + m->L.logits, (size_t)m->cfg.vocab * 4,
                              hipMemcpyDeviceToHost, m->stream));
    HIP_TRY(m, hipStreamSynchronize(m->stream));
  } else if (!wait_mirror(m)) {
    HIP_TRY(m, hipStreamSynchronize(m->stream));
  }
  m->pos = m->h_state->pos;
  if (m->h_state->fault) return placement_fault(m);
  if (m->h_state->bad) {
    m->have_token = false;
    return fail(m, WICI_E_NUMERIC, "non-finite logits at position %d", m->pos - 1);
  }
  *tok = m->h_state->token;
  m->have_token = true;
  return WICI_OK;
}

// Queue `n` decode steps: replays of the captured step graph (captured on first
// use), or eager launches when graphs are off or the stream is the null stream.
hipError_t launch_decode_steps(wici_model* m, int n) {
  const bool use_graph = m->stream != nullptr && !(m->cfg.flags & WICI_FLAG_NO_GRAPH);
  if (!use_graph) {
    for (int i = 0; i < n; ++i)
      if (hipError_t e = enqueue_decode(m)) return e;
    return hipSuccess;
  }
  if (!m->gexec) {
    if (hipError_t e = hipStreamBeginCapture(m->stream, hipStreamCaptureModeThreadLocal)) return e;
    const hipError_t e = enqueue_decode(m);
    hipGraph_t g = nullptr;
    const hipError_t e2 = hipStreamEndCapture(m->stream, &g);
    if (e != hipSuccess) {
      if (g) (void)hipGraphDestroy(g);
      return e;
    }
    if (e2 != hipSuccess) return e2;
    m->graph = g;
    if (hipError_t e3 = hipGraphInstantiate(&m->gexec, m->graph, nullptr, nullptr, 0)) return e3;
  }
  for (int i = 0; i < n; ++i)
    if (hipError_t e = hipGraphLaunch(m->gexec, m->stream)) return e;
  return hipSuccess;
}

}  // namespace

// ============================================================================ C ABI

extern "C" {

wici_status wici_memory_requirements(const wici_config* cfg, size_t* weight_bytes,
                                     size_t* kv_bytes, size_t* scratch_bytes) {
  if (!config_ok(cfg, nullptr) || !weight_bytes || !kv_bytes || !scratch_bytes) return WICI_E_ARG;
  const Layout L = make_layout(*cfg);
  *weight_bytes = L.weight_bytes;
  *kv_bytes = L.kv_bytes;
  *scratch_bytes = L.scratch_bytes;
  return WICI_OK;
}

wici_status wici_create(const wici_config* cfg, void* hip_stream, wici_model** out) {
  if (!out) return WICI_E_ARG;
  *out = nullptr;
  if (!config_ok(cfg, nullptr)) return WICI_E_ARG;
  wici_model* m = new (std::nothrow) wici_model();
  if (!m) return WICI_E_ARG;
  m->cfg = *cfg;
  m->L = make_layout(*cfg);
  m->stream = static_cast<hipStream_t>(hip_stream);
  build_specs(m);
  *out = m;
  return WICI_OK;
}

wici_status wici_bind_memory(wici_model* m, void* d_weights, size_t weight_bytes, void* d_kv,
                             size_t kv_bytes, void* d_scratch, size_t scratch_bytes) {
  if (!m) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (m->bound) return fail(m, WICI_E_STATE, "memory already bound");
  if (!d_weights || !d_kv || !d_scratch) return fail(m, WICI_E_ARG, "NULL device pointer");
  if (weight_bytes < m->L.weight_bytes || kv_bytes < m->L.kv_bytes ||
      scratch_bytes < m->L.scratch_bytes)
    return fail(m, WICI_E_ARG, "device region too small");
  if (((uintptr_t)d_weights | (uintptr_t)d_kv | (uintptr_t)d_scratch) % kAlign)
    return fail(m, WICI_E_ARG, "device regions must be 256-byte aligned");
  m->dw = static_cast<char*>(d_weights);
  m->dkv = static_cast<char*>(d_kv);
  m->ds = static_cast<char*>(d_scratch);
  HIP_TRY(m, alloc_state_mirror(m));
  // RoPE angle table: pos * base^(-2j/hd), evaluated in double, stored as fp32.
  const wici_config& c = m->cfg;
  const int half = c.head_dim / 2;
  std::vector<float> cs((size_t)c.max_seq * half), sn((size_t)c.max_seq * half);
  for (int j = 0; j < half; ++j) {
    const double inv = std::pow(c.rope_base, -2.0 * j / c.head_dim);
    for (int p = 0; p < c.max_seq; ++p) {
      const double ang = (double)p * inv;
      cs[(size_t)p * half + j] = (float)std::cos(ang);
      sn[(size_t)p * half + j] = (float)std::sin(ang);
    }
  }
  HIP_TRY(m, hipMemcpy(m->dw + m->L.rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(m, hipMemcpy(m->dw + m->L.rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice));
  HIP_TRY(m, wici::launch_init_block_table(m->S<int32_t>(m->L.table), m->L.n_pages, m->stream));
  HIP_TRY(m, wici::launch_reset_state(m->ds + m->L.state, m->stream));
  HIP_TRY(m, wici::launch_fill_i32(m->S<int32_t>(m->L.attn_sync),
                                   wici::attn_fuse_ints(m->cfg.n_kv_heads), 0, m->stream));
  HIP_TRY(m, wici::launch_fill_i32(m->S<int32_t>(m->L.gemm_sync), wici::kGemmRowsSyncInts, 0,
                                   m->stream));
  HIP_TRY(m, hipStreamSynchronize(m->stream));
  m->bound = true;
  m->pos = 0;
  m->have_token = false;
  return WICI_OK;
}

wici_status wici_load_weights(wici_model* m, const wici_tensor* tensors, int32_t n_tensors) {
  if (!m) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (!m->bound) return fail(m, WICI_E_STATE, "wici_bind_memory must come first");
  if (m->shared_weights)
    return fail(m, WICI_E_STATE, "weights are shared with another model (load them there)");
  if (n_tensors < 0 || (n_tensors > 0 && !tensors)) return fail(m, WICI_E_ARG, "bad tensor list");
  std::vector<int> idx(n_tensors);
  std::vector<uint8_t> seen(m->specs.size(), 0);
  for (int i = 0; i < n_tensors; ++i) {
    const wici_tensor& t = tensors[i];
    if (!t.name) return fail(m, WICI_E_ARG, "tensor %d has no name", i);
    auto it = m->spec_index.find(t.name);
    if (it == m->spec_index.end()) return fail(m, WICI_E_ARG, "unknown tensor '%s'", t.name);
    const TensorSpec& sp = m->specs[it->second];
    if (seen[it->second]) return fail(m, WICI_E_ARG, "tensor '%s' given twice", t.name);
    seen[it->second] = 1;
    const bool dtype_ok = sp.dtype == WICI_Q8 ? (t.dtype == WICI_BF16 || t.dtype == WICI_F32)
                                              : t.dtype == sp.dtype;
    if (!dtype_ok) return fail(m, WICI_E_ARG, "tensor '%s': wrong dtype", t.name);
    const bool shape_ok = sp.ndim == 1 ? (t.ndim == 1 && t.shape[0] == sp.rows)
                                       : (t.ndim == 2 && t.shape[0] == sp.rows && t.shape[1] == sp.cols);
    if (!shape_ok) return fail(m, WICI_E_ARG, "tensor '%s': wrong shape", t.name);
    if (!t.data) return fail(m, WICI_E_ARG, "tensor '%s': NULL data", t.name);
    idx[i] = it->second;
  }
  const wici_config& c = m->cfg;
  const Layout& L = m->L;
  const size_t ws = dsize(c.weight_dtype), d = c.d_model;
  const size_t qd = (size_t)c.n_heads * c.head_dim, kvd = (size_t)c.n_kv_heads * c.head_dim;
  if (c.weight_dtype == WICI_Q8) {
    // quantise every matrix first (host), so a bad tensor uploads nothing
    std::vector<std::vector<uint8_t>> codes(n_tensors);
    std::vector<std::vector<uint16_t>> scales(n_tensors);
    for (int i = 0; i < n_tensors; ++i) {
      const wici_tensor& t = tensors[i];
      const TensorSpec& sp = m->specs[idx[i]];
      if (sp.dtype != WICI_Q8) continue;
      const size_t n = (size_t)sp.rows * sp.cols, es = dsize(t.dtype);
      std::vector<char> host;
      const void* src = t.data;
      if (t.on_device) {
        host.resize(n * es);
        HIP_TRY(m, hipMemcpy(host.data(), t.data, n * es, hipMemcpyDeviceToHost));
        src = host.data();
      }
      codes[i].resize(n);
      scales[i].resize(n / 32);
      if (wici_quantize_q8(src, t.dtype, sp.rows, sp.cols, codes[i].data(), scales[i].data()) !=
          WICI_OK)
        return fail(m, WICI_E_ARG, "tensor '%s': non-finite weight or scale overflow", t.name);
    }
    for (int i = 0; i < n_tensors; ++i) {
      const wici_tensor& t = tensors[i];
      const TensorSpec& sp = m->specs[idx[i]];
      if (sp.dtype != WICI_Q8) continue;
      // region of the packed matrix, its row count and width, this tensor's first
      // row and row step (2 for the interleaved gate/up rows)
      size_t base = 0, rows = sp.rows, r0 = 0, step = 1;
      const size_t K = sp.cols;
      switch (sp.kind) {
        case T_EMBED: base = L.embed; break;
        case T_LM_HEAD: base = L.lm_head; break;
        case T_WQ: base = m->layer(sp.layer, L.l_wqkv); rows = qd + 2 * kvd; break;
        case T_WK: base = m->layer(sp.layer, L.l_wqkv); rows = qd + 2 * kvd; r0 = qd; break;
        case T_WV: base = m->layer(sp.layer, L.l_wqkv); rows = qd + 2 * kvd; r0 = qd + kvd; break;
        case T_WO: base = m->layer(sp.layer, L.l_wo); break;
        case T_DOWN: base = m->layer(sp.layer, L.l_wdown); break;
        case T_GATE:
        case T_UP:
          base = m->layer(sp.layer, L.l_wgu); rows = 2 * (size_t)sp.rows;
          r0 = sp.kind == T_UP ? 1 : 0; step = 2;
          break;
        default: return fail(m, WICI_E_ARG, "tensor '%s': not a matrix", t.name);
      }
      char* dc = m->dw + base;
      char* dsc = dc + wici::q8_scale_offset(rows, K);
      const size_t sb = K / 32 * 2;  // scale bytes per row
      HIP_TRY(m, hipMemcpy2D(dc + r0 * K, step * K, codes[i].data(), K, K, (size_t)sp.rows,
                             hipMemcpyHostToDevice));
      HIP_TRY(m, hipMemcpy2D(dsc + r0 * sb, step * sb, scales[i].data(), sb, sb, (size_t)sp.rows,
                             hipMemcpyHostToDevice));
    }
  }
  for (int i = 0; i < n_tensors; ++i) {
    const wici_tensor& t = tensors[i];
    const TensorSpec& sp = m->specs[idx[i]];
    if (sp.dtype == WICI_Q8) continue;
    const hipMemcpyKind kind = t.on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    const size_t es = dsize(sp.dtype);
    const size_t bytes = (size_t)sp.rows * sp.cols * es;
    char* dst = nullptr;
    switch (sp.kind) {
      case T_EMBED: dst = m->dw + L.embed; break;
      case T_FINAL_NORM: dst = m->dw + L.final_norm; break;
      case T_LM_HEAD: dst = m->dw + L.lm_head; break;
      case T_ANORM: dst = m->dw + m->layer(sp.layer, L.l_anorm); break;
      case T_FNORM: dst = m->dw + m->layer(sp.layer, L.l_fnorm); break;
      case T_WQ: dst = m->dw + m->layer(sp.layer, L.l_wqkv); break;
      case T_WK: dst = m->dw + m->layer(sp.layer, L.l_wqkv) + qd * d * ws; break;
      case T_WV: dst = m->dw + m->layer(sp.layer, L.l_wqkv) + (qd + kvd) * d * ws; break;
      case T_WO: dst = m->dw + m->layer(sp.layer, L.l_wo); break;
      case T_DOWN: dst = m->dw + m->layer(sp.layer, L.l_wdown); break;
      case T_GATE:
      case T_UP: {
        // gate row i -> packed row 2i, up row i -> packed row 2i+1
        const size_t rb = d * ws;
        char* base = m->dw + m->layer(sp.layer, L.l_wgu) + (sp.kind == T_UP ? rb : 0);
        HIP_TRY(m, hipMemcpy2DAsync(base, 2 * rb, t.data, rb, rb, (size_t)sp.rows, kind, m->stream));
        continue;
      }
    }
    HIP_TRY(m, hipMemcpyAsync(dst, t.data, bytes, kind, m->stream));
  }
  HIP_TRY(m, hipStreamSynchronize(m->stream));
  for (int i = 0; i < n_tensors; ++i)
    if (!m->loaded[idx[i]]) { m->loaded[idx[i]] = 1; ++m->n_loaded; }
  return WICI_OK;
}

wici_status wici_prefill(wici_model* m, const int32_t* tokens, int32_t n_tokens,
                         int32_t* first_token, float* logits) {
  if (!m) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (!tokens || !first_token) return fail(m, WICI_E_ARG, "NULL tokens or first_token");
  if (n_tokens < 1) return fail(m, WICI_E_ARG, "n_tokens must be >= 1");
  for (int i = 0; i < n_tokens; ++i)
    if (tokens[i] < 0 || tokens[i] >= m->cfg.vocab)
      return fail(m, WICI_E_ARG, "token id %d at %d outside [0, %d)", tokens[i], i, m->cfg.vocab);
  if (!m->ready()) return fail(m, WICI_E_STATE, "weights not bound/loaded");
  if ((int64_t)m->pos + n_tokens > m->cfg.max_seq)
    return fail(m, WICI_E_CAPACITY, "position %d + %d tokens exceeds max_seq %d", m->pos, n_tokens,
                m->cfg.max_seq);
  const wici_config& c = m->cfg;
  const Layout& L = m->L;
  const int C = c.prefill_chunk;
  int last_T = 0;
  arm_mirror(m);
  // every chunk's ids in one copy (the buffer holds max_seq ids), so the chunks
  // queue back to back with no host wait between them
  HIP_TRY(m, hipMemcpyAsync(m->ds + L.tokens, tokens, (size_t)n_tokens * 4, hipMemcpyHostToDevice,
                            m->stream));
  for (int c0 = 0; c0 < n_tokens; c0 += C) {
    const int T = std::min(C, n_tokens - c0);
    HIP_TRY(m, enqueue_prefill_chunk(m, m->pos + c0, T, c0));
    last_T = T;
  }
  int nb = 0;
  const int wb = c.weight_dtype;
  HIP_TRY(m, wici::launch_gemv(wb, wici::GEMV_ARGMAX, m->dw + L.lm_head, c.vocab, c.d_model,
                               m->S<float>(L.x) + (size_t)(last_T - 1) * c.d_model,
                               m->W<float>(L.final_norm), c.rms_eps, m->S<float>(L.logits),
                               m->S<ArgmaxPart>(L.parts), &nb, m->stream));
  HIP_TRY(m, wici::launch_argmax_final(m->S<ArgmaxPart>(L.parts), nb, m->ds + L.state,
                                       m->S<int32_t>(L.hist), 0, m->pos + n_tokens,
                                       m->d_state_mirror, m->stream));
  return finish_step(m, first_token, logits);
}

wici_status wici_decode_step(wici_model* m, int32_t token_in, int32_t* next_token, float* logits) {
  if (!m) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (!next_token) return fail(m, WICI_E_ARG, "NULL next_token");
  if (token_in >= m->cfg.vocab) return fail(m, WICI_E_ARG, "token id %d >= vocab", token_in);
  if (!m->ready()) return fail(m, WICI_E_STATE, "weights not bound/loaded");
  if (m->pos < 1) return fail(m, WICI_E_STATE, "decode before prefill");
  if (token_in < 0 && !m->have_token) return fail(m, WICI_E_STATE, "no previous token to feed");
  if (m->pos + 1 > m->cfg.max_seq)
    return fail(m, WICI_E_CAPACITY, "position %d reached max_seq", m->pos);
  arm_mirror(m);
  if (token_in >= 0) HIP_TRY(m, wici::launch_set_token(m->ds + m->L.state, token_in, m->stream));
  HIP_TRY(m, launch_decode_steps(m, 1));
  return finish_step(m, next_token, logits);
}

wici_status wici_decode_n(wici_model* m, int32_t token_in, int32_t n, int32_t* tokens_out,
                          int32_t* n_done, float* logits) {
  if (!m) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (!tokens_out || !n_done) return fail(m, WICI_E_ARG, "NULL tokens_out or n_done");
  *n_done = 0;
  if (n < 1) return fail(m, WICI_E_ARG, "n must be >= 1");
  if (token_in >= m->cfg.vocab) return fail(m, WICI_E_ARG, "token id %d >= vocab", token_in);
  if (!m->ready()) return fail(m, WICI_E_STATE, "weights not bound/loaded");
  if (m->pos < 1) return fail(m, WICI_E_STATE, "decode before prefill");
  if (token_in < 0 && !m->have_token) return fail(m, WICI_E_STATE, "no previous token to feed");
  if ((int64_t)m->pos + n > m->cfg.max_seq)
    return fail(m, WICI_E_CAPACITY, "position %d + %d steps exceeds max_seq %d", m->pos, n,
                m->cfg.max_seq);
  const int32_t pos0 = m->pos;
  if (token_in >= 0) HIP_TRY(m, wici::launch_set_token(m->ds + m->L.state, token_in, m->stream));
  HIP_TRY(m, launch_decode_steps(m, n));
  // hist[pos0 .. pos0+n) holds the token emitted after each processed position
  // (-1 from a failed step on); the state says how far the run got.
  HIP_TRY(m, hipMemcpyAsync(tokens_out, m->ds + m->L.hist + (size_t)pos0 * 4, (size_t)n * 4,
                            hipMemcpyDeviceToHost, m->stream));
  if (logits)
    HIP_TRY(m, hipMemcpyAsync(logits, m->ds + m->L.logits, (size_t)m->cfg.vocab * 4,
                              hipMemcpyDeviceToHost, m->stream));
  HIP_TRY(m, hipStreamSynchronize(m->stream));
  m->pos = m->h_state->pos;
  const int32_t steps = m->pos - pos0;
  if (m->h_state->fault) {
    *n_done = 0;
    return placement_fault(m);
  }
  if (m->h_state->bad) {
    m->have_token = false;
    *n_done = steps - 1;
    for (int32_t i = steps - 1; i < n; ++i) tokens_out[i] = -1;
    return fail(m, WICI_E_NUMERIC, "non-finite logits at position %d (step %d of %d)", m->pos - 1,
                steps, n);
  }
  if (steps != n) {
    m->failed = true;
    return fail(m, WICI_E_HIP, "device ran %d of %d steps", steps, n);
  }
  *n_done = n;
  m->have_token = true;
  return WICI_OK;
}

wici_status wici_profile_decode_step(wici_model* m, int32_t token_in, int32_t* next_token,
                                     float* durations_ms, int32_t capacity, int32_t* n_written) {
  if (!m) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (!next_token || !durations_ms || !n_written) return fail(m, WICI_E_ARG, "NULL output");
  const int need = 3 + 5 * m->cfg.n_layers;
  if (capacity < need) return fail(m, WICI_E_ARG, "capacity %d < %d launches", capacity, need);
  if (token_in >= m->cfg.vocab) return fail(m, WICI_E_ARG, "token id %d >= vocab", token_in);
  if (!m->ready()) return fail(m, WICI_E_STATE, "weights not bound/loaded");
  if (m->pos < 1) return fail(m, WICI_E_STATE, "decode before prefill");
  if (token_in < 0 && !m->have_token) return fail(m, WICI_E_STATE, "no previous token to feed");
  if (m->pos + 1 > m->cfg.max_seq)
    return fail(m, WICI_E_CAPACITY, "position %d reached max_seq", m->pos);
  arm_mirror(m);
  if (token_in >= 0) HIP_TRY(m, wici::launch_set_token(m->ds + m->L.state, token_in, m->stream));
  std::vector<wici::LaunchTimer> tv;
  const hipError_t e = enqueue_decode(m, &tv);
  const hipError_t e2 = e == hipSuccess ? hipStreamSynchronize(m->stream) : e;
  int n = 0;
  hipError_t e3 = hipSuccess;
  if (e2 == hipSuccess)
    for (const wici::LaunchTimer& t : tv) {
      float ms = 0.f;  // a slot without events: a step folded into another launch
      const hipError_t r = t.start ? hipEventElapsedTime(&ms, t.start, t.stop) : hipSuccess;
      if (r != hipSuccess && e3 == hipSuccess) e3 = r;
      durations_ms[n++] = ms;
    }
  for (const wici::LaunchTimer& t : tv) {
    if (t.start) (void)hipEventDestroy(t.start);
    if (t.stop) (void)hipEventDestroy(t.stop);
  }
  HIP_TRY(m, e2);
  HIP_TRY(m, e3);
  *n_written = n;
  return finish_step(m, next_token, nullptr);
}

wici_status wici_bind_memory_shared(wici_model* m, const wici_model* src, void* d_kv,
                                    size_t kv_bytes, void* d_scratch, size_t scratch_bytes) {
  if (!m || !src || m == src) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (m->bound) return fail(m, WICI_E_STATE, "memory already bound");
  if (src->failed || !src->ready())
    return fail(m, WICI_E_STATE, "the source model has no complete weights");
  if (!same_weights_geometry(m->cfg, src->cfg))
    return fail(m, WICI_E_ARG, "configuration differs from the source model's weights");
  if (!d_kv || !d_scratch) return fail(m, WICI_E_ARG, "NULL device pointer");
  if (kv_bytes < m->L.kv_bytes || scratch_bytes < m->L.scratch_bytes)
    return fail(m, WICI_E_ARG, "device region too small");
  if (((uintptr_t)d_kv | (uintptr_t)d_scratch) % kAlign)
    return fail(m, WICI_E_ARG, "device regions must be 256-byte aligned");
  m->dw = src->dw;
  m->dkv = static_cast<char*>(d_kv);
  m->ds = static_cast<char*>(d_scratch);
  HIP_TRY(m, alloc_state_mirror(m));
  HIP_TRY(m, wici::launch_init_block_table(m->S<int32_t>(m->L.table), m->L.n_pages, m->stream));
  HIP_TRY(m, wici::launch_reset_state(m->ds + m->L.state, m->stream));
  HIP_TRY(m, wici::launch_fill_i32(m->S<int32_t>(m->L.attn_sync),
                                   wici::attn_fuse_ints(m->cfg.n_kv_heads), 0, m->stream));
  HIP_TRY(m, wici::launch_fill_i32(m->S<int32_t>(m->L.gemm_sync), wici::kGemmRowsSyncInts, 0,
                                   m->stream));
  HIP_TRY(m, hipStreamSynchronize(m->stream));
  m->loaded.assign(m->specs.size(), 1);
  m->n_loaded = (int)m->specs.size();
  m->shared_weights = true;
  m->bound = true;
  m->pos = 0;
  m->have_token = false;
  return WICI_OK;
}

wici_status wici_decode_batch(wici_model* const* models, int32_t n, const int32_t* tokens_in,
                              int32_t* next_tokens, float* logits) {
  if (!models || n < 1 || !next_tokens) return WICI_E_ARG;
  wici_model* lead = models[0];
  if (!lead) return WICI_E_ARG;
  if (lead->failed) return WICI_E_STATE;
  if (n > kMaxBatch || n > lead->cfg.prefill_chunk)
    return fail(lead, WICI_E_ARG, "%d sequences: at most %d (and the prefill chunk)", n,
                kMaxBatch);
  const wici_config& c = lead->cfg;
  const Layout& L = lead->L;
  // the FFN buffer holds the attention partials and the logits of all sequences
  const size_t h_bytes = (size_t)c.prefill_chunk * c.ffn_dim * 6;
  const size_t need = std::max((size_t)n * c.n_heads * L.nsplit * (c.head_dim + 2) * 4,
                               (size_t)n * c.vocab * 4);
  if (need > h_bytes) return fail(lead, WICI_E_ARG, "%d sequences exceed the batch scratch", n);
  std::vector<wici::SeqDesc> sd(n);
  for (int b = 0; b < n; ++b) {
    wici_model* mb = models[b];
    if (!mb) return fail(lead, WICI_E_ARG, "NULL model %d", b);
    for (int j = 0; j < b; ++j)
      if (models[j] == mb) return fail(lead, WICI_E_ARG, "model %d appears twice", b);
    if (mb->failed || !mb->ready()) return fail(lead, WICI_E_STATE, "model %d not ready", b);
    if (mb->dw != lead->dw || !same_weights_geometry(mb->cfg, c) ||
        mb->cfg.kv_dtype != c.kv_dtype || mb->cfg.kv_page != c.kv_page)
      return fail(lead, WICI_E_ARG, "model %d does not share the lead's weights and config", b);
    const int32_t t = tokens_in ? tokens_in[b] : -1;
    if (t >= c.vocab) return fail(lead, WICI_E_ARG, "token id %d >= vocab", t);
    if (mb->pos < 1) return fail(lead, WICI_E_STATE, "model %d: decode before prefill", b);
    if (t < 0 && !mb->have_token) return fail(lead, WICI_E_STATE, "model %d: no token", b);
    if (mb->pos + 1 > c.max_seq) return fail(lead, WICI_E_CAPACITY, "model %d is full", b);
    sd[b].kv = mb->dkv;
    sd[b].kv_layer_stride = mb->L.kv_layer_stride;
    sd[b].table = mb->S<int32_t>(mb->L.table);
    sd[b].state = mb->ds + mb->L.state;
    sd[b].hist = mb->S<int32_t>(mb->L.hist);
  }
  // one sequence: its own step graph (the weight-streaming GEMVs), which the
  // batched matrix products cannot beat at a single row
  if (n == 1) return wici_decode_step(lead, tokens_in ? tokens_in[0] : -1, next_tokens, logits);
  for (int b = 0; b < n; ++b)
    if (tokens_in && tokens_in[b] >= 0)
      HIP_TRY(lead, wici::launch_set_token(models[b]->ds + models[b]->L.state, tokens_in[b],
                                           lead->stream));
  HIP_TRY(lead, hipMemcpyAsync(lead->ds + L.seqs, sd.data(), n * sizeof(wici::SeqDesc),
                               hipMemcpyHostToDevice, lead->stream));
  const bool use_graph = lead->stream != nullptr && !(c.flags & WICI_FLAG_NO_GRAPH);
  if (use_graph) {
    auto it = lead->batch_graphs.find(n);
    if (it == lead->batch_graphs.end()) {
      HIP_TRY(lead, hipStreamBeginCapture(lead->stream, hipStreamCaptureModeThreadLocal));
      const hipError_t e = enqueue_decode_batch(lead, n);
      hipGraph_t g = nullptr;
      const hipError_t e2 = hipStreamEndCapture(lead->stream, &g);
      if (e != hipSuccess && g) (void)hipGraphDestroy(g);
      HIP_TRY(lead, e);
      HIP_TRY(lead, e2);
      hipGraphExec_t ge = nullptr;
      const hipError_t e3 = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
      if (e3 != hipSuccess) (void)hipGraphDestroy(g);
      HIP_TRY(lead, e3);
      it = lead->batch_graphs.emplace(n, std::make_pair(g, ge)).first;
    }
    HIP_TRY(lead, hipGraphLaunch(it->second.second, lead->stream));
  } else {
    HIP_TRY(lead, enqueue_decode_batch(lead, n));
  }
  std::vector<DecodeState> st(n);
  for (int b = 0; b < n; ++b)
    HIP_TRY(lead, hipMemcpyAsync(&st[b], models[b]->ds + models[b]->L.state, sizeof(DecodeState),
                                 hipMemcpyDeviceToHost, lead->stream));
  if (logits)
    HIP_TRY(lead, hipMemcpyAsync(logits, lead->ds + L.h, (size_t)n * c.vocab * 4,
                                 hipMemcpyDeviceToHost, lead->stream));
  HIP_TRY(lead, hipStreamSynchronize(lead->stream));
  if (st[0].fault) return placement_fault(lead);
  int bad = -1;
  for (int b = 0; b < n; ++b) {
    models[b]->pos = st[b].pos;
    models[b]->have_token = !st[b].bad;
    next_tokens[b] = st[b].bad ? -1 : st[b].token;
    if (st[b].bad && bad < 0) bad = b;
  }
  if (bad >= 0) return fail(lead, WICI_E_NUMERIC, "non-finite logits in sequence %d", bad);
  return WICI_OK;
}

wici_status wici_reset_kv(wici_model* m) {
  if (!m) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (!m->bound) return fail(m, WICI_E_STATE, "memory not bound");
  HIP_TRY(m, wici::launch_init_block_table(m->S<int32_t>(m->L.table), m->L.n_pages, m->stream));
  HIP_TRY(m, wici::launch_reset_state(m->ds + m->L.state, m->stream));
  HIP_TRY(m, hipStreamSynchronize(m->stream));
  m->pos = 0;
  m->have_token = false;
  return WICI_OK;
}

wici_status wici_stream_read(const void* d_buf, size_t bytes, int32_t grid, int32_t reps,
                             void* d_sink, void* hip_stream, float* ms_per_read,
                             uint32_t* checksum) {
  if (!d_buf || !d_sink || !ms_per_read || grid < 1 || grid > 65536 || reps < 1 ||
      bytes < 16384 || bytes % 16384)
    return WICI_E_ARG;
  hipStream_t s = static_cast<hipStream_t>(hip_stream);
  unsigned* sink = static_cast<unsigned*>(d_sink);
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  if (e == hipSuccess) e = hipEventRecord(a, s);
  for (int i = 0; i < reps && e == hipSuccess; ++i)
    e = wici::launch_stream_read(d_buf, bytes, grid, sink, s);
  if (e == hipSuccess) e = hipEventRecord(b, s);
  if (e == hipSuccess && checksum) {
    const size_t n = (size_t)256 * grid;
    e = wici::launch_xor_reduce(sink, (int)n, sink + n, s);
    if (e == hipSuccess) e = hipMemcpyAsync(checksum, sink + n, 4, hipMemcpyDeviceToHost, s);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (e != hipSuccess) return WICI_E_HIP;
  *ms_per_read = ms / reps;
  return WICI_OK;
}

wici_status wici_position(const wici_model* m, int32_t* pos) {
  if (!m || !pos) return WICI_E_ARG;
  *pos = m->pos;
  return WICI_OK;
}

wici_status wici_read_kv(wici_model* m, int32_t layer, int32_t begin, int32_t end, void* host_k,
                         void* host_v) {
  if (!m) return WICI_E_ARG;
  if (m->failed) return WICI_E_STATE;
  if (!m->bound) return fail(m, WICI_E_STATE, "memory not bound");
  const wici_config& c = m->cfg;
  if (layer < 0 || layer >= c.n_layers || begin < 0 || end < begin || end > m->pos || !host_k ||
      !host_v)
    return fail(m, WICI_E_ARG, "bad layer/range/pointer");
  const size_t es = dsize(c.kv_dtype), hd = c.head_dim, page = c.kv_page, nkv = c.n_kv_heads;
  std::vector<int32_t> table(m->L.n_pages);
  HIP_TRY(m, hipMemcpyAsync(table.data(), m->ds + m->L.table, table.size() * 4,
                            hipMemcpyDeviceToHost, m->stream));
  HIP_TRY(m, hipStreamSynchronize(m->stream));
  const char* base = m->dkv + (size_t)layer * m->L.kv_layer_stride;
  for (int p = begin; p < end; ++p) {
    const size_t phys = table[p / page], slot = p % page;
    for (int w = 0; w < 2; ++w) {
      const char* src = base + (((phys * 2 + w) * nkv) * page + slot) * hd * es;
      char* dst = static_cast<char*>(w ? host_v : host_k) + (size_t)(p - begin) * nkv * hd * es;
      HIP_TRY(m, hipMemcpy2DAsync(dst, hd * es, src, page * hd * es, hd * es, nkv,
                                  hipMemcpyDeviceToHost, m->stream));
    }
  }
  HIP_TRY(m, hipStreamSynchronize(m->stream));
  return WICI_OK;
}

const char* wici_last_error(const wici_model* m) { return m ? m->err.c_str() : "NULL model"; }

void wici_destroy(wici_model* m) {
  if (!m) return;
  if (m->gexec) (void)hipGraphExecDestroy(m->gexec);
  if (m->graph) (void)hipGraphDestroy(m->graph);
  for (auto& kv : m->batch_graphs) {
    (void)hipGraphExecDestroy(kv.second.second);
    (void)hipGraphDestroy(kv.second.first);
  }
  if (m->h_state) (void)hipHostFree(m->h_state);
  delete m;
}

}  // extern "C"
