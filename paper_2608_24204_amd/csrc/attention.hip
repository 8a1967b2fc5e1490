// Causal grouped-query attention over the paged KV cache.
//
// Decode (one query position per head): split-K over the context.  A block loads
// each cached key/value of its range once and serves all query heads of the KV
// head's group with it (GQA), so every cached byte is read once per step.  The
// new position's k/v are rotated, rounded to the storage type, written to the
// cache and used straight from LDS (no block reads a position another block of
// the same launch writes).  The splits are merged by a second small kernel, or,
// for a bf16 cache with few splits, by the last split block of each head in the
// same launch (through the L2 of the XCD all of that head's blocks run on).
//
// Prefill: one block per (64 queries, query head), keys streamed through LDS in
// blocks of 64 with an online softmax; on the matrix cores for a bf16 cache (the
// fp32 query and probabilities split into bf16 terms), else fp32 vector code.
#include <type_traits>

#include "attn_decode.h"
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wici {

constexpr int kMaxGroup = 8;   // query heads per KV head

__device__ __forceinline__ size_t kv_off(const KvLayout& kv, int pos, int which, int h) {
  const int ps = __ffs(kv.page) - 1;  // pages are a power of two
  const int phys = kv.table[pos >> ps], slot = pos & (kv.page - 1);
  return ((((size_t)phys * 2 + which) * kv.n_kv + h) * kv.page + slot) * (size_t)kv.hd;
}

// ------------------------------------------------------------------- decode
// Grid (nsplit, Hkv): block (s, g) owns positions [64 s, 64 s + 64) of KV head g;
// blocks past the current context exit at once, so one captured launch serves
// every position.  The queries arrive rotated and pre-scaled, and the new
// position's key and value are already in the cache (both done by the QKV
// projection's epilogue), so a block's loads depend only on its page-table
// entries and on the position, which arrive together: every slot of the chunk
// is then requested at once (slots past the context are loaded and ignored).
// Each block writes its unnormalised output and (max, sum) statistics; a second
// kernel merges the splits.  (Merging in the last block of each head through
// device-scope fences, whose L2 write-back and invalidate fall on every block,
// measured slower than the extra launch; the matrix-core kernel merges in the
// last block only through one XCD's L2, see attn_merge_in_last_split.)
constexpr int kMaxSplits = 256;  // splits the merge kernel holds in LDS

// With seqs != nullptr the launch is batched: blockIdx.z is the sequence, whose
// KV pool, page table and position come from seqs[z] (layer `layer`), whose
// queries start at q_in + z * q_stride and whose partials follow the previous
// sequence's.
template <int HD, typename KT, int G>
__global__ __launch_bounds__(256) void k_attn_decode(const float* __restrict__ q_in,
                                                     KvLayout kv,
                                                     const DecodeState* __restrict__ st,
                                                     float* __restrict__ part_o,
                                                     float* __restrict__ part_ml,
                                                     const SeqDesc* __restrict__ seqs, int layer,
                                                     int q_stride) {
  if (seqs) {
    const SeqDesc sd = seqs[blockIdx.z];
    kv.base = static_cast<char*>(sd.kv) + (size_t)layer * sd.kv_layer_stride;
    kv.table = sd.table;
    st = static_cast<const DecodeState*>(sd.state);
    q_in += (size_t)blockIdx.z * q_stride;
    const size_t heads = (size_t)kv.n_kv * G * gridDim.x;
    part_o += (size_t)blockIdx.z * heads * HD;
    part_ml += (size_t)blockIdx.z * heads * 2;
  }
  constexpr int LPP = HD / 8;       // lanes per position (8 elements each)
  constexpr int PPW = 64 / LPP;     // positions per wave per pass
  constexpr int PPB = 4 * PPW;      // positions per block per pass
  constexpr int NP = kChunk / PPB;  // passes over the chunk
  __shared__ float qs[G][HD];
  __shared__ float sc[G][kChunk];
  __shared__ float accs[4][G][HD];
  __shared__ float mls[G][2];

  const int nsplit = gridDim.x;
  const int split = blockIdx.x, g = blockIdx.y;
  const int Hkv = kv.n_kv;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int pg = lane / LPP, sub = lane % LPP;
  const int start = split * kChunk;
  const KT* base = static_cast<const KT*>(kv.base);
  const size_t head_stride = (size_t)kv.page * HD;
  const int ps = __ffs(kv.page) - 1;  // pages are a power of two
  // page of each of this lane's positions (clamped into the table)
  int phys[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int j = start + i * PPB + wave * PPW + pg;
    phys[i] = kv.table[min(j, kv.max_pos - 1) >> ps];
  }
  // queries of the group (independent of the position)
  float qv[(G * HD + 255) / 256];
#pragma unroll
  for (int k = 0; k < (G * HD + 255) / 256; ++k)
    qv[k] = q_in[(size_t)g * G * HD + min(tid + k * 256, G * HD - 1)];
  // the position (a scalar load, back as soon as the table entries): blocks past
  // the context stop before requesting anything more
  const int pos = st->pos, n = pos + 1;
  if (start >= n) return;
  const int end = min(n, start + kChunk);
  // every slot of the chunk: keys and values
  float kr[NP][8], vr[NP][8];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int j = start + i * PPB + wave * PPW + pg;
    const KT* pk = base + (((size_t)phys[i] * 2 + 0) * Hkv + g) * head_stride +
                   (size_t)(j & (kv.page - 1)) * HD + sub * 8;
    load8(pk, kr[i]);
    load8(pk + (size_t)Hkv * head_stride, vr[i]);
  }
#pragma unroll
  for (int k = 0; k < (G * HD + 255) / 256; ++k)
    if (tid + k * 256 < G * HD) (&qs[0][0])[tid + k * 256] = qv[k];
  __syncthreads();

  // ---- scores ------------------------------------------------------------------------
  float q[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float4 a = *reinterpret_cast<const float4*>(&qs[h][sub * 8]);
    const float4 b = *reinterpret_cast<const float4*>(&qs[h][sub * 8 + 4]);
    q[h][0] = a.x; q[h][1] = a.y; q[h][2] = a.z; q[h][3] = a.w;
    q[h][4] = b.x; q[h][5] = b.y; q[h][6] = b.z; q[h][7] = b.w;
  }
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int j = start + i * PPB + wave * PPW + pg;
    if (j >= end) {  // past the context: whatever the slot holds is not used
#pragma unroll
      for (int e = 0; e < 8; ++e) { kr[i][e] = 0.f; vr[i][e] = 0.f; }
    }
    float s[G];
#pragma unroll
    for (int h = 0; h < G; ++h) {
      s[h] = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) s[h] += q[h][e] * kr[i][e];
    }
#pragma unroll
    for (int h = 0; h < G; ++h) s[h] = group_sum<LPP>(s[h]);
    if (sub == 0 && j < end) {
#pragma unroll
      for (int h = 0; h < G; ++h) sc[h][j - start] = s[h];
    }
  }
  __syncthreads();

  // ---- softmax statistics (one wave per head) ----------------------------------------
  const int len = end - start;
#pragma unroll
  for (int h0 = 0; h0 < G; h0 += 4) {
    const int h = h0 + wave;
    if (h < G) {
      const float v = lane < len ? sc[h][lane] : -INFINITY;
      const float m = wave_max(v);
      const float p = lane < len ? __expf(v - m) : 0.f;
      if (lane < len) sc[h][lane] = p;
      const float l = wave_sum(p);
      if (lane == 0) { mls[h][0] = m; mls[h][1] = l; }
    }
  }
  __syncthreads();

  // ---- weighted values -----------------------------------------------------------------
  float acc[G][8];
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int j = start + i * PPB + wave * PPW + pg;
    const int jj = j < end ? j - start : 0;
    const bool ok = j < end;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float p = ok ? sc[h][jj] : 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[h][e] += p * vr[i][e];
    }
  }
  // sum the positions held by the wave's rows (lanes 16 or 32 apart share a slice)
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float a = acc[h][e];
#pragma unroll
      for (int m = LPP; m < 64; m <<= 1) a += __shfl_xor(a, m);
      acc[h][e] = a;
    }
  if (pg == 0) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      *reinterpret_cast<float4*>(&accs[wave][h][sub * 8]) =
          make_float4(acc[h][0], acc[h][1], acc[h][2], acc[h][3]);
      *reinterpret_cast<float4*>(&accs[wave][h][sub * 8 + 4]) =
          make_float4(acc[h][4], acc[h][5], acc[h][6], acc[h][7]);
    }
  }
  __syncthreads();
  for (int i = tid; i < G * HD; i += 256) {
    const int hl = i / HD, d = i % HD, h = g * G + hl;
    part_o[((size_t)h * nsplit + split) * HD + d] =
        accs[0][hl][d] + accs[1][hl][d] + accs[2][hl][d] + accs[3][hl][d];
  }
  if (tid < G) {
    const int h = g * G + tid;
    part_ml[((size_t)h * nsplit + split) * 2 + 0] = mls[tid][0];
    part_ml[((size_t)h * nsplit + split) * 2 + 1] = mls[tid][1];
  }
}

// The same split (64 positions of one KV head, all G query heads) on the matrix
// cores, for a bf16 cache.  Wavefront w takes positions 16 w .. 16 w + 15 of the
// split.  S^T = K Q^T on v_mfma_f32_16x16x32_bf16: lane l's 16 bytes of keys
// (position l % 16, dimensions 8 (l / 16) + 32 s) are exactly its A operand, the
// query heads are the 16 columns (zero past G) and the fp32 query enters as
// three bf16 terms accumulated into the same tile, so the scores keep fp32
// precision.  The result leaves lane l with 4 positions of head l % 16, which is
// the A-operand order of P V on v_mfma_f32_16x16x16_bf16 (the probabilities
// again as three bf16 terms); the values go through LDS transposed to
// [dimension][position] for the B operand.  Each wavefront keeps its own
// (max, sum) per head; one barrier, then the four are combined and the split's
// unnormalised output and statistics written as by k_attn_decode.  Up to G = 5
// the registers are held to 96 per lane, so five workgroups share a CU (the LDS
// allows five): a long context's grid (8 KV heads x 129 splits at 8.2K
// positions) then fits the chip in one round instead of leaving a tail.
template <int HD, int G, bool FUSE, bool ROPE = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(G <= 5 && !FUSE ? (ROPE ? 4 : 5) : 1))) void
k_attn_decode_mfma(const float* __restrict__ q_in,
                   KvLayout kv,
                   const DecodeState* __restrict__ st,
                   float* __restrict__ part_o,
                   float* __restrict__ part_ml,
                   const SeqDesc* __restrict__ seqs,
                   int layer,
                   int q_stride,
                   AttnFuse fz,
                   RopeIn rope) {
  static_assert(G <= 16, "query heads are the 16 columns of a tile");
  static_assert(!FUSE || G * HD <= 512, "the merge holds at most 16 partials per thread");
  if (seqs) {
    const SeqDesc sd = seqs[blockIdx.z];
    kv.base = static_cast<char*>(sd.kv) + (size_t)layer * sd.kv_layer_stride;
    kv.table = sd.table;
    st = static_cast<const DecodeState*>(sd.state);
    q_in += (size_t)blockIdx.z * q_stride;
    const size_t heads = (size_t)kv.n_kv * G * gridDim.x;
    part_o += (size_t)blockIdx.z * heads * HD;
    part_ml += (size_t)blockIdx.z * heads * 2;
  }
  const int Hkv = kv.n_kv;
  int nsplit, split, g;
  if constexpr (FUSE) {
    // 1-D grid dealt to the XCDs in turn, starting wherever the previous launch
    // left off (measured: after a one-workgroup launch the next grid's block 0
    // is not on XCD 0), so blocks with equal b % 8 share an XCD; every split of
    // KV head g is placed in class g % 8 (blocks of absent heads exit)
    const int b = blockIdx.x, x = b & 7, r = b >> 3, h8 = (Hkv + 7) >> 3;
    g = x + 8 * (r % h8);
    split = r / h8;
    nsplit = fz.nsplit;
    if (g >= Hkv) return;
  } else {
    nsplit = gridDim.x;
    split = blockIdx.x;
    g = blockIdx.y;
  }
  const int n = attn_split_mfma<HD, G, ROPE>(q_in, kv, st, part_o, part_ml, g, split, nsplit, rope);
  if constexpr (FUSE)
    if (n > 0) attn_merge_in_last_split<HD, G>(fz, g, split, nsplit, n, part_o, part_ml);
}

// Long contexts (more 64-position splits than the merge in the last split block
// takes): the same launch with each block walking `span` consecutive sub-chunks
// (attn_span_mfma, four teams of four wavefronts), so that the splits of a head
// are at most kFuseMaxSplits, and the merge in the last of them.  Block
// placement as k_attn_decode_mfma's FUSE.
constexpr int kSpanTeams = 4;  // workgroups of 4 x 4 wavefronts
template <int HD, int G>
__global__ __launch_bounds__(256 * kSpanTeams) void k_attn_decode_span(const float* __restrict__ q_in,
                                                          KvLayout kv,
                                                          const DecodeState* __restrict__ st,
                                                          float* __restrict__ part_o,
                                                          float* __restrict__ part_ml,
                                                          AttnFuse fz, int span) {
  static_assert(G <= 16 && G * HD <= 512, "as the merge in the last split block");
  const int Hkv = kv.n_kv;
  const int b = blockIdx.x, x = b & 7, r = b >> 3, h8 = (Hkv + 7) >> 3;
  const int g = x + 8 * (r % h8), split = r / h8, nsplit = fz.nsplit;
  if (g >= Hkv) return;
  const int n =
      attn_span_mfma<HD, G, kSpanTeams>(q_in, kv, st, part_o, part_ml, g, split, nsplit, span);
  if (n > 0) attn_merge_in_last_split<HD, G>(fz, g, split, nsplit, n, part_o, part_ml, span);
}

// out[h, d] = sum_s e^(m_s - M) o_s[d] / sum_s e^(m_s - M) l_s over the active
// splits s of head h, for launches of at most kMergePf splits (grid Hq, HD
// threads).  The position, the first 64 splits' statistics and the thread's
// column of every split are requested at once (clamped into the split range), so
// the merge costs one memory round trip; each wavefront reduces the statistics
// itself (no barrier before the weights exist).
constexpr int kMergePf = 32;
template <int HD>
__global__ __launch_bounds__(HD) void k_attn_merge_head(const float* __restrict__ part_o,
                                                        const float* __restrict__ part_ml,
                                                        int nsplit,
                                                        const DecodeState* __restrict__ st,
                                                        float* __restrict__ out) {
  __shared__ float w[kMaxSplits];
  const int h = blockIdx.x, d = threadIdx.x, lane = d & 63, wv = d >> 6;
  const float* ml = part_ml + (size_t)h * nsplit * 2;
  const float* po = part_o + (size_t)h * nsplit * HD + d;
  const int pos = st->pos;
  const float2 s0 = reinterpret_cast<const float2*>(ml)[min(lane, nsplit - 1)];
  float pv[kMergePf];
#pragma unroll
  for (int k = 0; k < kMergePf; ++k) pv[k] = po[(size_t)min(k, nsplit - 1) * HD];
  const int active = min((pos + kChunk) / kChunk, nsplit);  // ceil((pos + 1) / chunk)
  float mloc = lane < active ? s0.x : -INFINITY;
  for (int s = lane + 64; s < active; s += 64) mloc = fmaxf(mloc, ml[2 * s]);
  const float M = wave_max(mloc);
  float lsum = 0.f;
  if (lane < active) {
    const float e = __expf(s0.x - M);
    lsum = e * s0.y;
    if (wv == 0) w[lane] = e;
  }
  for (int s = lane + 64; s < active; s += 64) {
    const float e = __expf(ml[2 * s] - M);
    lsum += e * ml[2 * s + 1];
    if (wv == 0) w[s] = e;
  }
  const float L = wave_sum(lsum);
  __syncthreads();
  float o = 0.f;
#pragma unroll
  for (int k = 0; k < kMergePf; ++k)
    if (k < active) o += w[k] * pv[k];
  for (int s = kMergePf; s < active; ++s) o += w[s] * po[(size_t)s * HD];
  out[(size_t)h * HD + d] = o / L;
}

// The same merge for launches of more than kMergePf splits.  Workgroup (h, c)
// merges columns 32 c .. 32 c + 31 (grid Hq x HD/32, 256 threads): thread t
// takes column t % 32 of splits t / 32, t / 32 + 8, ...  Every partial below the
// launch's split count and every split's statistics are requested before the
// position is known (addresses clamped into the split range), so a context of
// up to kMaxSplits splits costs one memory round trip and the splits' reads are
// spread over Hq * HD/32 workgroups.  Each wavefront reduces the statistics itself; slots of inactive
// splits are skipped, not weighted by zero (they may hold anything).
constexpr int kMergeRows = 8;                     // split rows of a workgroup
constexpr int kMergeK = kMaxSplits / kMergeRows;  // partials per thread
template <int HD>
__global__ __launch_bounds__(256) void k_attn_merge_cols(const float* __restrict__ part_o,
                                                         const float* __restrict__ part_ml,
                                                         int nsplit,
                                                         const DecodeState* __restrict__ st,
                                                         float* __restrict__ out) {
  static_assert(HD % 32 == 0, "32-column slices");
  __shared__ float w[kMaxSplits];
  __shared__ float red[4][32];
  const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int c = tid & 31, r = tid >> 5;
  const int col = 32 * blockIdx.y + c;
  const float* ml = part_ml + (size_t)h * nsplit * 2;
  const float* po = part_o + (size_t)h * nsplit * HD + col;
  const int pos = st->pos;
  float2 sm[kMaxSplits / 64];
#pragma unroll
  for (int i = 0; i < kMaxSplits / 64; ++i)
    if (64 * i < nsplit) sm[i] = reinterpret_cast<const float2*>(ml)[min(lane + 64 * i, nsplit - 1)];
  float pv[kMergeK];
#pragma unroll
  for (int k = 0; k < kMergeK; ++k)
    if (kMergeRows * k < nsplit) pv[k] = po[(size_t)min(r + kMergeRows * k, nsplit - 1) * HD];
  const int active = min((pos + kChunk) / kChunk, nsplit);  // ceil((pos + 1) / chunk)
  float mloc = -INFINITY;
#pragma unroll
  for (int i = 0; i < kMaxSplits / 64; ++i)
    if (64 * i < nsplit && lane + 64 * i < active) mloc = fmaxf(mloc, sm[i].x);
  const float M = wave_max(mloc);
  float lsum = 0.f;
#pragma unroll
  for (int i = 0; i < kMaxSplits / 64; ++i) {
    const int s = lane + 64 * i;
    if (64 * i < nsplit && s < active) {
      const float e = __expf(sm[i].x - M);
      lsum += e * sm[i].y;
      if (wv == 0) w[s] = e;
    }
  }
  const float L = wave_sum(lsum);
  __syncthreads();
  float o = 0.f;
#pragma unroll
  for (int k = 0; k < kMergeK; ++k) {
    const int s = r + kMergeRows * k;
    if (kMergeRows * k < nsplit && s < active) o += w[s] * pv[k];
  }
  o += __shfl_xor(o, 32);
  if (lane < 32) red[wv][c] = o;
  __syncthreads();
  if (tid < 32) out[(size_t)h * HD + col] = (red[0][c] + red[1][c] + red[2][c] + red[3][c]) / L;
}

// Batched merge: block (h, b) merges head h of sequence b into the activation
// buffer of the O projection (row b).
template <int HD>
__global__ __launch_bounds__(HD) void k_attn_merge_batch(const float* __restrict__ part_o,
                                                         const float* __restrict__ part_ml,
                                                         int nsplit,
                                                         const SeqDesc* __restrict__ seqs,
                                                         ActBuf out) {
  __shared__ float w[kMaxSplits];
  __shared__ float red[HD / 64];
  const int h = blockIdx.x, b = blockIdx.y, Hq = gridDim.x;
  const int d = threadIdx.x, lane = d & 63, wv = d >> 6;
  const size_t head = (size_t)b * Hq + h;
  const float* ml = part_ml + head * nsplit * 2;
  const float* po = part_o + head * nsplit * HD + d;
  // Up to 32 splits this thread's column of every split is requested with the
  // position, before the split count is known (clamped; the unused ones are
  // dropped), so the merge is one memory round trip; the arithmetic and its
  // order are the loop form's below.
  constexpr int PS = 32;
  if (nsplit <= PS && HD >= PS) {
    float pv[PS];
#pragma unroll
    for (int s = 0; s < PS; ++s) pv[s] = po[(size_t)min(s, nsplit - 1) * HD];
    const float2 mlv = *reinterpret_cast<const float2*>(ml + 2 * min(d, nsplit - 1));
    const int pos = static_cast<const DecodeState*>(seqs[b].state)->pos;
    const int active = (pos + kChunk) / kChunk;
    float mloc = d < active ? mlv.x : -INFINITY;
    mloc = wave_max(mloc);
    if (lane == 0) red[wv] = mloc;
    __syncthreads();
    float M = red[0];
#pragma unroll
    for (int i = 1; i < HD / 64; ++i) M = fmaxf(M, red[i]);
    float lsum = 0.f;
    if (d < active) {
      const float e = __expf(mlv.x - M);
      w[d] = e;
      lsum += e * mlv.y;
    }
    lsum = wave_sum(lsum);
    __syncthreads();
    if (lane == 0) red[wv] = lsum;
    __syncthreads();
    float L = 0.f;
#pragma unroll
    for (int i = 0; i < HD / 64; ++i) L += red[i];
    float o = 0.f;
#pragma unroll
    for (int s = 0; s < PS; ++s)
      if (s < active) o += w[s] * pv[s];
    store_act(out, ((size_t)b * Hq + h) * HD + d, o / L);
    return;
  }
  const int pos = static_cast<const DecodeState*>(seqs[b].state)->pos;
  const int active = (pos + kChunk) / kChunk;
  float mloc = -INFINITY;
  for (int s = d; s < active; s += HD) mloc = fmaxf(mloc, ml[2 * s]);
  mloc = wave_max(mloc);
  if (lane == 0) red[wv] = mloc;
  __syncthreads();
  float M = red[0];
#pragma unroll
  for (int i = 1; i < HD / 64; ++i) M = fmaxf(M, red[i]);
  float lsum = 0.f;
  for (int s = d; s < active; s += HD) {
    const float e = __expf(ml[2 * s] - M);
    w[s] = e;
    lsum += e * ml[2 * s + 1];
  }
  lsum = wave_sum(lsum);
  __syncthreads();
  if (lane == 0) red[wv] = lsum;
  __syncthreads();
  float L = 0.f;
#pragma unroll
  for (int i = 0; i < HD / 64; ++i) L += red[i];
  float o = 0.f;
  for (int s = 0; s < active; ++s) o += w[s] * po[(size_t)s * HD];
  store_act(out, ((size_t)b * Hq + h) * HD + d, o / L);
}

template <int HD, typename KT, int G>
static hipError_t attn_decode_t(const float* q, int Hq, KvLayout kv, const DecodeState* st,
                                int nsplit, float* part_o, float* part_ml, float* out,
                                const AttnFuse* fuse, hipStream_t s) {
  if constexpr (sizeof(KT) == 2 && G * HD <= 512) {
    // the merge in the last split block (one launch) when the splits fit it
    if (fuse && nsplit <= kFuseMaxSplits) {
      AttnFuse fz = *fuse;
      fz.out = out;
      fz.nsplit = nsplit;
      fz.n_heads = Hq;
      fz.n_kv = kv.n_kv;
      const int blocks = 8 * ((kv.n_kv + 7) / 8) * nsplit;
      launch_k(k_attn_decode_mfma<HD, G, true>, dim3(blocks), dim3(256), 0, s, kOnly, q, kv, st,
               part_o, part_ml, (const SeqDesc*)nullptr, 0, 0, fz, RopeIn{});
      return hipGetLastError();
    }
    // longer: splits of several sub-chunks, as few as keep them within the merge
    // (8.2K positions: 26 splits of 5 sub-chunks instead of 130 splits and a
    // merge kernel)
    const int span = (nsplit + kFuseMaxSplits - 1) / kFuseMaxSplits;
    if (fuse && span <= kMaxSpan) {
      AttnFuse fz = *fuse;
      fz.out = out;
      fz.nsplit = (nsplit + span - 1) / span;
      fz.n_heads = Hq;
      fz.n_kv = kv.n_kv;
      const int blocks = 8 * ((kv.n_kv + 7) / 8) * fz.nsplit;
      launch_k(k_attn_decode_span<HD, G>, dim3(blocks), dim3(256 * kSpanTeams), 0, s, kOnly, q,
               kv, st, part_o, part_ml, fz, span);
      return hipGetLastError();
    }
  }
  if constexpr (sizeof(KT) == 2)
    launch_k(k_attn_decode_mfma<HD, G, false>, dim3(nsplit, kv.n_kv), dim3(256), 0, s, kFirst, q,
             kv, st, part_o, part_ml, (const SeqDesc*)nullptr, 0, 0, AttnFuse{}, RopeIn{});
  else
    launch_k(k_attn_decode<HD, KT, G>, dim3(nsplit, kv.n_kv), dim3(256), 0, s, kFirst, q, kv,
             st, part_o, part_ml, (const SeqDesc*)nullptr, 0, 0);
  if (nsplit <= kMergePf)
    launch_k(k_attn_merge_head<HD>, dim3(Hq), dim3(HD), 0, s, kLast, part_o, part_ml, nsplit, st,
             out);
  else
    launch_k(k_attn_merge_cols<HD>, dim3(Hq, HD / 32), dim3(256), 0, s, kLast, part_o, part_ml,
             nsplit, st, out);
  return hipGetLastError();
}

template <int HD, typename KT, int G>
static hipError_t attn_decode_batch_t(const float* q, int q_stride, int B, int Hq, KvLayout kv,
                                      const SeqDesc* seqs, int layer, int nsplit, float* part_o,
                                      float* part_ml, const ActBuf& out, hipStream_t s,
                                      const RopeIn* rope) {
  if (rope && sizeof(KT) != 2) return hipErrorInvalidValue;
  if constexpr (sizeof(KT) == 2) {
    if (rope)
      hipLaunchKernelGGL((k_attn_decode_mfma<HD, G, false, true>), dim3(nsplit, kv.n_kv, B),
                         dim3(256), 0, s, q, kv, (const DecodeState*)nullptr, part_o, part_ml,
                         seqs, layer, q_stride, AttnFuse{}, *rope);
    else
      hipLaunchKernelGGL((k_attn_decode_mfma<HD, G, false>), dim3(nsplit, kv.n_kv, B), dim3(256),
                         0, s, q, kv, (const DecodeState*)nullptr, part_o, part_ml, seqs, layer,
                         q_stride, AttnFuse{}, RopeIn{});
  } else
    hipLaunchKernelGGL((k_attn_decode<HD, KT, G>), dim3(nsplit, kv.n_kv, B), dim3(256), 0, s, q,
                       kv, (const DecodeState*)nullptr, part_o, part_ml, seqs, layer, q_stride);
  hipLaunchKernelGGL((k_attn_merge_batch<HD>), dim3(Hq, B), dim3(HD), 0, s, part_o, part_ml,
                     nsplit, seqs, out);
  return hipGetLastError();
}

template <int HD, typename KT>
static hipError_t attn_decode_g(int G, const float* q, int Hq, KvLayout kv,
                                const DecodeState* st, int nsplit, float* part_o,
                                float* part_ml, float* out, const AttnFuse* fz, hipStream_t s) {
  switch (G) {
    case 1: return attn_decode_t<HD, KT, 1>(q, Hq, kv, st, nsplit, part_o, part_ml, out, fz, s);
    case 2: return attn_decode_t<HD, KT, 2>(q, Hq, kv, st, nsplit, part_o, part_ml, out, fz, s);
    case 4: return attn_decode_t<HD, KT, 4>(q, Hq, kv, st, nsplit, part_o, part_ml, out, fz, s);
    case 5: return attn_decode_t<HD, KT, 5>(q, Hq, kv, st, nsplit, part_o, part_ml, out, fz, s);
    case 8: return attn_decode_t<HD, KT, 8>(q, Hq, kv, st, nsplit, part_o, part_ml, out, fz, s);
    default: return hipErrorInvalidValue;
  }
}

template <int HD, typename KT>
static hipError_t attn_decode_batch_g(int G, const float* q, int q_stride, int B, int Hq,
                                      KvLayout kv, const SeqDesc* seqs, int layer, int nsplit,
                                      float* part_o, float* part_ml, const ActBuf& out,
                                      hipStream_t s, const RopeIn* rope) {
#define WICI_B(GG) \
  case GG: return attn_decode_batch_t<HD, KT, GG>(q, q_stride, B, Hq, kv, seqs, layer, nsplit, part_o, part_ml, out, s, rope)
  switch (G) {
    WICI_B(1); WICI_B(2); WICI_B(4); WICI_B(5); WICI_B(8);
    default: return hipErrorInvalidValue;
  }
#undef WICI_B
}

hipError_t launch_attn_decode_batch(bool kv_bf16, const float* q, int q_stride, int B, int Hq,
                                    KvLayout kv, const SeqDesc* seqs, int layer, int nsplit,
                                    float* part_o, float* part_ml, const ActBuf& out,
                                    hipStream_t s, const RopeIn* rope) {
  if (B < 1 || nsplit > kMaxSplits || nsplit * kChunk < kv.max_pos || kv.n_kv < 1 ||
      Hq % kv.n_kv || kv.page < 1 || (kv.page & (kv.page - 1)))
    return hipErrorInvalidValue;
  const int G = Hq / kv.n_kv;
  if (kv.hd == 128) {
    if (kv_bf16) return attn_decode_batch_g<128, bf16_t>(G, q, q_stride, B, Hq, kv, seqs, layer, nsplit, part_o, part_ml, out, s, rope);
    return attn_decode_batch_g<128, float>(G, q, q_stride, B, Hq, kv, seqs, layer, nsplit, part_o, part_ml, out, s, rope);
  }
  if (kv.hd == 64) {
    if (kv_bf16) return attn_decode_batch_g<64, bf16_t>(G, q, q_stride, B, Hq, kv, seqs, layer, nsplit, part_o, part_ml, out, s, rope);
    return attn_decode_batch_g<64, float>(G, q, q_stride, B, Hq, kv, seqs, layer, nsplit, part_o, part_ml, out, s, rope);
  }
  return hipErrorInvalidValue;
}

int attn_decode_splits(int max_seq) { return (max_seq + kChunk - 1) / kChunk; }
bool attn_group_supported(int G) { return G == 1 || G == 2 || G == 4 || G == 5 || G == 8; }

hipError_t launch_attn_decode(bool kv_bf16, const float* q, int Hq, KvLayout kv,
                              const void* state, int nsplit, float* part_o, float* part_ml,
                              float* out, const AttnFuse* fuse, hipStream_t s) {
  if (nsplit > kMaxSplits || nsplit * kChunk < kv.max_pos || kv.n_kv < 1 || Hq % kv.n_kv ||
      kv.page < 1 || (kv.page & (kv.page - 1)))
    return hipErrorInvalidValue;
  if (fuse && (!fuse->cnt || !fuse->xcc || !fuse->state)) return hipErrorInvalidValue;
  const DecodeState* st = static_cast<const DecodeState*>(state);
  const int G = Hq / kv.n_kv;
  if (kv.hd == 128) {
    if (kv_bf16) return attn_decode_g<128, bf16_t>(G, q, Hq, kv, st, nsplit, part_o, part_ml, out, fuse, s);
    return attn_decode_g<128, float>(G, q, Hq, kv, st, nsplit, part_o, part_ml, out, fuse, s);
  }
  if (kv.hd == 64) {
    if (kv_bf16) return attn_decode_g<64, bf16_t>(G, q, Hq, kv, st, nsplit, part_o, part_ml, out, fuse, s);
    return attn_decode_g<64, float>(G, q, Hq, kv, st, nsplit, part_o, part_ml, out, fuse, s);
  }
  return hipErrorInvalidValue;
}

int attn_fuse_ints(int n_kv) { return 2 * n_kv * kFuseLine; }

// ------------------------------------------------------------------- prefill
template <int HD, typename KT>
__global__ __launch_bounds__(256) void k_attn_prefill(const float* __restrict__ qkv, int T,
                                                      int p0, int Hq, KvLayout kv, ActBuf out,
                                                      int cus) {
  constexpr int BQ = 64, BKEY = 64, DPT = HD / 4;
  __shared__ float Ks[BKEY][HD + 4];
  __shared__ float Vs[BKEY][HD + 4];
  // the grid is dealt out in order, one workgroup per CU and then a second, so
  // workgroups b and b + (CUs) share a CU, and the causal walk of query block i
  // is i + 1 key blocks: alternate runs of heads, each run as many heads as
  // (CUs) workgroups hold, take their query blocks in reverse order, pairing
  // long walks with short ones on every CU (the order is a function of the head
  // alone, so every (head, query block) is taken exactly once)
  const int h = blockIdx.y, run = max(1, cus / (int)gridDim.x);
  const int qbi = (h / run) & 1 ? gridDim.x - 1 - blockIdx.x : blockIdx.x;
  const int qb = qbi * BQ;
  const int Hkv = kv.n_kv, g = h / (Hq / Hkv);
  const int tid = threadIdx.x, ql = tid >> 2, part = tid & 3;
  const int t = qb + ql;
  const bool valid = t < T;
  const int qpos = p0 + t;
  const int width = (Hq + 2 * Hkv) * HD;
  const float scale = 1.0f / sqrtf((float)HD);
  const KT* base = static_cast<const KT*>(kv.base);

  float q[DPT], acc[DPT];
  const float* qrow = qkv + (size_t)(valid ? t : 0) * width + (size_t)h * HD + part * DPT;
#pragma unroll
  for (int e = 0; e < DPT; ++e) { q[e] = qrow[e] * scale; acc[e] = 0.f; }
  float m = -INFINITY, l = 0.f;
  const int kend = p0 + min(T, qb + BQ);

  for (int kb = 0; kb < kend; kb += BKEY) {
    __syncthreads();
    for (int idx = tid; idx < BKEY * (HD / 8); idx += 256) {
      const int jj = idx / (HD / 8), c = (idx % (HD / 8)) * 8, j = kb + jj;
      float kk[8], vv[8];
      if (j < kend) {
        load8(base + kv_off(kv, j, 0, g) + c, kk);
        load8(base + kv_off(kv, j, 1, g) + c, vv);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) { kk[e] = 0.f; vv[e] = 0.f; }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) { Ks[jj][c + e] = kk[e]; Vs[jj][c + e] = vv[e]; }
    }
    __syncthreads();
    float s[BKEY];
    float bm = -INFINITY;
#pragma unroll
    for (int jj = 0; jj < BKEY; ++jj) {
      float d = 0.f;
#pragma unroll
      for (int e = 0; e < DPT; ++e) d += q[e] * Ks[jj][part * DPT + e];
      d += __shfl_xor(d, 1);
      d += __shfl_xor(d, 2);
      const int j = kb + jj;
      s[jj] = (j <= qpos && j < kend) ? d : -INFINITY;
      bm = fmaxf(bm, s[jj]);
    }
    const float mn = fmaxf(m, bm);
    if (mn == -INFINITY) continue;  // no visible key yet (cannot happen for key 0)
    const float corr = expf(m - mn);
    l *= corr;
#pragma unroll
    for (int e = 0; e < DPT; ++e) acc[e] *= corr;
#pragma unroll
    for (int jj = 0; jj < BKEY; ++jj) {
      const float p = expf(s[jj] - mn);
      l += p;
#pragma unroll
      for (int e = 0; e < DPT; ++e) acc[e] += p * Vs[jj][part * DPT + e];
    }
    m = mn;
  }
  if (valid) {
    const size_t o = (size_t)t * Hq * HD + (size_t)h * HD + part * DPT;
    const float inv = 1.0f / l;
#pragma unroll
    for (int e = 0; e < DPT; ++e) store_act(out, o + e, acc[e] * inv);
  }
}

// ------------------------------------------------------------- prefill, MFMA
// Flash attention on the matrix cores.  Block = 4 wavefronts = 64 query rows of
// one query head (16 per wavefront); keys stream through LDS in blocks of 64
// (K as [key][d], V transposed to [d][key]), the next two blocks' loads in
// flight while the current one is processed.  Per key block a wavefront computes
// S^T = K Q^T (so each lane ends up with 16 keys of one query, the row layout the
// A operand of the next product needs), the online-softmax update, and
// O += P V.  The query and the probabilities are fp32 values split into NT bf16
// terms (K and V are stored in bf16, hence exact), so both products keep the
// precision of their fp32 operands.
template <int HD, int NT>
__global__ __launch_bounds__(256) void k_attn_prefill_mfma(const float* __restrict__ qkv, int T,
                                                           int p0, int Hq, KvLayout kv,
                                                           ActBuf out, int cus) {
  // V^T rows of 68 bf16 (34 dwords), key pairs XOR-swizzled by row group (see
  // vt_col): the transposing 4-byte stores of a wavefront land on 64 distinct
  // banks (8 rows x 8 pairs per store instruction otherwise share 8 banks)
  constexpr int BQ = 64, BKEY = 64, KP = HD + 8, VP = BKEY + 4;
  constexpr int DS = HD / 32;   // 32-deep steps over the head dimension
  constexpr int DT = HD / 16;   // 16-wide output column tiles
  __shared__ __attribute__((aligned(16))) bf16_t Ks[BKEY][KP];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[HD][VP];
  // element column of key pair kp in V^T row group rg (rows 16 rg .. 16 rg + 15)
  auto vt_col = [](int rg, int kp) { return 2 * (kp ^ (8 * ((rg >> 1) & 3))); };

  // A 1-D grid of (query block, head) pairs, padded to a multiple of 8.
  // Workgroups are dealt to the 8 XCDs in turn, so those of one index mod 8
  // share an XCD's L2: each such class takes a contiguous range of the pairs,
  // head-major, which keeps the query heads of a KV head (and so its keys and
  // values) on one XCD.  The grid is dealt out one workgroup per CU and then a
  // second, so workgroups b and b + (CUs) share a CU; their pairs lie CUs / 8
  // apart.  The causal walk of query block i is i + 1 key blocks, so alternate
  // runs of heads, each run as long as that distance, take their query blocks
  // in reverse order, pairing long walks with short ones on every CU.  The
  // order is a function of the head alone, so every (head, query block) is
  // still taken exactly once.
  const int nqb = (T + BQ - 1) / BQ;
  const int lin = blockIdx.x, pair = (lin % 8) * (gridDim.x / 8) + lin / 8;
  if (pair >= nqb * Hq) return;
  const int h = pair / nqb, qq = pair % nqb;
  const int run = max(1, cus / 8 / nqb);  // heads per run
  const int qbi = (h / run) & 1 ? nqb - 1 - qq : qq;
  const int qb = qbi * BQ;
  const int Hkv = kv.n_kv, g = h / (Hq / Hkv);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l16 = lane & 15, lg = lane >> 4;
  const int width = (Hq + 2 * Hkv) * HD;
  const bf16_t* base = static_cast<const bf16_t*>(kv.base);
  const size_t head_stride = (size_t)kv.page * HD;
  const int ps = __ffs(kv.page) - 1;  // pages are a power of two

  // ---- this lane's query (B operand of S^T = K Q^T): row l16 of the wavefront ----
  const int tq = qb + wave * 16 + l16;        // query row in the chunk
  const bool qvalid = tq < T;
  const int qpos = p0 + tq;
  const float scale = 1.0f / sqrtf((float)HD);
  bf16x8_t qf[NT][DS];
  {
    const float* qr = qkv + (size_t)(qvalid ? tq : 0) * width + (size_t)h * HD;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = qvalid ? qr[32 * s + 8 * lg + e] * scale : 0.f;
#pragma unroll
      for (int p = 0; p < NT; ++p) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bf16_t t = f32_to_bf16(v[e]);
          qf[p][s][e] = __builtin_bit_cast(__bf16, t);
          v[e] -= bf16_to_f32(t);
        }
      }
    }
  }

  // ---- key/value loading: thread -> (key pair, 16-wide column chunk) --------------
  constexpr int NCH = HD / 16;                // column chunks per key
  constexpr int ITEMS = BKEY / 2 * NCH;       // (pair, chunk) items per block
  static_assert(ITEMS <= 256, "one (pair, chunk) item per thread at most");
  const bool has_item = tid < ITEMS;
  const int pr = min(tid, ITEMS - 1) / NCH, ch = min(tid, ITEMS - 1) % NCH;
  const int kend = p0 + min(T, qb + BQ);      // keys [0, kend) are visible to this block
  // Two key blocks are in flight ahead of the one being multiplied (two
  // register sets used in turn).  Every load is unconditional, keys past the
  // visible range clamped to the last visible one (finite values that the mask
  // gives zero weight): a load under a branch makes the compiler wait for every
  // load in flight where the paths join, which would expose each block's load
  // latency.  The physical pages of a block's keys are requested one block
  // before its keys and values, which keeps the page lookup off their path.
  auto tload = [&](int kb, int& pg0, int& pg1) {
    pg0 = kv.table[min(kb + 2 * pr, kend - 1) >> ps];
    pg1 = kv.table[min(kb + 2 * pr + 1, kend - 1) >> ps];
  };
  const bf16_t* kbase = base + (size_t)g * head_stride + ch * 16;
  const size_t pstride = (size_t)2 * Hkv * head_stride;  // elements per physical page
  const size_t vofs = (size_t)Hkv * head_stride;         // values after the keys
  // a thread's (key pair, chunk) item of one key block, in one of two register
  // sets: keys 0/1 and values 0/1 of the pair, 16-byte halves a/b
  uint4 ka0a, ka0b, ka1a, ka1b, va0a, va0b, va1a, va1b;
  uint4 kb0a, kb0b, kb1a, kb1b, vb0a, vb0b, vb1a, vb1b;
  auto gload = [&](uint4& k0a, uint4& k0b, uint4& k1a, uint4& k1b, uint4& v0a, uint4& v0b,
                   uint4& v1a, uint4& v1b, int kb, int pg0, int pg1) {
    const int j0 = min(kb + 2 * pr, kend - 1), j1 = min(kb + 2 * pr + 1, kend - 1);
    const bf16_t* kp0 = kbase + (size_t)pg0 * pstride + (size_t)(j0 & (kv.page - 1)) * HD;
    const bf16_t* kp1 = kbase + (size_t)pg1 * pstride + (size_t)(j1 & (kv.page - 1)) * HD;
    k0a = *reinterpret_cast<const uint4*>(kp0);
    k0b = *reinterpret_cast<const uint4*>(kp0 + 8);
    k1a = *reinterpret_cast<const uint4*>(kp1);
    k1b = *reinterpret_cast<const uint4*>(kp1 + 8);
    v0a = *reinterpret_cast<const uint4*>(kp0 + vofs);
    v0b = *reinterpret_cast<const uint4*>(kp0 + vofs + 8);
    v1a = *reinterpret_cast<const uint4*>(kp1 + vofs);
    v1b = *reinterpret_cast<const uint4*>(kp1 + vofs + 8);
  };
  auto sstore = [&](const uint4& k0a, const uint4& k0b, const uint4& k1a, const uint4& k1b,
                    const uint4& v0a, const uint4& v0b, const uint4& v1a, const uint4& v1b) {
    if (has_item) {
      *reinterpret_cast<uint4*>(&Ks[2 * pr][ch * 16]) = k0a;
      *reinterpret_cast<uint4*>(&Ks[2 * pr][ch * 16 + 8]) = k0b;
      *reinterpret_cast<uint4*>(&Ks[2 * pr + 1][ch * 16]) = k1a;
      *reinterpret_cast<uint4*>(&Ks[2 * pr + 1][ch * 16 + 8]) = k1b;
      // V transposed: column d of the pair's two keys packed in one dword
      const uint32_t a[8] = {v0a.x, v0a.y, v0a.z, v0a.w, v0b.x, v0b.y, v0b.z, v0b.w};
      const uint32_t b[8] = {v1a.x, v1a.y, v1a.z, v1a.w, v1b.x, v1b.y, v1b.z, v1b.w};
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        // elements 2w, 2w+1 of the chunk
        *reinterpret_cast<uint32_t*>(&Vt[ch * 16 + 2 * w][vt_col(ch, pr)]) = (a[w] & 0xffffu) | (b[w] << 16);
        *reinterpret_cast<uint32_t*>(&Vt[ch * 16 + 2 * w + 1][vt_col(ch, pr)]) =
            (a[w] >> 16) | (b[w] & 0xffff0000u);
      }
    }
  };

  floatx4_t o[DT];
#pragma unroll
  for (int u = 0; u < DT; ++u) o[u] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_part = 0.f;

  auto compute = [&](int kb) {
    // S^T tile t: lane holds S[query l16][key 16 t + 4 lg + r]
    floatx4_t st[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      st[t] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < DS; ++s) {
        const bf16x8_t kf = *reinterpret_cast<const bf16x8_t*>(&Ks[16 * t + l16][32 * s + 8 * lg]);
#pragma unroll
        for (int p = 0; p < NT; ++p)
          st[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[p][s], st[t], 0, 0, 0);
      }
    }
    // causal mask and block max, probabilities split into NT bf16 terms in the
    // A-operand key order, and the rescale of the output rows.  Key blocks that
    // every query of this wavefront sees whole (all but the diagonal and the last
    // one) take the path without the mask and its -inf tests; a wavefront whose
    // running maxima all stay put has correction factors of exactly 1 and skips
    // the rescale.  Both paths give the same bits as the general one.
    bf16x8_t pf[NT][2];
    auto softmax = [&](auto masked_t) {
      constexpr bool MASKED = decltype(masked_t)::value;
      float bm = -INFINITY;
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if (MASKED) {
            const int j = kb + 16 * t + 4 * lg + r;
            if (j > qpos || j >= kend) st[t][r] = -INFINITY;
          }
          bm = fmaxf(bm, st[t][r]);
        }
      bm = fmaxf(bm, __shfl_xor(bm, 16));
      bm = fmaxf(bm, __shfl_xor(bm, 32));
      const float m_old = m_run, m_new = fmaxf(m_old, bm);
      m_run = m_new;
      const bool grow = __any(m_new > m_old);
      float pvs[16];
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float sv = st[2 * c + (e >> 2)][e & 3];
          float pv = MASKED && sv == -INFINITY ? 0.f : __expf(sv - m_new);
          pvs[8 * c + e] = pv;
#pragma unroll
          for (int p = 0; p < NT; ++p) {
            const bf16_t tb = f32_to_bf16(pv);
            pf[p][c][e] = __builtin_bit_cast(__bf16, tb);
            pv -= bf16_to_f32(tb);
          }
        }
      // l = l corr + p_0 + ... + p_15, the first step fused (with corr = 1, as
      // when no maximum grew, the fused step is the plain sum)
      float corr = 1.f;
      if (grow) {
        corr = m_new == -INFINITY ? 1.f : __expf(m_old - m_new);
        l_part = __builtin_fmaf(l_part, corr, pvs[0]);
      } else {
        l_part += pvs[0];
      }
#pragma unroll
      for (int i = 1; i < 16; ++i) l_part += pvs[i];
      if (grow) {
        // the output rows (queries 4 lg + r) by their correction factors
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float cr = __shfl(corr, 4 * lg + r);
#pragma unroll
          for (int u = 0; u < DT; ++u) o[u][r] *= cr;
        }
      }
    };
    if (kb + BKEY - 1 > p0 + qb + 16 * wave || kb + BKEY > kend)
      softmax(std::true_type{});
    else
      softmax(std::false_type{});
    // O += P V: B operand = V^T rows d, keys in the same slot order as P
#pragma unroll
    for (int u = 0; u < DT; ++u) {
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        // keys 32 c + 4 lg .. + 3 (pairs 16 c + 2 lg, + 1) and 16 further on
        const bf16_t* vrow = &Vt[16 * u + l16][0];
        const uint2 lo = *reinterpret_cast<const uint2*>(vrow + vt_col(u, 16 * c + 2 * lg));
        const uint2 hi = *reinterpret_cast<const uint2*>(vrow + vt_col(u, 16 * c + 2 * lg + 8));
        const uint4 w4 = make_uint4(lo.x, lo.y, hi.x, hi.y);
        const bf16x8_t vf = __builtin_bit_cast(bf16x8_t, w4);
#pragma unroll
        for (int p = 0; p < NT; ++p)
          o[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pf[p][c], vf, o[u], 0, 0, 0);
      }
    }
  };

  // blocks kb (set a) and kb + BKEY (set b) in turn; each step stores its set,
  // refills it with the block two ahead and multiplies the stored block
#define WICI_SET_A ka0a, ka0b, ka1a, ka1b, va0a, va0b, va1a, va1b
#define WICI_SET_B kb0a, kb0b, kb1a, kb1b, vb0a, vb0b, vb1a, vb1b
  int pa0, pa1, pb0, pb1;  // pages of the next block to load into set a / b
  tload(0, pa0, pa1);
  gload(WICI_SET_A, 0, pa0, pa1);
  tload(BKEY, pb0, pb1);
  gload(WICI_SET_B, BKEY, pb0, pb1);
  tload(2 * BKEY, pa0, pa1);
  for (int kb = 0; kb < kend; kb += 2 * BKEY) {
    __syncthreads();          // previous block's readers are done with LDS
    sstore(WICI_SET_A);
    __syncthreads();
    gload(WICI_SET_A, kb + 2 * BKEY, pa0, pa1);
    tload(kb + 3 * BKEY, pb0, pb1);
    compute(kb);
    if (kb + BKEY >= kend) break;
    __syncthreads();
    sstore(WICI_SET_B);
    __syncthreads();
    gload(WICI_SET_B, kb + 3 * BKEY, pb0, pb1);
    tload(kb + 4 * BKEY, pa0, pa1);
    compute(kb + BKEY);
  }
#undef WICI_SET_A
#undef WICI_SET_B

  // ---- normalise and write: lane holds O[query 4 lg + r][d 16 u + l16] -----------
  float l_tot = l_part + __shfl_xor(l_part, 16);
  l_tot += __shfl_xor(l_tot, 32);
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int qrow = 4 * lg + r;
    const float inv = 1.0f / __shfl(l_tot, qrow);
    const int t = qb + wave * 16 + qrow;
    if (t < T) {
      const size_t ob = (size_t)t * Hq * HD + (size_t)h * HD;
#pragma unroll
      for (int u = 0; u < DT; ++u) store_act(out, ob + 16 * u + l16, o[u][r] * inv);
    }
  }
}

// Compute units of the current device (the prefill attention's workgroup
// pairing), looked up once per device.
static int device_cus() {
  static int cached[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        v < 1)
      v = 256;
    cached[dev] = v;
  }
  return cached[dev];
}

template <int HD, typename KT>
static hipError_t attn_prefill_t(const float* qkv, int T, int p0, int Hq, KvLayout kv,
                                 const ActBuf& out, hipStream_t s) {
  hipLaunchKernelGGL((k_attn_prefill<HD, KT>), dim3((T + 63) / 64, Hq), dim3(256), 0, s, qkv, T,
                     p0, Hq, kv, out, device_cus());
  return hipGetLastError();
}

template <int HD>
static hipError_t attn_prefill_mfma(const float* qkv, int T, int p0, int Hq, KvLayout kv,
                                    const ActBuf& out, int terms, hipStream_t s) {
  const dim3 grid(((T + 63) / 64 * Hq + 7) / 8 * 8);
  const int cus = device_cus();
  switch (terms) {
    case 1: hipLaunchKernelGGL((k_attn_prefill_mfma<HD, 1>), grid, dim3(256), 0, s, qkv, T, p0, Hq, kv, out, cus); break;
    case 2: hipLaunchKernelGGL((k_attn_prefill_mfma<HD, 2>), grid, dim3(256), 0, s, qkv, T, p0, Hq, kv, out, cus); break;
    case 3: hipLaunchKernelGGL((k_attn_prefill_mfma<HD, 3>), grid, dim3(256), 0, s, qkv, T, p0, Hq, kv, out, cus); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// bf16 cache with split-activation output: matrix cores, with the query and the
// probabilities carried in `terms` bf16 terms (0: as many as the output stores);
// otherwise the fp32 vector kernel.
hipError_t launch_attn_prefill(bool kv_bf16, const float* qkv, int T, int p0, int Hq,
                               KvLayout kv, const ActBuf& out, hipStream_t s, int terms) {
  if (kv.page < 1 || (kv.page & (kv.page - 1)) || terms < 0 || terms > 3)
    return hipErrorInvalidValue;
  if (kv_bf16 && out.nt >= 1) {
    const int nt = terms > 0 ? terms : out.nt;
    if (kv.hd == 128) return attn_prefill_mfma<128>(qkv, T, p0, Hq, kv, out, nt, s);
    if (kv.hd == 64) return attn_prefill_mfma<64>(qkv, T, p0, Hq, kv, out, nt, s);
    return hipErrorInvalidValue;
  }
  if (kv.hd == 128) {
    if (kv_bf16) return attn_prefill_t<128, bf16_t>(qkv, T, p0, Hq, kv, out, s);
    return attn_prefill_t<128, float>(qkv, T, p0, Hq, kv, out, s);
  }
  if (kv.hd == 64) {
    if (kv_bf16) return attn_prefill_t<64, bf16_t>(qkv, T, p0, Hq, kv, out, s);
    return attn_prefill_t<64, float>(qkv, T, p0, Hq, kv, out, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace wici
