// Token-selection kernels: RocketKV top-k, H2O eviction, H2O and SnapKV prefill eviction.
//
// MetaKV Section 2.1: H2O keeps the tokens with the highest accumulated attention and evicts the
// lowest-scoring older token once over budget; RocketKV first keeps the prompt tokens the
// observation window votes for (SnapKV), then attends to a top-k subset per decode step.
// Selections are block-wide radix selects on order-preserving 32-bit keys followed by an
// ascending-position compaction, so ties resolve by position exactly as specified.
#include "kernels_common.h"

namespace mkv {

namespace {

constexpr int NT = 256;
constexpr int kTopkLdsKeys = 10240;  // score keys of up to this many retained tokens stay in LDS

// Compact positions [0, n) whose flag is set into ascending slots; calls emit(j, slot) for each.
// flag(j, eq_before) may use eq_before = number of keys equal to the threshold at indices < j.
template <typename Flag, typename IsEq, typename Emit>
MKV_DEV int compact_ascending(int n, Flag flag, IsEq is_eq, Emit emit, int *s_tmp) {
  int run = 0, eq_run = 0;
  for (int a = 0; a < n; a += NT) {
    const int j = a + (int)threadIdx.x;
    const bool in = j < n;
    const int e = (in && is_eq(j)) ? 1 : 0;
    int eq_tot;
    const int eq_before = eq_run + block_exclusive_scan<NT>(e, s_tmp, &eq_tot);
    const int f = (in && flag(j, eq_before)) ? 1 : 0;
    int tot;
    const int ex = block_exclusive_scan<NT>(f, s_tmp, &tot);
    if (f) emit(j, run + ex);
    run += tot;
    eq_run += eq_tot;
  }
  return run;
}

// ---- RocketKV decode top-k ---------------------------------------------------------------------
// Radix select of the k-th largest of n keys (4 passes of 8 bits) for a workgroup of NT threads:
// one histogram per wave, two sets used in turn so that the set of the next pass is cleared
// while wave 0 searches the digit of this one (2 barriers per pass).  hist[0] must be zero and
// visible on entry.  Returns the k-th key, how many keys equal it and how many of those are needed.
template <int NTH, typename Get>
MKV_DEV void topk_radix(int n, int k, Get get, int (*hist)[NTH / 64][256], int *s3, uint32_t *kth, int *n_equal,
                        int *need) {
  constexpr int NWV = NTH / 64;
  const int wid = threadIdx.x >> 6, lane = threadIdx.x & 63;
  uint32_t prefix = 0, mask = 0;
  int remaining = k, eq = 0;
  for (int pass = 0; pass < 4; ++pass) {
    const int buf = pass & 1, shift = 24 - 8 * pass;
    for (int i = threadIdx.x; i < n; i += NTH) {
      const uint32_t key = get(i);
      if ((key & mask) == prefix) atomicAdd(&hist[buf][wid][(key >> shift) & 255u], 1);
    }
    __syncthreads();
    if (wid == 0) {
      // lane l owns digits 255 - 4l .. 252 - 4l (descending), so the exclusive scan over lanes
      // gives the count of larger digits
      int cnt[4], tot = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = 255 - (4 * lane + i);
        int c = 0;
#pragma unroll
        for (int w = 0; w < NWV; ++w) c += hist[buf][w][d];
        cnt[i] = c;
        tot += c;
      }
      int inc = tot;
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const int y = __shfl_up(inc, o);
        if (lane >= o) inc += y;
      }
      int above = inc - tot;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (above < remaining && remaining <= above + cnt[i]) {
          s3[0] = 255 - (4 * lane + i);
          s3[1] = remaining - above;
          s3[2] = cnt[i];
        }
        above += cnt[i];
      }
    } else {
      for (int e = threadIdx.x - 64; e < NWV * 256; e += NTH - 64) (&hist[buf ^ 1][0][0])[e] = 0;
    }
    __syncthreads();
    prefix |= (uint32_t)s3[0] << shift;
    mask |= 255u << shift;
    remaining = s3[1];
    eq = s3[2];
  }
  *kth = prefix;
  *n_equal = eq;
  *need = remaining;
}


// Approximate scores of the T consecutive tokens [j0, j0 + T) (T = 4 or 8) from the channel-major
// key copy: one 2T-byte load per selected channel, R channels' loads issued before any is used,
// channels ascending, every product and sum rounded to fp32 separately (no fused multiply-add).
// Rows are padded to 8 tokens and j0 is a multiple of T, so no load leaves its row.
template <int T, int R>
MKV_DEV void score_tokens(const uint16_t *kcm, int cstride, int j0, int nch, const int *sel_ch, const float *sel_qb,
                          float (&acc)[T]) {
#pragma unroll
  for (int t = 0; t < T; ++t) acc[t] = 0.f;
  for (int i0 = 0; i0 < nch; i0 += R) {
    uint32_t w[R][T / 2];
#pragma unroll
    for (int ii = 0; ii < R; ++ii) {
      const int i = min(i0 + ii, nch - 1);
      const uint32_t *p = reinterpret_cast<const uint32_t *>(kcm + (size_t)sel_ch[i] * cstride + j0);
#pragma unroll
      for (int u = 0; u < T / 2; ++u) w[ii][u] = gld(p + u);
    }
#pragma unroll
    for (int ii = 0; ii < R; ++ii) {
      if (i0 + ii < nch) {
        const float qb = sel_qb[i0 + ii];
#pragma unroll
        for (int u = 0; u < T / 2; ++u) {
          acc[2 * u] = __fadd_rn(acc[2 * u], __fmul_rn(qb, h2f(w[ii][u])));
          acc[2 * u + 1] = __fadd_rn(acc[2 * u + 1], __fmul_rn(qb, h2f(w[ii][u] >> 16)));
        }
      }
    }
  }
}


// One workgroup of 1024 threads per (sequence, kv head): a kept set of up to a few thousand
// tokens is scored with ~4 tokens per thread and selected by radix passes over LDS keys.
constexpr int kTopkThreads = 1024;
template <int D, int G>
__global__ __launch_bounds__(kTopkThreads) void k_topk(const SeqDesc *__restrict__ seqs, int32_t *state,
                                             const uint16_t *__restrict__ q, int32_t *pos_out, int topk_max,
                                             int Hkv) {
  __shared__ float s_a[D];
  __shared__ float s_qb[D];
  __shared__ int s_ch[D];
  __shared__ int s_beats[kTopkThreads];
  __shared__ int whist[2][kTopkThreads / 64][256];
  __shared__ int s3[3];
  __shared__ int s_tmp[kTopkThreads / 64];
  __shared__ uint32_t s_keys[kTopkLdsKeys];
  const int seq = blockIdx.x / Hkv, h = blockIdx.x % Hkv;
  const SeqDesc &sd = seqs[seq];
  if (sd.method != ROCKET) return;
  int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  const int n = st[ST_COUNT];
  const int k = sd.topk;
  int32_t *sel = reinterpret_cast<int32_t *>(sd.sel) + h * stride_sel(sd);
  const int32_t *pos = reinterpret_cast<const int32_t *>(sd.pos) + h * stride_slots(sd);
  int32_t *chan_out = reinterpret_cast<int32_t *>(sd.aux1) + (size_t)h * D;
  const int Hq = Hkv * G;
  const uint16_t *qh = q + ((size_t)seq * Hq + h * G) * D;

  // channel magnitudes and head sums, float32 in ascending head order
  for (int c = threadIdx.x; c < D; c += kTopkThreads) {
    float a = 0.f, qb = 0.f;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float x = h2f(qh[(size_t)g * D + c]);
      a = __fadd_rn(a, fabsf(x));
      qb = __fadd_rn(qb, x);
    }
    s_a[c] = a;
    s_qb[c] = qb;
  }
  __syncthreads();
  const int nch = min(sd.nch, D);
  // channel c is selected iff fewer than nch channels beat it (larger a, or equal a and lower
  // index); the kTopkThreads / D threads of channel c each count a slice of the others
  {
    static_assert(kTopkThreads % D == 0, "whole slices per channel");
    constexpr int P = kTopkThreads / D, W = D / P;
    const int c = threadIdx.x % D, part = threadIdx.x / D;
    const float a = s_a[c];
    int beats = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
      const int c2 = part * W + i;
      const float b = s_a[c2];
      beats += (b > a || (b == a && c2 < c)) ? 1 : 0;
    }
    s_beats[threadIdx.x] = beats;
  }
  __syncthreads();
  if (threadIdx.x < D) {
    int t = 0;
#pragma unroll
    for (int p = 0; p < kTopkThreads / D; ++p) t += s_beats[p * D + threadIdx.x];
    s_ch[threadIdx.x] = t < nch ? 1 : 0;
  }
  __syncthreads();
  __shared__ int s_sel_ch[D];
  __shared__ float s_sel_qb[D];
  __shared__ int s_wcnt[(D + 63) / 64];
  // ascending compaction of the selected channels: rank = selected channels below c
  {
    const int c = threadIdx.x;
    const bool f = c < D && s_ch[c] != 0;
    const uint64_t m = __ballot(f);
    const int lane = c & 63, w = c >> 6;
    if (c < D && lane == 0) s_wcnt[w] = __popcll(m);
    __syncthreads();
    if (f) {
      int r = __popcll(m & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
      for (int i = 0; i < w; ++i) r += s_wcnt[i];
      s_sel_ch[r] = c;
      s_sel_qb[r] = s_qb[c];
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nch; i += kTopkThreads) chan_out[i] = s_sel_ch[i];

  if (k >= n) {
    for (int j = threadIdx.x; j < n; j += kTopkThreads) sel[j] = j;
    if (pos_out != nullptr)
      for (int i = threadIdx.x; i < topk_max; i += kTopkThreads)
        pos_out[((size_t)seq * Hkv + h) * topk_max + i] = i < n ? pos[i] : -1;
    if (threadIdx.x == 0) st[ST_SEL_COUNT] = n;
    return;
  }

  // approximate scores from the channel-major key copy, channels ascending,
  // acc = fl32(acc + fl32(qbar_c * k_jc)); the keys stay in LDS when they fit.  A lane scores 4
  // consecutive tokens (8 for sets of more than 4 kTopkThreads tokens, so that one pass covers up
  // to 8 kTopkThreads)
  const uint16_t *kcm = reinterpret_cast<const uint16_t *>(sd.kcm) + h * stride_kcm(sd, D);
  uint32_t *akeys = reinterpret_cast<uint32_t *>(sd.akeys) + h * stride_slots(sd);
  const bool in_lds = n <= kTopkLdsKeys;
  const int cstride = sd.cstride;
  auto put = [&](int j, float a) {
    if (j < n) {
      if (in_lds) s_keys[j] = float_key(a);
      else gst(akeys + j, float_key(a));
    }
  };
  if (n <= 4 * kTopkThreads) {
    const int j0 = 4 * (int)threadIdx.x;
    if (j0 < n) {
      float acc[4];
      score_tokens<4, 32>(kcm, cstride, j0, nch, s_sel_ch, s_sel_qb, acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) put(j0 + r, acc[r]);
    }
  } else {
    for (int j0 = 8 * (int)threadIdx.x; j0 < n; j0 += 8 * kTopkThreads) {
      float acc[8];
      score_tokens<8, 16>(kcm, cstride, j0, nch, s_sel_ch, s_sel_qb, acc);
#pragma unroll
      for (int r = 0; r < 8; ++r) put(j0 + r, acc[r]);
    }
  }
  for (int e = threadIdx.x; e < (kTopkThreads / 64) * 256; e += kTopkThreads) (&whist[0][0][0])[e] = 0;
  __syncthreads();
  auto getk = [&](int i) { return in_lds ? s_keys[i] : gld(akeys + i); };
  uint32_t kth;
  int n_eq, need;
  topk_radix<kTopkThreads>(n, k, getk, whist, s3, &kth, &n_eq, &need);
  // each thread takes a contiguous run of tokens; counts of keys above and equal to the
  // threshold before its run place its selected tokens in ascending order
  const int per = (n + kTopkThreads - 1) / kTopkThreads;
  const int ja = min(n, (int)threadIdx.x * per), jb = min(n, ja + per);
  int gt = 0, eq = 0;
  for (int j = ja; j < jb; ++j) {
    const uint32_t kk = getk(j);
    gt += kk > kth ? 1 : 0;
    eq += kk == kth ? 1 : 0;
  }
  // one scan of both counts when n < 2^15 keeps them apart in the two halves of a word
  int tot, gt_before, eq_run;
  if (n < 32768) {
    const int both = block_exclusive_scan<kTopkThreads>((gt << 16) | eq, s_tmp, &tot);
    gt_before = both >> 16;
    eq_run = both & 0xFFFF;
  } else {
    gt_before = block_exclusive_scan<kTopkThreads>(gt, s_tmp, &tot);
    eq_run = block_exclusive_scan<kTopkThreads>(eq, s_tmp, &tot);
  }
  int slot = gt_before + min(eq_run, need);
  for (int j = ja; j < jb; ++j) {
    const uint32_t kk = getk(j);
    const bool take = kk > kth || (kk == kth && eq_run < need);
    eq_run += kk == kth ? 1 : 0;
    if (take && slot < k) gst(sel + slot, j);
    slot += take ? 1 : 0;
  }
  __syncthreads();
  if (pos_out != nullptr)
    for (int i = threadIdx.x; i < topk_max; i += kTopkThreads)
      pos_out[((size_t)seq * Hkv + h) * topk_max + i] = i < k ? gld(pos + gld(sel + i)) : -1;
  if (threadIdx.x == 0) st[ST_SEL_COUNT] = k;
}

// ---- causal prefill attention statistics for H2O scoring, on the matrix cores ------------------
// Logit tiles S = Q K^T of 16 query rows x 16 keys come from v_mfma_f32_16x16x32_f16: Q and K are
// fp16 exactly, products exact, sums in float32.  Operand lane roles (lr = lane % 16, lq = lane /
// 16): A (16 rows x 32 channels) row lr, channels 8 lq .. 8 lq + 7 of the k-step; B (32 channels x
// 16 keys) key lr, the same channels; result rows 4 lq + j (j = 0..3), key lr.
constexpr int TB = 64;

typedef _Float16 h8v __attribute__((ext_vector_type(8)));
typedef float f4v __attribute__((ext_vector_type(4)));

MKV_DEV f4v mfma_k32(const uint4 &a, const uint4 &b, f4v c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(h8v, a), __builtin_bit_cast(h8v, b), c, 0, 0, 0);
}

// Sum and max over the 16 lanes of a row (lanes with the same lq).
MKV_DEV float row16_max(float x) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
MKV_DEV float row16_sum(float x) {
#pragma unroll
  for (int o = 1; o < 16; o <<= 1) x += __shfl_xor(x, o);
  return x;
}

// Row statistics (max, sum of exp2) of query head gq's causal logits over the prompt keys: a
// workgroup takes 64 query rows (16 per wave, their Q operands in registers) and walks the
// 64-key tiles up to the diagonal, each staged once in LDS for the four waves.  Every lane keeps
// a running (max, sum) for its 4 rows over the keys of its column, merged across the row's 16
// lanes at the end.
template <int D>
__global__ __launch_bounds__(NT) void k_h2o_rowstats(const SeqDesc *__restrict__ seqs, int seq,
                                                     const uint16_t *__restrict__ qrows, int Hq, int G,
                                                     float scale2) {
  constexpr int KS = D / 32, U = D / 8;  // k-steps; 16-byte units per row
  __shared__ uint4 sk[TB][U + 1];
  const SeqDesc &sd = seqs[seq];
  const int n0 = sd.n0;
  const int rb = blockIdx.x, gq = blockIdx.y, h = gq / G, g = gq % G;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, lr = lane & 15, lq = lane >> 4;
  const int r0 = rb * TB + 16 * wave;  // this wave's first row
  uint4 qa[KS];
  {
    const uint4 *qp = reinterpret_cast<const uint4 *>(qrows + (size_t)min(r0 + lr, n0 - 1) * Hq * D + (size_t)gq * D);
#pragma unroll
    for (int s = 0; s < KS; ++s) qa[s] = gld16(qp + 4 * s + lq);
  }
  const uint4 *ks = reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(sd.stage_k) +
                                                    h * stride_stage(sd, D));
  float m[4], l[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    m[j] = -INFINITY;
    l[j] = 0.f;
  }
  // the next tile's loads are in flight while the current one is computed
  constexpr int PER = TB * U / NT;  // 16-byte units per thread and tile
  uint4 nxt[PER];
#pragma unroll
  for (int k = 0; k < PER; ++k) {
    const int e = threadIdx.x + k * NT, r = e / U, u = e % U;
    nxt[k] = gld16(ks + (size_t)min(r, n0 - 1) * U + u);
  }
  for (int kb = 0; kb <= rb; ++kb) {
    __syncthreads();
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int e = threadIdx.x + k * NT;
      sk[e / U][e % U] = nxt[k];
    }
    __syncthreads();
    if (kb < rb) {
#pragma unroll
      for (int k = 0; k < PER; ++k) {
        const int e = threadIdx.x + k * NT, r = e / U, u = e % U;
        nxt[k] = gld16(ks + (size_t)min((kb + 1) * TB + r, n0 - 1) * U + u);
      }
    }
    if (kb * TB > r0 + 15) continue;  // the tile lies wholly above this wave's rows
    float v[4][4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      f4v S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) S = mfma_k32(qa[s], sk[16 * n + lr][4 * s + lq], S);
      const int key = kb * TB + 16 * n + lr;
#pragma unroll
      for (int j = 0; j < 4; ++j) v[n][j] = (key <= r0 + 4 * lq + j && key < n0) ? S[j] * scale2 : -INFINITY;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float mx = fmaxf(fmaxf(m[j], fmaxf(v[0][j], v[1][j])), fmaxf(v[2][j], v[3][j]));
      if (mx == -INFINITY) continue;
      float acc = l[j] * fexp2(m[j] - mx);
#pragma unroll
      for (int n = 0; n < 4; ++n) acc += fexp2(v[n][j] - mx);
      l[j] = acc;
      m[j] = mx;
    }
  }
  float2 *out = reinterpret_cast<float2 *>(sd.aux1) + (size_t)h * G * n0 + (size_t)g * n0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float M = row16_max(m[j]);
    const float L = row16_sum(m[j] == -INFINITY ? 0.f : l[j] * fexp2(m[j] - M));
    const int i = r0 + 4 * lq + j;
    if (lr == 0 && i < n0) out[i] = make_float2(M, L);
  }
}

// Column sums S_j = sum_g sum_{i >= j} p_gij over a block of 64 keys: every wave holds the
// block's K operands in registers and takes every fourth 16-row chunk of the rows at or below
// the block, for each of the kv head's query heads; the waves' sums meet in LDS.
template <int D>
__global__ __launch_bounds__(NT) void k_h2o_colsums(const SeqDesc *__restrict__ seqs, int seq,
                                                    const uint16_t *__restrict__ qrows, int Hq, int G,
                                                    float scale2) {
  constexpr int KS = D / 32, U = D / 8;
  __shared__ float scol[NT / 64][TB];
  const SeqDesc &sd = seqs[seq];
  const int n0 = sd.n0;
  const int kb = blockIdx.x, h = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, lr = lane & 15, lq = lane >> 4;
  const uint4 *ks = reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(sd.stage_k) +
                                                    h * stride_stage(sd, D));
  uint4 kop[4][KS];
#pragma unroll
  for (int n = 0; n < 4; ++n)
#pragma unroll
    for (int s = 0; s < KS; ++s) kop[n][s] = gld16(ks + (size_t)min(kb * TB + 16 * n + lr, n0 - 1) * U + 4 * s + lq);
  const float2 *stat = reinterpret_cast<const float2 *>(sd.aux1) + (size_t)h * G * n0;
  float col[4] = {0.f, 0.f, 0.f, 0.f};
  const int nchunk = (n0 + 15) / 16;
  // (query head, 16-row chunk) items of this wave in order, the next item's loads in flight while
  // the current one is computed
  const int c0 = kb * (TB / 16) + wave, per_g = c0 < nchunk ? (nchunk - c0 + NT / 64 - 1) / (NT / 64) : 0;
  const int items = G * per_g;
  auto load = [&](int it, uint4 (&qa)[KS], float (&M)[4], float (&iL)[4]) {
    const int g = it / per_g, c = c0 + (it % per_g) * (NT / 64);
    const uint4 *qp = reinterpret_cast<const uint4 *>(qrows + (size_t)min(16 * c + lr, n0 - 1) * Hq * D +
                                                      (size_t)(h * G + g) * D);
#pragma unroll
    for (int s = 0; s < KS; ++s) qa[s] = gld16(qp + 4 * s + lq);
    const float2 *sg = stat + (size_t)g * n0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float *ml = reinterpret_cast<const float *>(sg + min(16 * c + 4 * lq + j, n0 - 1));
      M[j] = gld(ml);
      iL[j] = gld(ml + 1);
    }
  };
  uint4 qn[KS];
  float Mn[4], Ln[4];
  if (items > 0) load(0, qn, Mn, Ln);
  for (int it = 0; it < items; ++it) {
    const int c = c0 + (it % per_g) * (NT / 64);
    uint4 qa[KS];
    float M[4], iL[4];
#pragma unroll
    for (int s = 0; s < KS; ++s) qa[s] = qn[s];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      M[j] = Mn[j];
      iL[j] = 1.f / Ln[j];
    }
    if (it + 1 < items) load(it + 1, qn, Mn, Ln);
    {
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        f4v S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) S = mfma_k32(qa[s], kop[n][s], S);
        const int key = kb * TB + 16 * n + lr;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = 16 * c + 4 * lq + j;
          // arguments <= 0 wherever the row statistics hold this logit
          col[n] += (i < n0 && key <= i && key < n0) ? fexp2(S[j] * scale2 - M[j]) * iL[j] : 0.f;
        }
      }
    }
  }
#pragma unroll
  for (int n = 0; n < 4; ++n) {
    float x = col[n];
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    if (lq == 0) scol[wave][16 * n + lr] = x;
  }
  __syncthreads();
  if (threadIdx.x < TB) {
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) acc += scol[w][threadIdx.x];
    const int jj = kb * TB + threadIdx.x;
    if (jj < n0) (reinterpret_cast<float *>(sd.aux0) + (size_t)h * n0)[jj] = acc;
  }
}

// Keep the R most recent prompt tokens plus the top B - R scores of the rest (newer on ties),
// compact them into slots 0..kept-1 in ascending position order.
template <int D>
__global__ __launch_bounds__(NT) void k_h2o_keep(const SeqDesc *__restrict__ seqs, int seq, int32_t *state,
                                                 int Hkv) {
  __shared__ int hist[256];
  __shared__ int s3[3];
  __shared__ int s_tmp[NT / 64];
  const SeqDesc &sd = seqs[seq];
  const int h = blockIdx.x, n0 = sd.n0;
  const float *S = reinterpret_cast<const float *>(sd.aux0) + (size_t)h * n0;
  const int B = sd.B, R = sd.R;
  const bool all = B >= n0;
  const int ncand = all ? 0 : n0 - R;
  const int H = all ? 0 : B - R;
  uint32_t kth = 0xFFFFFFFFu;
  int n_eq = 0, need = 0;
  if (H > 0) radix_select_kth<NT>(ncand, H, [&](int i) { return float_key(S[i]); }, hist, s3, &kth, &n_eq, &need);
  const uint16_t *sk = reinterpret_cast<const uint16_t *>(sd.stage_k) + h * stride_stage(sd, D);
  const uint16_t *sv = reinterpret_cast<const uint16_t *>(sd.stage_v) + h * stride_stage(sd, D);
  uint16_t *dk = reinterpret_cast<uint16_t *>(sd.k) + h * stride_rows(sd, D);
  uint16_t *dvv = reinterpret_cast<uint16_t *>(sd.v) + h * stride_rows(sd, D);
  int32_t *pos = reinterpret_cast<int32_t *>(sd.pos) + h * stride_slots(sd);
  float *score = reinterpret_cast<float *>(sd.score) + h * stride_slots(sd);
  const int kept = compact_ascending(
      n0,
      [&](int j, int eq_before) {
        if (all || j >= ncand) return true;
        if (H == 0) return false;
        const uint32_t kk = float_key(S[j]);
        return kk > kth || (kk == kth && eq_before >= n_eq - need);
      },
      [&](int j) { return !all && H > 0 && j < ncand && float_key(S[j]) == kth; },
      [&](int j, int slot) {
        if (slot >= sd.cap) return;
        pos[slot] = j;
        score[slot] = S[j];
        for (int c = 0; c < D; c += 8) {
          *reinterpret_cast<uint4 *>(dk + (size_t)slot * D + c) = *reinterpret_cast<const uint4 *>(sk + (size_t)j * D + c);
          *reinterpret_cast<uint4 *>(dvv + (size_t)slot * D + c) = *reinterpret_cast<const uint4 *>(sv + (size_t)j * D + c);
        }
      },
      s_tmp);
  if (threadIdx.x == 0) {
    int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
    st[ST_COUNT] = kept;
    st[ST_FREE_SLOT] = kept;
    st[ST_KEPT] = kept;
  }
}

// ---- SnapKV prefill -------------------------------------------------------------------------------
// Window row r = i * G + g (query head h*G + g at position n0 - w + i).  Pass 1: per 256-key chunk
// and wave, the partial (max, sum of exp2) of every row.  Pass 2: merge, then votes of the
// chunk's keys.  Pass 3: pool, select, compact.
constexpr int SNAP_CHUNK = 256;

template <int D>
MKV_DEV void load_key_row(const uint16_t *ks, int j, int n0, float *kr) {
  if (j < n0) {
#pragma unroll
    for (int c = 0; c < D; c += 8) {
      const uint4 u = *reinterpret_cast<const uint4 *>(ks + (size_t)j * D + c);
      unpack8(u, kr + c);
    }
  } else {
#pragma unroll
    for (int c = 0; c < D; ++c) kr[c] = 0.f;
  }
}

template <int D>
MKV_DEV void load_window(float (*sq)[D], const uint16_t *qw, int h, int G, int Hq, int w, int wfull,
                         int r0, int nr) {
  for (int e = threadIdx.x; e < nr * D; e += NT) {
    const int rr = e / D, c = e % D;
    const int r = r0 + rr, i = r / G, g = r % G;
    // the last w of the `wfull` window rows
    sq[rr][c] = h2f(qw[((size_t)(wfull - w + i) * Hq + h * G + g) * D + c]);
  }
}

constexpr int SNAP_ROWS = 64;   // window rows staged in LDS at a time

template <int D>
__global__ __launch_bounds__(NT) void k_snap_rowstats(const SeqDesc *__restrict__ seqs, int seq,
                                                      const uint16_t *__restrict__ qw, int Hq, int G,
                                                      float scale2) {
  __shared__ float sq[SNAP_ROWS][D];
  const SeqDesc &sd = seqs[seq];
  const int n0 = sd.n0, w = sd.w_eff, wfull = sd.window;
  const int chunk = blockIdx.x, h = blockIdx.y;
  const int nchunk = (n0 + SNAP_CHUNK - 1) / SNAP_CHUNK;
  const int j = chunk * SNAP_CHUNK + (int)threadIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint16_t *ks = reinterpret_cast<const uint16_t *>(sd.stage_k) + h * stride_stage(sd, D);
  float kr[D];
  load_key_row<D>(ks, j, n0, kr);
  const int rows = w * G;
  float2 *part = reinterpret_cast<float2 *>(sd.aux1) + (size_t)h * rows * nchunk * 4;
  for (int r0 = 0; r0 < rows; r0 += SNAP_ROWS) {
    const int nr = min(SNAP_ROWS, rows - r0);
    __syncthreads();
    load_window<D>(sq, qw, h, G, Hq, w, wfull, r0, nr);
    __syncthreads();
    for (int rr = 0; rr < nr; ++rr) {
      const int r = r0 + rr, i = r / G;
      const int posr = n0 - w + i;
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < D; ++c) acc = fmaf(sq[rr][c], kr[c], acc);
      const float s = (j <= posr && j < n0) ? acc * scale2 : -INFINITY;
      const float M = wave_max(s);
      const float L = wave_sum(M == -INFINITY ? 0.f : exp2f(s - M));
      if (lane == 0) part[((size_t)r * nchunk + chunk) * 4 + wave] = make_float2(M, L);
    }
  }
}

template <int D>
__global__ __launch_bounds__(NT) void k_snap_votes(const SeqDesc *__restrict__ seqs, int seq,
                                                   const uint16_t *__restrict__ qw, int Hq, int G,
                                                   float scale2) {
  __shared__ float sq[SNAP_ROWS][D];
  __shared__ float2 sml[SNAP_ROWS];
  const SeqDesc &sd = seqs[seq];
  const int n0 = sd.n0, w = sd.w_eff, wfull = sd.window;
  const int chunk = blockIdx.x, h = blockIdx.y;
  const int nchunk = (n0 + SNAP_CHUNK - 1) / SNAP_CHUNK;
  const int j = chunk * SNAP_CHUNK + (int)threadIdx.x;
  const uint16_t *ks = reinterpret_cast<const uint16_t *>(sd.stage_k) + h * stride_stage(sd, D);
  float kr[D];
  load_key_row<D>(ks, j, n0, kr);
  const int rows = w * G;
  const float2 *part = reinterpret_cast<const float2 *>(sd.aux1) + (size_t)h * rows * nchunk * 4;
  float vote = 0.f;
  for (int r0 = 0; r0 < rows; r0 += SNAP_ROWS) {
    const int nr = min(SNAP_ROWS, rows - r0);
    __syncthreads();
    load_window<D>(sq, qw, h, G, Hq, w, wfull, r0, nr);
    for (int rr = threadIdx.x; rr < nr; rr += NT) {
      const float2 *pp = part + (size_t)(r0 + rr) * nchunk * 4;
      float M = -INFINITY;
      for (int e = 0; e < nchunk * 4; ++e) M = fmaxf(M, pp[e].x);
      float L = 0.f;
      for (int e = 0; e < nchunk * 4; ++e)
        if (pp[e].x != -INFINITY) L += pp[e].y * exp2f(pp[e].x - M);
      sml[rr] = make_float2(M, L);
    }
    __syncthreads();
    for (int rr = 0; rr < nr; ++rr) {
      const int r = r0 + rr, i = r / G;
      const int posr = n0 - w + i;
      float acc = 0.f;
#pragma unroll
      for (int c = 0; c < D; ++c) acc = fmaf(sq[rr][c], kr[c], acc);
      if (j <= posr && j < n0) vote += exp2f(acc * scale2 - sml[rr].x) / sml[rr].y;
    }
  }
  if (j < n0 - w) (reinterpret_cast<float *>(sd.aux0) + (size_t)h * n0)[j] = vote;
}

template <int D>
__global__ __launch_bounds__(NT) void k_snap_keep(const SeqDesc *__restrict__ seqs, int seq, int32_t *state,
                                                  int Hkv) {
  __shared__ int hist[256];
  __shared__ int s3[3];
  __shared__ int s_tmp[NT / 64];
  const SeqDesc &sd = seqs[seq];
  const int h = blockIdx.x, n0 = sd.n0, w = sd.w_eff;
  const bool all = sd.T >= n0;
  const int ncand = all ? 0 : n0 - w;
  const int want = all ? 0 : sd.T - w;
  const float *votes = reinterpret_cast<const float *>(sd.aux0) + (size_t)h * n0;
  const int half = sd.pool / 2;
  auto pooled = [&](int j) {
    float m = votes[j];
    const int lo = max(0, j - half), hi = min(ncand - 1, j + half);
    for (int x = lo; x <= hi; ++x) m = fmaxf(m, votes[x]);
    return float_key(m);
  };
  uint32_t kth = 0xFFFFFFFFu;
  int n_eq = 0, need = 0;
  if (want > 0) radix_select_kth<NT>(ncand, want, pooled, hist, s3, &kth, &n_eq, &need);
  const uint16_t *sk = reinterpret_cast<const uint16_t *>(sd.stage_k) + h * stride_stage(sd, D);
  const uint16_t *sv = reinterpret_cast<const uint16_t *>(sd.stage_v) + h * stride_stage(sd, D);
  uint16_t *dk = reinterpret_cast<uint16_t *>(sd.k) + h * stride_rows(sd, D);
  uint16_t *dvv = reinterpret_cast<uint16_t *>(sd.v) + h * stride_rows(sd, D);
  uint16_t *kcm = reinterpret_cast<uint16_t *>(sd.kcm) + h * stride_kcm(sd, D);
  int32_t *pos = reinterpret_cast<int32_t *>(sd.pos) + h * stride_slots(sd);
  const int cap = sd.cap, cstride = sd.cstride;
  const int kept = compact_ascending(
      n0,
      [&](int j, int eq_before) {
        if (all || j >= ncand) return true;
        if (want == 0) return false;
        const uint32_t kk = pooled(j);
        return kk > kth || (kk == kth && eq_before < need);
      },
      [&](int j) { return !all && want > 0 && j < ncand && pooled(j) == kth; },
      [&](int j, int slot) {
        if (slot >= cap) return;
        pos[slot] = j;
        for (int c = 0; c < D; c += 8) {
          const uint4 a = *reinterpret_cast<const uint4 *>(sk + (size_t)j * D + c);
          *reinterpret_cast<uint4 *>(dk + (size_t)slot * D + c) = a;
          *reinterpret_cast<uint4 *>(dvv + (size_t)slot * D + c) = *reinterpret_cast<const uint4 *>(sv + (size_t)j * D + c);
          const uint32_t wv[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
          for (int e = 0; e < 8; ++e) kcm[(size_t)(c + e) * cstride + slot] = (uint16_t)(wv[e / 2] >> (16 * (e & 1)));
        }
      },
      s_tmp);
  if (threadIdx.x == 0) {
    int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
    st[ST_COUNT] = kept;
    st[ST_KEPT] = kept;
  }
}

template <int D, int G>
hipError_t topk_impl(const Dev &dv, const Shape &sh, const uint16_t *q, int32_t *pos_out, int topk_max,
                     hipStream_t st, LaunchEv ev) {
  hipExtLaunchKernelGGL((k_topk<D, G>), dim3(sh.S * sh.Hkv), dim3(kTopkThreads), 0, st, ev.start, ev.stop, 0,
                        dv.seqs, dv.state, q, pos_out, topk_max, sh.Hkv);
  return hipGetLastError();
}

template <int D>
hipError_t h2o_prefill_impl(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq, const uint16_t *q,
                            hipStream_t st) {
  const float scale2 = kLog2e / sqrtf((float)D);
  const int nb = (hs.n0 + TB - 1) / TB;
  hipLaunchKernelGGL(k_h2o_rowstats<D>, dim3(nb, sh.Hq), dim3(NT), 0, st, dv.seqs, seq, q, sh.Hq, sh.G, scale2);
  hipLaunchKernelGGL(k_h2o_colsums<D>, dim3(nb, sh.Hkv), dim3(NT), 0, st, dv.seqs, seq, q, sh.Hq, sh.G, scale2);
  hipLaunchKernelGGL(k_h2o_keep<D>, dim3(sh.Hkv), dim3(NT), 0, st, dv.seqs, seq, dv.state, sh.Hkv);
  return hipGetLastError();
}

template <int D>
hipError_t snap_prefill_impl(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq, const uint16_t *qw,
                             hipStream_t st) {
  const float scale2 = kLog2e / sqrtf((float)D);
  if (hs.T < hs.n0) {
    const int nchunk = (hs.n0 + SNAP_CHUNK - 1) / SNAP_CHUNK;
    hipLaunchKernelGGL(k_snap_rowstats<D>, dim3(nchunk, sh.Hkv), dim3(NT), 0, st, dv.seqs, seq, qw, sh.Hq, sh.G,
                       scale2);
    hipLaunchKernelGGL(k_snap_votes<D>, dim3(nchunk, sh.Hkv), dim3(NT), 0, st, dv.seqs, seq, qw, sh.Hq, sh.G,
                       scale2);
  }
  hipLaunchKernelGGL(k_snap_keep<D>, dim3(sh.Hkv), dim3(NT), 0, st, dv.seqs, seq, dv.state, sh.Hkv);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_topk(const Dev &dv, const Shape &sh, const uint16_t *q, int32_t *pos_out, int topk_max,
                       hipStream_t st, LaunchEv ev) {
  switch (sh.D * 16 + sh.G) {
    case 64 * 16 + 1: return topk_impl<64, 1>(dv, sh, q, pos_out, topk_max, st, ev);
    case 64 * 16 + 2: return topk_impl<64, 2>(dv, sh, q, pos_out, topk_max, st, ev);
    case 64 * 16 + 4: return topk_impl<64, 4>(dv, sh, q, pos_out, topk_max, st, ev);
    case 64 * 16 + 8: return topk_impl<64, 8>(dv, sh, q, pos_out, topk_max, st, ev);
    case 128 * 16 + 1: return topk_impl<128, 1>(dv, sh, q, pos_out, topk_max, st, ev);
    case 128 * 16 + 2: return topk_impl<128, 2>(dv, sh, q, pos_out, topk_max, st, ev);
    case 128 * 16 + 4: return topk_impl<128, 4>(dv, sh, q, pos_out, topk_max, st, ev);
    case 128 * 16 + 8: return topk_impl<128, 8>(dv, sh, q, pos_out, topk_max, st, ev);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_h2o_prefill_seq(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq,
                                  const uint16_t *q_rows, hipStream_t st) {
  return sh.D == 64 ? h2o_prefill_impl<64>(dv, sh, hs, seq, q_rows, st)
                    : h2o_prefill_impl<128>(dv, sh, hs, seq, q_rows, st);
}

hipError_t launch_snap_prefill_seq(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq,
                                   const uint16_t *q_window, hipStream_t st) {
  return sh.D == 64 ? snap_prefill_impl<64>(dv, sh, hs, seq, q_window, st)
                    : snap_prefill_impl<128>(dv, sh, hs, seq, q_window, st);
}

}  // namespace mkv
