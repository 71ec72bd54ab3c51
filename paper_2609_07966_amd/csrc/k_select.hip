// Token-selection kernels: RocketKV top-k, H2O eviction, H2O and SnapKV prefill eviction.
//
// MetaKV Section 2.1: H2O keeps the tokens with the highest accumulated attention and evicts the
// lowest-scoring older token once over budget; RocketKV first keeps the prompt tokens the
// observation window votes for (SnapKV), then attends to a top-k subset per decode step.
// Selections are block-wide radix selects on order-preserving 32-bit keys followed by an
// ascending-position compaction, so ties resolve by position exactly as specified.
#include "select_dev.h"

namespace mkv {

namespace {

constexpr int NT = 256;

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
// One workgroup of kTopkThreads threads per (sequence, kv head) over the tokens already appended
// (a decode step instead spreads the scores over several workgroups, in k_append.hip).
template <int D, int G>
__global__ __launch_bounds__(kTopkThreads, 8) void k_topk(const SeqDesc *__restrict__ seqs, int32_t *state,
                                                       const uint16_t *__restrict__ q, int32_t *pos_out,
                                                       int topk_max, int Hkv) {
  __shared__ TopkLds<D> L;
  const int seq = blockIdx.x / Hkv, h = blockIdx.x % Hkv;
  const SeqDesc &sd = seqs[seq];
  if (sd.method != ROCKET) return;
  int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  topk_pair<D, G>(sd, st, seq, h, Hkv, st[ST_COUNT], q, pos_out, topk_max, L);
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
  // no eviction candidates before the first attention pass
  uint32_t *vb = reinterpret_cast<uint32_t *>(sd.vbest) + (size_t)h * sd.vparts * 4;
  for (int p = threadIdx.x; p < sd.vparts; p += NT) {
    vb[4 * p] = 0xFFFFFFFFu;
    vb[4 * p + 1] = 0xFFFFFFFFu;
    vb[4 * p + 2] = 0xFFFFFFFFu;
    vb[4 * p + 3] = 0u;
  }
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
