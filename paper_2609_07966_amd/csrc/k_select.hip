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
// gathered into slots 0..kept-1 in ascending position order.  The selection runs over the
// candidates in reverse order (index ncand - 1 - j), so that its lower-index tie rule prefers
// newer tokens; its ascending output, reversed, is ascending in position.
template <int D>
__global__ __launch_bounds__(kTopkThreads) void k_h2o_keep(const SeqDesc *__restrict__ seqs, int seq, int32_t *state,
                                                           int Hkv) {
  __shared__ SelLds L;
  const SeqDesc &sd = seqs[seq];
  const int h = blockIdx.x, n0 = sd.n0;
  const float *S = reinterpret_cast<const float *>(sd.aux0) + (size_t)h * n0;
  const int B = sd.B, R = sd.R;
  const bool all = B >= n0;
  const int ncand = all ? 0 : n0 - R;
  const int H = all ? 0 : B - R;
  const int kept = all ? n0 : min(B, sd.cap);
  int32_t *pos = reinterpret_cast<int32_t *>(sd.pos) + h * stride_slots(sd);
  if (all) {
    for (int j = threadIdx.x; j < n0; j += kTopkThreads) pos[j] = j;
  } else {
    if (H > 0) {
      // the scratch of the row statistics (no longer needed) takes the reversed selection
      int32_t *rsel = reinterpret_cast<int32_t *>(sd.aux1) + (size_t)h * n0;
      select_keys<kTopkThreads, 32>(ncand, H, [&](int i) { return float_key(gld(S + (ncand - 1 - i))); }, rsel, L);
      __syncthreads();
      for (int i = threadIdx.x; i < H; i += kTopkThreads) pos[H - 1 - i] = ncand - 1 - gld(rsel + i);
    }
    for (int i = threadIdx.x; i < R; i += kTopkThreads) pos[H + i] = ncand + i;
  }
  __syncthreads();
  const uint16_t *sk = reinterpret_cast<const uint16_t *>(sd.stage_k) + h * stride_stage(sd, D);
  const uint16_t *sv = reinterpret_cast<const uint16_t *>(sd.stage_v) + h * stride_stage(sd, D);
  uint16_t *dk = reinterpret_cast<uint16_t *>(sd.k) + h * stride_rows(sd, D);
  uint16_t *dvv = reinterpret_cast<uint16_t *>(sd.v) + h * stride_rows(sd, D);
  float *score = reinterpret_cast<float *>(sd.score) + h * stride_slots(sd);
  for (int it = threadIdx.x; it < kept * (D / 8); it += kTopkThreads) {
    const int slot = it / (D / 8), u = it % (D / 8);
    const int j = gld(pos + slot);
    *reinterpret_cast<uint4 *>(dk + (size_t)slot * D + 8 * u) = gld16(sk + (size_t)j * D + 8 * u);
    *reinterpret_cast<uint4 *>(dvv + (size_t)slot * D + 8 * u) = gld16(sv + (size_t)j * D + 8 * u);
    if (u == 0) score[slot] = gld(S + j);
  }
  // no eviction candidates before the first attention pass
  uint32_t *vb = reinterpret_cast<uint32_t *>(sd.vbest) + (size_t)h * sd.vparts * 4;
  for (int p = threadIdx.x; p < sd.vparts; p += kTopkThreads) {
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
// Window row r = i * G + g (query head h*G + g at position n0 - w + i; it attends to keys
// 0 .. n0 - w + i).  Pass 1: per 256-key chunk and wave, the partial (max, sum of exp2) of every
// row, from v_mfma_f32_16x16x32_f16 logit tiles.  Pass 2: each row's partials merged.  Pass 3: the
// votes of a chunk's keys, the logits recomputed on the matrix cores.  Pass 4: max pooling into
// order-preserving keys.  Pass 5: select, gather the kept rows.
constexpr int SNAP_CHUNK = 256;  // keys per workgroup: 64 per wave, 4 key tiles of 16
constexpr int SNAP_ROWS = 64;    // window rows staged in LDS at a time (4 row tiles of 16)

// The window rows [r0, r0 + 64) (clamped to the last row) as fp16 operands in LDS.
template <int D>
MKV_DEV void stage_window(uint4 (*sq)[D / 8 + 1], const uint16_t *qw, int h, int G, int Hq, int w, int wfull,
                          int rows, int r0) {
  constexpr int U = D / 8;
  for (int e = threadIdx.x; e < SNAP_ROWS * U; e += NT) {
    const int rr = e / U, u = e % U;
    const int r = min(r0 + rr, rows - 1), i = r / G, g = r % G;
    // the last w of the `wfull` window rows
    sq[rr][u] = gld16(reinterpret_cast<const uint4 *>(qw + ((size_t)(wfull - w + i) * Hq + h * G + g) * D) + u);
  }
}

// A wave's 4 key tiles (16 keys each) of the chunk as matrix operands: key 16 n + lr, channels
// 8 lq .. 8 lq + 7 of k-step s.
template <int D>
MKV_DEV void snap_key_operands(const uint16_t *ks, int key0, int n0, uint4 (&kop)[4][D / 32]) {
  constexpr int U = D / 8;
  const int lane = threadIdx.x & 63, lr = lane & 15, lq = lane >> 4;
#pragma unroll
  for (int n = 0; n < 4; ++n)
#pragma unroll
    for (int s = 0; s < D / 32; ++s)
      kop[n][s] = gld16(reinterpret_cast<const uint4 *>(ks) + (size_t)min(key0 + 16 * n + lr, n0 - 1) * U + 4 * s + lq);
}

template <int D>
__global__ __launch_bounds__(NT) void k_snap_rowstats(const SeqDesc *__restrict__ seqs, int seq,
                                                      const uint16_t *__restrict__ qw, int Hq, int G,
                                                      float scale2) {
  constexpr int KS = D / 32;
  __shared__ uint4 sq[SNAP_ROWS][D / 8 + 1];
  const SeqDesc &sd = seqs[seq];
  const int n0 = sd.n0, w = sd.w_eff, wfull = sd.window;
  const int chunk = blockIdx.x, h = blockIdx.y;
  const int nchunk = (n0 + SNAP_CHUNK - 1) / SNAP_CHUNK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, lr = lane & 15, lq = lane >> 4;
  const int key0 = chunk * SNAP_CHUNK + 64 * wave;
  uint4 kop[4][KS];
  snap_key_operands<D>(reinterpret_cast<const uint16_t *>(sd.stage_k) + h * stride_stage(sd, D), key0, n0, kop);
  const int rows = w * G;
  float2 *part = reinterpret_cast<float2 *>(sd.aux1) + (size_t)h * rows * nchunk * 4;
  for (int r0 = 0; r0 < rows; r0 += SNAP_ROWS) {
    __syncthreads();
    stage_window<D>(sq, qw, h, G, Hq, w, wfull, rows, r0);
    __syncthreads();
#pragma unroll 1
    for (int t = 0; t < SNAP_ROWS / 16 && r0 + 16 * t < rows; ++t) {
      float v[4][4];
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        f4v S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) S = mfma_k32(sq[16 * t + lr][4 * s + lq], kop[n][s], S);
        const int key = key0 + 16 * n + lr;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int r = r0 + 16 * t + 4 * lq + j, posr = n0 - w + r / G;
          v[n][j] = (key <= posr && key < n0) ? S[j] * scale2 : -INFINITY;
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float M = row16_max(fmaxf(fmaxf(v[0][j], v[1][j]), fmaxf(v[2][j], v[3][j])));
        float e = 0.f;
        if (M != -INFINITY) {
#pragma unroll
          for (int n = 0; n < 4; ++n) e += fexp2(v[n][j] - M);  // arguments <= 0
        }
        const float L = row16_sum(e);
        const int r = r0 + 16 * t + 4 * lq + j;
        if (lr == 0 && r < rows) part[((size_t)r * nchunk + chunk) * 4 + wave] = make_float2(M, L);
      }
    }
  }
}

// Merge each window row's 4 nchunk partials (one wave per row); entry 0 of the row then holds
// (max, sum of exp2) over all its keys.
template <int D>
__global__ __launch_bounds__(NT) void k_snap_merge(const SeqDesc *__restrict__ seqs, int seq, int G) {
  const SeqDesc &sd = seqs[seq];
  const int n0 = sd.n0, rows = sd.w_eff * G, h = blockIdx.y;
  const int nchunk = (n0 + SNAP_CHUNK - 1) / SNAP_CHUNK, np = 4 * nchunk;
  const int lane = threadIdx.x & 63, r = blockIdx.x * (NT / 64) + (threadIdx.x >> 6);
  if (r >= rows) return;
  float2 *pr = reinterpret_cast<float2 *>(sd.aux1) + ((size_t)h * rows + r) * np;
  float m = -INFINITY, l = 0.f;
  for (int e = lane; e < np; e += 64) {
    const float xm = gld(reinterpret_cast<const float *>(pr + e)), xl = gld(reinterpret_cast<const float *>(pr + e) + 1);
    if (xm == -INFINITY) continue;
    const float mx = fmaxf(m, xm);
    l = l * fexp2(m - mx) + xl * fexp2(xm - mx);  // arguments <= 0 (m = -inf gives 0)
    m = mx;
  }
  const float M = wave_max(m);
  const float L = wave_sum(m == -INFINITY ? 0.f : l * fexp2(m - M));
  if (lane == 0) pr[0] = make_float2(M, L);
}

// Votes of a chunk's keys: sum over the window rows of exp2(s - M_r) / L_r.
template <int D>
__global__ __launch_bounds__(NT) void k_snap_votes(const SeqDesc *__restrict__ seqs, int seq,
                                                   const uint16_t *__restrict__ qw, int Hq, int G,
                                                   float scale2) {
  constexpr int KS = D / 32;
  __shared__ uint4 sq[SNAP_ROWS][D / 8 + 1];
  __shared__ float2 sml[SNAP_ROWS];  // (M, 1 / L) of the staged rows
  const SeqDesc &sd = seqs[seq];
  const int n0 = sd.n0, w = sd.w_eff, wfull = sd.window;
  const int chunk = blockIdx.x, h = blockIdx.y;
  const int nchunk = (n0 + SNAP_CHUNK - 1) / SNAP_CHUNK;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, lr = lane & 15, lq = lane >> 4;
  const int key0 = chunk * SNAP_CHUNK + 64 * wave;
  uint4 kop[4][KS];
  snap_key_operands<D>(reinterpret_cast<const uint16_t *>(sd.stage_k) + h * stride_stage(sd, D), key0, n0, kop);
  const int rows = w * G;
  const float2 *part = reinterpret_cast<const float2 *>(sd.aux1) + (size_t)h * rows * nchunk * 4;
  float col[4] = {0.f, 0.f, 0.f, 0.f};
  for (int r0 = 0; r0 < rows; r0 += SNAP_ROWS) {
    __syncthreads();
    stage_window<D>(sq, qw, h, G, Hq, w, wfull, rows, r0);
    if (threadIdx.x < SNAP_ROWS) {
      const float *ml = reinterpret_cast<const float *>(part + (size_t)min(r0 + (int)threadIdx.x, rows - 1) * nchunk * 4);
      sml[threadIdx.x] = make_float2(gld(ml), 1.f / gld(ml + 1));
    }
    __syncthreads();
#pragma unroll 1
    for (int t = 0; t < SNAP_ROWS / 16 && r0 + 16 * t < rows; ++t) {
#pragma unroll
      for (int n = 0; n < 4; ++n) {
        f4v S = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) S = mfma_k32(sq[16 * t + lr][4 * s + lq], kop[n][s], S);
        const int key = key0 + 16 * n + lr;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int rr = 16 * t + 4 * lq + j, r = r0 + rr, posr = n0 - w + r / G;
          // arguments <= 0 wherever the row statistics hold this logit
          if (r < rows && key <= posr && key < n0) col[n] += fexp2(S[j] * scale2 - sml[rr].x) * sml[rr].y;
        }
      }
    }
  }
  float *votes = reinterpret_cast<float *>(sd.aux0) + (size_t)h * n0;
#pragma unroll
  for (int n = 0; n < 4; ++n) {
    float x = col[n];
    x += __shfl_xor(x, 16);
    x += __shfl_xor(x, 32);
    const int key = key0 + 16 * n + lr;
    if (lq == 0 && key < n0 - w) votes[key] = x;
  }
}

// Max pooling of the candidates' votes (odd kernel `pool`, clipped to [0, n0 - w)) into
// order-preserving keys, one thread per candidate.
__global__ __launch_bounds__(NT) void k_snap_pool(const SeqDesc *__restrict__ seqs, int seq) {
  const SeqDesc &sd = seqs[seq];
  const int n0 = sd.n0, ncand = n0 - sd.w_eff, h = blockIdx.y, half = sd.pool / 2;
  const int j = blockIdx.x * NT + (int)threadIdx.x;
  if (j >= ncand) return;
  const float *votes = reinterpret_cast<const float *>(sd.aux0) + (size_t)h * n0;
  float m = gld(votes + j);
  const int lo = max(0, j - half), hi = min(ncand - 1, j + half);
  for (int x = lo; x <= hi; ++x) m = fmaxf(m, gld(votes + x));
  gst(reinterpret_cast<uint32_t *>(sd.aux1) + (size_t)h * n0 + j, float_key(m));
}

// Keep the T - w highest pooled votes among the candidates (lower position on a tie) and the w
// window tokens; gather their rows (and the channel-major key copy) into slots 0..kept-1 in
// ascending position order.
template <int D>
__global__ __launch_bounds__(kTopkThreads) void k_snap_keep(const SeqDesc *__restrict__ seqs, int seq,
                                                            int32_t *state, int Hkv) {
  __shared__ SelLds L;
  const SeqDesc &sd = seqs[seq];
  const int h = blockIdx.x, n0 = sd.n0, w = sd.w_eff;
  const bool all = sd.T >= n0;
  const int ncand = n0 - w, want = sd.T - w;
  const int kept = all ? n0 : sd.T;
  int32_t *pos = reinterpret_cast<int32_t *>(sd.pos) + h * stride_slots(sd);
  if (all) {
    for (int j = threadIdx.x; j < n0; j += kTopkThreads) pos[j] = j;
  } else {
    if (want > 0) {
      const uint32_t *keys = reinterpret_cast<const uint32_t *>(sd.aux1) + (size_t)h * n0;
      select_keys<kTopkThreads, 32>(ncand, want, [&](int j) { return gld(keys + j); }, pos, L);
    }
    for (int i = threadIdx.x; i < w; i += kTopkThreads) pos[want + i] = ncand + i;
  }
  __syncthreads();
  // gather: item (16-byte chunk u, slot) with slots consecutive across lanes, so the 2-byte
  // stores into the channel-major copy are coalesced
  const uint16_t *sk = reinterpret_cast<const uint16_t *>(sd.stage_k) + h * stride_stage(sd, D);
  const uint16_t *sv = reinterpret_cast<const uint16_t *>(sd.stage_v) + h * stride_stage(sd, D);
  uint16_t *dk = reinterpret_cast<uint16_t *>(sd.k) + h * stride_rows(sd, D);
  uint16_t *dvv = reinterpret_cast<uint16_t *>(sd.v) + h * stride_rows(sd, D);
  uint16_t *kcm = reinterpret_cast<uint16_t *>(sd.kcm) + h * stride_kcm(sd, D);
  const int cstride = sd.cstride, total = kept * (D / 8);
  // batches of kGather items per thread: every position and row load in flight before the stores
  constexpr int kGather = 8;
  for (int base = threadIdx.x; base < total; base += kGather * kTopkThreads) {
    int jj[kGather];
    uint4 a[kGather], b[kGather];
#pragma unroll
    for (int q = 0; q < kGather; ++q) {
      const int it = min(base + q * kTopkThreads, total - 1);
      jj[q] = gld(pos + it % kept);
    }
#pragma unroll
    for (int q = 0; q < kGather; ++q) {
      const int u = min(base + q * kTopkThreads, total - 1) / kept;
      a[q] = gld16(sk + (size_t)jj[q] * D + 8 * u);
      b[q] = gld16(sv + (size_t)jj[q] * D + 8 * u);
    }
#pragma unroll
    for (int q = 0; q < kGather; ++q) {
      const int it = base + q * kTopkThreads;
      if (it >= total) break;
      const int u = it / kept, slot = it % kept;
      *reinterpret_cast<uint4 *>(dk + (size_t)slot * D + 8 * u) = a[q];
      *reinterpret_cast<uint4 *>(dvv + (size_t)slot * D + 8 * u) = b[q];
      const uint32_t wv[4] = {a[q].x, a[q].y, a[q].z, a[q].w};
#pragma unroll
      for (int e = 0; e < 8; ++e)
        kcm[(size_t)(8 * u + e) * cstride + slot] = (uint16_t)(wv[e / 2] >> (16 * (e & 1)));
    }
  }
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
  // one query head per workgroup: sharing a staged key tile among several heads of a kv head was
  // measured slower (fewer, longer workgroups at lower occupancy)
  hipLaunchKernelGGL(k_h2o_rowstats<D>, dim3(nb, sh.Hq), dim3(NT), 0, st, dv.seqs, seq, q, sh.Hq, sh.G, scale2);
  hipLaunchKernelGGL(k_h2o_colsums<D>, dim3(nb, sh.Hkv), dim3(NT), 0, st, dv.seqs, seq, q, sh.Hq, sh.G, scale2);
  hipLaunchKernelGGL(k_h2o_keep<D>, dim3(sh.Hkv), dim3(kTopkThreads), 0, st, dv.seqs, seq, dv.state, sh.Hkv);
  return hipGetLastError();
}

template <int D>
hipError_t snap_prefill_impl(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq, const uint16_t *qw,
                             hipStream_t st) {
  const float scale2 = kLog2e / sqrtf((float)D);
  if (hs.T < hs.n0) {
    const int nchunk = (hs.n0 + SNAP_CHUNK - 1) / SNAP_CHUNK, rows = hs.w_eff * sh.G;
    hipLaunchKernelGGL(k_snap_rowstats<D>, dim3(nchunk, sh.Hkv), dim3(NT), 0, st, dv.seqs, seq, qw, sh.Hq, sh.G,
                       scale2);
    hipLaunchKernelGGL(k_snap_merge<D>, dim3((rows + NT / 64 - 1) / (NT / 64), sh.Hkv), dim3(NT), 0, st, dv.seqs,
                       seq, sh.G);
    hipLaunchKernelGGL(k_snap_votes<D>, dim3(nchunk, sh.Hkv), dim3(NT), 0, st, dv.seqs, seq, qw, sh.Hq, sh.G,
                       scale2);
    hipLaunchKernelGGL(k_snap_pool, dim3((hs.n0 - hs.w_eff + NT - 1) / NT, sh.Hkv), dim3(NT), 0, st, dv.seqs, seq);
  }
  hipLaunchKernelGGL(k_snap_keep<D>, dim3(sh.Hkv), dim3(kTopkThreads), 0, st, dv.seqs, seq, dv.state, sh.Hkv);
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
