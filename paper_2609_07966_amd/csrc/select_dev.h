// RocketKV decode-time top-k, device side: the channel pick, the approximate scores and the
// selection, shared by the stand-alone top-k launch and the two launches a decode step uses
// (scores spread over several workgroups per kv head, then one selecting workgroup per kv head).
//
// MetaKV Section 2.1 (RocketKV): after the SnapKV prefill eviction every decode step attends to a
// top-k subset of the retained tokens, chosen by approximate scores over a few query channels.
// The channels are the nch largest of sum_g |q_g,c| (ties to the lower channel); a token's score
// is sum over those channels, ascending, of (sum_g q_g,c) * k_c, every product and sum rounded to
// float32 separately; the k best scores are kept (ties to the lower slot) and listed in ascending
// slot order.
#pragma once

#include "kernels_common.h"

namespace mkv {

namespace {

constexpr int kTopkThreads = 1024;   // the selecting workgroup (and the stand-alone top-k)
constexpr int kScoreThreads = 256;   // a scoring workgroup: 4 tokens per thread
constexpr int kScoreTokens = kScoreTokensPerPart;  // tokens per scoring workgroup, 4 per thread
static_assert(kScoreTokens == 4 * kScoreThreads, "a scoring thread takes 4 tokens");
constexpr int kTopkLdsKeys = 10240;  // stand-alone top-k: score keys of up to this many tokens in LDS
constexpr int kTopkHists = 4;        // digit histograms; waves w, w + 4, w + 8, ... share one
constexpr int kRegKeys = 8;          // keys a decode-step selecting thread holds in registers

// The channel pick of a workgroup of NTH threads.
template <int D, int NTH>
struct ChanLds {
  float a[D];
  float qb[D];
  int beats[NTH];
  int wcnt[(D + 63) / 64];
  int sel_ch[D];
  float sel_qb[D];
  uint16_t knew[D];  // the key of a token appended in the same launch (fp16 bits)
};

struct SelLds {
  __attribute__((aligned(16))) int hist[2][kTopkHists][256];
  int s3[3];
  int tmp[kTopkThreads / 64];
};

template <int D>
struct TopkLds {
  ChanLds<D, kTopkThreads> c;
  SelLds s;
  uint32_t keys[kTopkLdsKeys];
};

// Query channel tid (tid < D; other threads read channel D - 1 and ignore it) of each of the G
// rows of the kv head's query group qh; loaded by the caller before anything it waits on.
template <int D, int G>
MKV_DEV void load_qcol(const uint16_t *qh, uint16_t (&qr)[G]) {
  const int c = min((int)threadIdx.x, D - 1);
#pragma unroll
  for (int g = 0; g < G; ++g) qr[g] = gld(qh + (size_t)g * D + c);
}

// The nch channels of a kv head's query group (thread c < D holds channel c of its G rows, from
// load_qcol) into L.sel_ch / L.sel_qb in ascending channel order; returns nch.  Ends with a
// barrier.
template <int D, int G, int NTH>
MKV_DEV int channel_pick(const SeqDesc &sd, const uint16_t (&qr)[G], ChanLds<D, NTH> &L) {
  static_assert(NTH % D == 0, "whole slices per channel");
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  // channel magnitudes and head sums, float32 in ascending head order
  if (tid < D) {
    float a = 0.f, qb = 0.f;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float x = h2f(qr[g]);
      a = __fadd_rn(a, fabsf(x));
      qb = __fadd_rn(qb, x);
    }
    L.a[tid] = a;
    L.qb[tid] = qb;
  }
  __syncthreads();
  const int nch = min(sd.nch, D);
  // channel c is selected iff fewer than nch channels beat it (larger a, or equal a and lower
  // index); the NTH / D threads of channel c each count a slice of the others
  {
    constexpr int P = NTH / D, W = D / P;
    const int c = tid % D, part = tid / D;
    const float a = L.a[c];
    int beats = 0;
#pragma unroll
    for (int i = 0; i < W; ++i) {
      const int c2 = part * W + i;
      const float b = L.a[c2];
      beats += (b > a || (b == a && c2 < c)) ? 1 : 0;
    }
    L.beats[tid] = beats;
  }
  __syncthreads();
  // ascending compaction of the selected channels: rank = selected channels below c
  bool f = false;
  if (tid < D) {
    int t = 0;
#pragma unroll
    for (int p = 0; p < NTH / D; ++p) t += L.beats[p * D + tid];
    f = t < nch;
  }
  const uint64_t m = __ballot(f);
  if (tid < D && lane == 0) L.wcnt[wid] = __popcll(m);
  __syncthreads();
  if (f) {
    int r = __popcll(m & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
    for (int i = 0; i < wid; ++i) r += L.wcnt[i];
    L.sel_ch[r] = tid;
    L.sel_qb[r] = L.qb[tid];
  }
  __syncthreads();
  return nch;
}

// Approximate scores of the T consecutive tokens [j0, j0 + T) (T = 4 or 8) from the channel-major
// key copy: one 2T-byte load per selected channel, R channels' loads issued before any is used,
// channels ascending, every product and sum rounded to fp32 separately (no fused multiply-add).
// Token jn, if in range, takes its key from `knew` (LDS) instead of the copy.  Rows are padded to
// 8 tokens and j0 is a multiple of T, so no load leaves its row.
template <int T, int R>
MKV_DEV void score_tokens(const uint16_t *kcm, int cstride, int j0, int nch, const int *sel_ch, const float *sel_qb,
                          int jn, const uint16_t *knew, float (&acc)[T]) {
#pragma unroll
  for (int t = 0; t < T; ++t) acc[t] = 0.f;
  const bool patch = jn >= j0 && jn < j0 + T;  // true in one thread at most
  for (int i0 = 0; i0 < nch; i0 += R) {
    uint32_t w[R][T / 2];
#pragma unroll
    for (int ii = 0; ii < R; ++ii) {
      const int i = min(i0 + ii, nch - 1);
      const uint32_t *p = reinterpret_cast<const uint32_t *>(kcm + (size_t)sel_ch[i] * cstride + j0);
#pragma unroll
      for (int u = 0; u < T / 2; ++u) w[ii][u] = gld(p + u);
    }
    if (patch) {
      const int t = jn - j0;
#pragma unroll
      for (int ii = 0; ii < R; ++ii) {
        const uint32_t kb = knew[sel_ch[min(i0 + ii, nch - 1)]];
#pragma unroll
        for (int u = 0; u < T / 2; ++u) {
          if (t == 2 * u) w[ii][u] = (w[ii][u] & 0xFFFF0000u) | kb;
          if (t == 2 * u + 1) w[ii][u] = (w[ii][u] & 0xFFFFu) | (kb << 16);
        }
      }
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

// The k largest of the n keys src(j) (1 <= k < n; order-preserving keys, ties to the lower
// index) by a workgroup of NTH threads: their indices go to sel[0..k) in ascending order.
// Thread t owns the run [t per, t per + per) (per = ceil(n / NTH)) and holds its keys in
// registers when per <= KR (else re-reads src in every pass).  The k-th key comes from 4
// radix passes of 8 bits: digit counts go to kTopkHists LDS histograms by atomics (one per run of
// equal digits in a thread's keys), and wave 0
// finds the digit by a scan over lanes while the other waves clear the next pass's histogram set
// (2 barriers per pass).  Then counts of keys above and equal to the threshold before each run,
// by one block scan, place every thread's selected indices.  Keys written by other threads of the
// workgroup must be visible on entry.
template <int NTH, int KR = kRegKeys, typename Src>
MKV_DEV void select_keys(int n, int k, Src src, int32_t *sel, SelLds &L) {
  const int tid = threadIdx.x, wid = tid >> 6, lane = tid & 63;
  const int per = (n + NTH - 1) / NTH;
  const int ja = min(n, tid * per), m = min(n, ja + per) - ja;
  const bool regs = per <= KR;  // block-uniform
  uint32_t kr[KR];
#pragma unroll
  for (int u = 0; u < KR; ++u) kr[u] = (regs && u < m) ? src(ja + u) : 0u;
  // f(u, key) over this thread's keys in index order
  auto each = [&](auto f) {
    if (regs) {
#pragma unroll
      for (int u = 0; u < KR; ++u)
        if (u < m) f(u, kr[u]);
    } else {
      for (int u = 0; u < m; ++u) f(u, src(ja + u));
    }
  };
  for (int e = tid; e < kTopkHists * 256; e += NTH) (&L.hist[0][0][0])[e] = 0;
  __syncthreads();
  uint32_t prefix = 0, mask = 0;
  int remaining = k;
  for (int pass = 0; pass < 4; ++pass) {
    const int buf = pass & 1, shift = 24 - 8 * pass;
    int *hw = L.hist[buf][wid % kTopkHists];
    // a thread's consecutive keys often share the digit (the leading digits of similar scores
    // coincide): one atomic per run of equal digits
    int run_d = 0, run_c = 0;
    each([&](int, uint32_t key) {
      if ((key & mask) == prefix) {
        const int d = (int)((key >> shift) & 255u);
        if (run_c > 0 && d != run_d) {
          atomicAdd(&hw[run_d], run_c);
          run_c = 0;
        }
        run_d = d;
        ++run_c;
      }
    });
    if (run_c > 0) atomicAdd(&hw[run_d], run_c);
    __syncthreads();
    if (wid == 0) {
      // lane l owns digits 255 - 4l .. 252 - 4l (descending), so the exclusive scan over lanes
      // gives the count of larger digits
      int cnt[4] = {0, 0, 0, 0};
#pragma unroll
      for (int w = 0; w < kTopkHists; ++w) {
        const int4 c4 = *reinterpret_cast<const int4 *>(&L.hist[buf][w][252 - 4 * lane]);
        cnt[0] += c4.w;
        cnt[1] += c4.z;
        cnt[2] += c4.y;
        cnt[3] += c4.x;
      }
      const int tot = cnt[0] + cnt[1] + cnt[2] + cnt[3];
      int above = wave_incl_scan(tot) - tot;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (above < remaining && remaining <= above + cnt[i]) {
          L.s3[0] = 255 - (4 * lane + i);
          L.s3[1] = remaining - above;
        }
        above += cnt[i];
      }
    } else {
      for (int e = tid - 64; e < kTopkHists * 256; e += NTH - 64) (&L.hist[buf ^ 1][0][0])[e] = 0;
    }
    __syncthreads();
    prefix |= (uint32_t)L.s3[0] << shift;
    mask |= 255u << shift;
    remaining = L.s3[1];
  }
  const uint32_t kth = prefix;
  const int need = remaining;  // keys equal to kth that are taken (the lowest indices)
  int gt = 0, eq = 0;
  each([&](int, uint32_t key) {
    gt += key > kth ? 1 : 0;
    eq += key == kth ? 1 : 0;
  });
  // one scan of both counts when n < 2^15 keeps them apart in the two halves of a word
  int tot, gt_before, eq_run;
  if (n < 32768) {
    const int both = block_exclusive_scan<NTH>((gt << 16) | eq, L.tmp, &tot);
    gt_before = both >> 16;
    eq_run = both & 0xFFFF;
  } else {
    gt_before = block_exclusive_scan<NTH>(gt, L.tmp, &tot);
    eq_run = block_exclusive_scan<NTH>(eq, L.tmp, &tot);
  }
  int slot = gt_before + min(eq_run, need);
  each([&](int u, uint32_t key) {
    const bool take = key > kth || (key == kth && eq_run < need);
    eq_run += key == kth ? 1 : 0;
    if (take && slot < k) gst(sel + slot, ja + u);
    slot += take ? 1 : 0;
  });
}

// ---- a decode step's scoring workgroups -----------------------------------------------------------
// Part `part` of a RocketKV (sequence, kv head) with n retained tokens (the new one included):
// the channel pick (every part makes it, from the query channels qr; part 0 also writes it out)
// and the scores of tokens [part kScoreTokens, (part + 1) kScoreTokens), as keys into the
// head's global key array.
// L.knew must hold the new token's key (token n - 1) when `has_new`; the pick's barriers publish it.
template <int D, int G>
MKV_DEV void score_part(const SeqDesc &sd, int h, int n, int part, bool has_new, const uint16_t (&qr)[G],
                        ChanLds<D, kScoreThreads> &L) {
  const int tid = threadIdx.x;
  const int nch = channel_pick<D, G, kScoreThreads>(sd, qr, L);
  if (part == 0)
    for (int i = tid; i < nch; i += kScoreThreads) (reinterpret_cast<int32_t *>(sd.aux1) + (size_t)h * D)[i] = L.sel_ch[i];
  if (sd.topk >= n) return;  // every token is selected; no scores needed
  const uint16_t *kcm = reinterpret_cast<const uint16_t *>(sd.kcm) + h * stride_kcm(sd, D);
  uint32_t *akeys = reinterpret_cast<uint32_t *>(sd.akeys) + h * stride_slots(sd);
  const int j0 = part * kScoreTokens + 4 * tid;
  if (j0 >= n) return;
  float acc[4];
  score_tokens<4, 32>(kcm, sd.cstride, j0, nch, L.sel_ch, L.sel_qb, has_new ? n - 1 : -1, L.knew, acc);
#pragma unroll
  for (int r = 0; r < 4; ++r)
    if (j0 + r < n) gst(akeys + j0 + r, float_key(acc[r]));
}

// ---- the stand-alone top-k: one workgroup of kTopkThreads threads per (sequence, kv head) -------
// Over the n tokens already appended; with pos_out, also the selected positions (topk_max per
// pair, -1 padded).  Writes the chosen channels, the selected slots and ST_SEL_COUNT.
template <int D, int G>
MKV_DEV void topk_pair(const SeqDesc &sd, int32_t *st, int seq, int h, int Hkv, int n, const uint16_t *q,
                       int32_t *pos_out, int topk_max, TopkLds<D> &L) {
  constexpr int NTH = kTopkThreads;
  const int tid = threadIdx.x;
  const int k = sd.topk;
  int32_t *sel = reinterpret_cast<int32_t *>(sd.sel) + h * stride_sel(sd);
  const int32_t *pos = reinterpret_cast<const int32_t *>(sd.pos) + h * stride_slots(sd);
  uint16_t qr[G];
  load_qcol<D, G>(q + ((size_t)seq * Hkv * G + h * G) * D, qr);
  const int nch = channel_pick<D, G, NTH>(sd, qr, L.c);
  for (int i = tid; i < nch; i += NTH) (reinterpret_cast<int32_t *>(sd.aux1) + (size_t)h * D)[i] = L.c.sel_ch[i];
  if (k >= n) {
    for (int j = tid; j < n; j += NTH) sel[j] = j;
    if (pos_out != nullptr)
      for (int i = tid; i < topk_max; i += NTH)
        pos_out[((size_t)seq * Hkv + h) * topk_max + i] = i < n ? pos[i] : -1;
    if (tid == 0) st[ST_SEL_COUNT] = n;
    return;
  }
  // approximate scores; the keys stay in LDS when they fit.  A lane scores 4 consecutive tokens
  // (8 for sets of more than 4 NTH tokens, so that one pass covers up to 8 NTH)
  const uint16_t *kcm = reinterpret_cast<const uint16_t *>(sd.kcm) + h * stride_kcm(sd, D);
  uint32_t *akeys = reinterpret_cast<uint32_t *>(sd.akeys) + h * stride_slots(sd);
  const bool in_lds = n <= kTopkLdsKeys;
  auto put = [&](int j, float a) {
    if (j < n) {
      if (in_lds) L.keys[j] = float_key(a);
      else gst(akeys + j, float_key(a));
    }
  };
  if (n <= 4 * NTH) {
    const int j0 = 4 * tid;
    if (j0 < n) {
      float acc[4];
      score_tokens<4, 16>(kcm, sd.cstride, j0, nch, L.c.sel_ch, L.c.sel_qb, -1, nullptr, acc);
#pragma unroll
      for (int r = 0; r < 4; ++r) put(j0 + r, acc[r]);
    }
  } else {
    for (int j0 = 8 * tid; j0 < n; j0 += 8 * NTH) {
      float acc[8];
      score_tokens<8, 8>(kcm, sd.cstride, j0, nch, L.c.sel_ch, L.c.sel_qb, -1, nullptr, acc);
#pragma unroll
      for (int r = 0; r < 8; ++r) put(j0 + r, acc[r]);
    }
  }
  __syncthreads();
  select_keys<NTH>(n, k, [&](int j) { return in_lds ? L.keys[j] : gld(akeys + j); }, sel, L.s);
  if (pos_out != nullptr) {
    __syncthreads();
    for (int i = tid; i < topk_max; i += NTH)
      pos_out[((size_t)seq * Hkv + h) * topk_max + i] = i < k ? gld(pos + gld(sel + i)) : -1;
  }
  if (tid == 0) st[ST_SEL_COUNT] = k;
}

}  // namespace

}  // namespace mkv
