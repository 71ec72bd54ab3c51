// Append and quantize-on-append kernels (prefill and decode).
//
// Every method first writes the new token's key and value into its cache (MetaKV Section 2.1):
// plain fp16 rows (FP16, H2O, RocketKV), uniform 4-bit group codes, or KVQuant-style codes with
// per-channel key thresholds calibrated on the prompt and fp16 outliers.  The quantizer steps are
// written with explicit round-to-nearest float32 operations (__fmul_rn, __fsub_rn, __fdiv_rn)
// so that codes are reproducible bit for bit.
#include "select_dev.h"

namespace mkv {

namespace {

// ---- shared quantizer pieces -----------------------------------------------------------------

MKV_DEV int code_from_mid(float xhat, const float *mid, int nmid) {
  int c = 0;
  for (int i = 0; i < nmid; ++i) c += (xhat > mid[i]) ? 1 : 0;
  return c;
}

// Outlier entry of token slot t (layout in outlier_pack): the (clamped) code stays in the entry.
MKV_DEV uint32_t outlier_entry(uint32_t bits16, int t, int code, int ch) {
  return outlier_pack(bits16 & 0xFFFFu, t, code, ch);
}

// Word w of a packed code row: code i sits at bits [bits*i, bits*i + bits) of the row (bit 0 =
// least significant bit of byte 0), so two consecutive codes form one 2*bits-bit field.
MKV_DEV uint32_t packed_word(const uint8_t *codes, int n, int bits, int w) {
  uint32_t word = 0;
  const int lo = 32 * w;
  const int first = max(0, lo / bits - 1), last = min(n, (lo + 32) / bits + 1);
  for (int i = first; i < last; ++i) {
    const int off = bits * i - lo;
    const uint32_t code = codes[i];
    if (off >= 0 && off < 32) word |= code << off;
    else if (off < 0 && off > -bits) word |= code >> (-off);
  }
  return word;
}

// Pack one code per thread (thread c = channel c of threads 0..D-1) into a key row (see
// packed_word).  `s_code` is D bytes of LDS.
template <int D>
MKV_DEV void pack_row(int code, int bits, uint8_t *s_code, uint8_t *row) {
  const int c = threadIdx.x;
  s_code[c] = (uint8_t)code;
  __syncthreads();
  const int words = D * bits / 32;
  if (c < words) gst(reinterpret_cast<uint32_t *>(row) + c, packed_word(s_code, D, bits, c));
  __syncthreads();
}

// Value codes are stored in blocks of 4 tokens: code (channel c, token j) at bit bits*(4c + j)
// of the block, so the 4 tokens of a channel form two 2*bits-bit fields.  OR one code per thread
// into the LDS copy `s_blk` of a block.
MKV_DEV void or_quad_code(uint32_t *s_blk, int c, int j, int code, int bits) {
  const int bit = bits * (4 * c + j);
  atomicOr(&s_blk[bit >> 5], (uint32_t)code << (bit & 31));
  const int spill = (bit & 31) + bits - 32;
  if (spill > 0) atomicOr(&s_blk[(bit >> 5) + 1], (uint32_t)code >> (bits - spill));
}

// Inclusive rank among flagged threads 0..D-1 (D <= 128, the threads that reach the barriers).
template <int D>
MKV_DEV int flag_rank(bool f, int *s_tmp, int *total) {
  const uint64_t m = __ballot(f);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int before = __popcll(m & ((lane == 0) ? 0ull : (~0ull >> (64 - lane))));
  if (lane == 0) s_tmp[w] = __popcll(m);
  __syncthreads();
  int base = 0, tot = 0;
  for (int i = 0; i < D / 64; ++i) {
    if (i < w) base += s_tmp[i];
    tot += s_tmp[i];
  }
  __syncthreads();
  *total = tot;
  return base + before;
}

// KVQ value of one token: per-token scale = n_ov-th largest |v| (0-based), outliers (written),
// and this thread's code (returned; the caller places it in the token's 4-token block).
template <int D>
MKV_DEV int kvq_value_token(const SeqDesc &sd, int h, int t, uint32_t vbits, const float *cbtab,
                            float *s_abs, float *s_scale, int *s_tmp) {
  const int c = threadIdx.x;
  const float x = h2f(vbits);
  const float ax = fabsf(x);
  const int nov = sd.bp > 0 ? sd.n_ov : 0;
  float s;
  if (nov <= 1) {
    // the largest |v| or, for n_ov = 1, the largest after one occurrence of it is set aside:
    // wave maxima with their multiplicities, then (maximum unique) the largest value below it
    constexpr int NWV = D / 64;
    const int lane = c & 63, w = c >> 6;
    const float wm = wave_max(ax);
    const int wc = __popcll(__ballot(ax == wm));
    if (lane == 0) {
      s_abs[w] = wm;
      s_tmp[w] = wc;
    }
    __syncthreads();
    float m1 = s_abs[0];
#pragma unroll
    for (int i = 1; i < NWV; ++i) m1 = fmaxf(m1, s_abs[i]);
    int cnt = 0;
#pragma unroll
    for (int i = 0; i < NWV; ++i) cnt += s_abs[i] == m1 ? s_tmp[i] : 0;
    s = m1;
    if (nov == 1 && cnt < 2) {  // block-uniform
      __syncthreads();
      const float wm2 = wave_max(ax < m1 ? ax : -1.f);
      if (lane == 0) s_abs[w] = wm2;
      __syncthreads();
      s = s_abs[0];
#pragma unroll
      for (int i = 1; i < NWV; ++i) s = fmaxf(s, s_abs[i]);
    }
    __syncthreads();  // s_abs and s_tmp are free again
  } else {
    s_abs[c] = ax;
    __syncthreads();
    int gt = 0, ge = 0;
    for (int j = 0; j < D; ++j) {
      const float y = s_abs[j];
      gt += (y > ax) ? 1 : 0;
      ge += (y >= ax) ? 1 : 0;
    }
    if (gt <= nov && nov < ge) *s_scale = ax;
    __syncthreads();
    s = *s_scale;
    __syncthreads();
  }
  const float inv = s > 0.f ? __fdiv_rn(1.0f, s) : 0.f;
  const float xhat = __fmul_rn(x, inv);
  const int nc = 1 << sd.bits;
  const float *mid = cbtab + cb_offset(sd.bits) + 2 * nc + (nc - 1);
  const int code = code_from_mid(xhat, mid, nc - 1);
  const bool outl = sd.bp > 0 && ax > s;
  int total;
  const int r = flag_rank<D>(outl, s_tmp, &total);
  // slot-major: entry r of token t at r * cap + t
  uint32_t *vo = reinterpret_cast<uint32_t *>(sd.vout) + h * stride_vout(sd) + t;
  uint32_t *vd = reinterpret_cast<uint32_t *>(sd.vdel) + h * stride_vout(sd) + t;
  if (outl && r < sd.nov_slots) {
    vo[(size_t)r * sd.cap] = outlier_entry(vbits, t, code, c);
    // the attention's form: the outlier minus the value its code stands for, and the channel
    const float cbv = cbtab[cb_offset(sd.bits) + nc + code];
    vd[(size_t)r * sd.cap] = vdel_pack(__fsub_rn(x, __fmul_rn(s, cbv)), c);
  }
  if (c >= total && c < sd.nov_slots) {
    vo[(size_t)c * sd.cap] = kNoOutlier;
    vd[(size_t)c * sd.cap] = 0u;
  }
  if (c == 0) (reinterpret_cast<float *>(sd.vmeta) + h * stride_slots(sd))[t] = s;
  return code;
}

// Write the value codes of tokens t0..t0+3 (one 4-token block) from an LDS block image.
MKV_DEV void store_quad(const SeqDesc &sd, int h, int t0, const uint32_t *s_blk, int D) {
  const int words = D * sd.bits / 8;  // 4 tokens x D codes x bits / 32
  uint32_t *dst = reinterpret_cast<uint32_t *>(reinterpret_cast<uint8_t *>(sd.vc) + h * stride_codes(sd) +
                                               (size_t)(t0 / 4) * 4 * sd.rowbytes);
  for (int w = threadIdx.x; w < words; w += D) gst(dst + w, s_blk[w]);
}

// The frozen (threshold, 1 / threshold) pair of KVQ key channel c of kv head h.
MKV_DEV float2 kvq_key_tau(const SeqDesc &sd, int h, int c, int D) {
  return (reinterpret_cast<const float2 *>(sd.kmeta) + (size_t)h * D)[c];
}

// KVQ key of one token: code under the frozen per-channel threshold ti (kvq_key_tau), and the
// outlier flag.
MKV_DEV int kvq_key_code(const SeqDesc &sd, float2 ti, uint32_t kbits, const float *cbtab, bool *outl) {
  const float x = h2f(kbits);
  const float xhat = __fmul_rn(x, ti.y);
  const int nc = 1 << sd.bits;
  const float *mid = cbtab + cb_offset(sd.bits) + 2 * nc;
  *outl = sd.bp > 0 && fabsf(x) > ti.x;
  return code_from_mid(xhat, mid, nc - 1);
}

// UQ value of one token: 64-channel groups, one wave per group; returns this thread's code
// (the caller places it in the token's 4-token block) and writes the group's (min, step).
template <int D>
MKV_DEV int uq_value_token(const SeqDesc &sd, int h, int t, uint32_t vbits) {
  const int c = threadIdx.x;
  const float x = h2f(vbits);
  const float mn = wave_min(x), mx = wave_max(x);
  const float r = __fsub_rn(mx, mn);
  const float inv = r > 0.f ? __fdiv_rn(15.0f, r) : 0.f;
  const float y = __fmul_rn(__fsub_rn(x, mn), inv);
  const int code = (int)fminf(fmaxf(rintf(y), 0.f), 15.f);
  if ((c & 63) == 0)
    (reinterpret_cast<float2 *>(sd.vmeta) + h * stride_uq_vmeta(sd, D))[(size_t)t * (D / 64) + c / 64] =
        make_float2(mn, __fdiv_rn(r, 15.0f));
  return code;
}

// OR a UQ value code into an LDS image of its 4-token block (nibbles never straddle words).
MKV_DEV void or_uq_code(uint32_t *s_blk, int ch, int j, int code, int D) {
  const int bit = uq_vbit(ch, j, D);
  atomicOr(&s_blk[bit >> 5], (uint32_t)code << (bit & 31));
}

// Write a 4-token block (D/2 words) from an LDS image by D threads; t0 is the block's first slot.
template <int D>
MKV_DEV void store_block(uint8_t *codes, int h_stride_bytes, int h, int t0, int rowbytes, const uint32_t *s_blk,
                         int words) {
  uint32_t *dst = reinterpret_cast<uint32_t *>(codes + (size_t)h * h_stride_bytes + (size_t)(t0 / 4) * 4 * rowbytes);
  for (int w = threadIdx.x; w < words; w += D) gst(dst + w, s_blk[w]);
}

// UQ key block: thread c quantizes channel c over 64 tokens read through `get(t)`.
template <int D, typename Get>
MKV_DEV void uq_key_block(const SeqDesc &sd, int h, int blk, Get get) {
  const int c = threadIdx.x;
  float mn = INFINITY, mx = -INFINITY;
  for (int t = 0; t < 64; ++t) {
    const float x = h2f(get(t));
    mn = fminf(mn, x);
    mx = fmaxf(mx, x);
  }
  const float r = __fsub_rn(mx, mn);
  const float inv = r > 0.f ? __fdiv_rn(15.0f, r) : 0.f;
  uint8_t *base = reinterpret_cast<uint8_t *>(sd.kc) + h * stride_codes(sd) + (size_t)blk * 64 * (D / 2);
  for (int t = 0; t < 64; ++t) {
    const float x = h2f(get(t));
    const float y = __fmul_rn(__fsub_rn(x, mn), inv);
    const int code = (int)fminf(fmaxf(rintf(y), 0.f), 15.f);
    const int partner = __shfl_down(code, 1);
    if ((c & 1) == 0) base[(size_t)t * (D / 2) + c / 2] = (uint8_t)(code | (partner << 4));
  }
  (reinterpret_cast<float2 *>(sd.kmeta) + h * stride_uq_kmeta(sd, D))[(size_t)blk * D + c] =
      make_float2(mn, __fdiv_rn(r, 15.0f));
}

// ---- decode append: D threads per (sequence, kv head) ------------------------------------------
template <int D>
struct AppendLds {
  float abs[D];
  float scale;
  uint8_t code[D];
  int tmp[4];
  uint32_t blk[D / 2];
  float cbt[kCbTableFloats];  // codebooks and midpoints, read many times below
  unsigned long long vkey[D / 64];
  int vslot;
};

// H2O: the slot the last attention pass chose for eviction (-1: none), the lowest (score,
// position) key among its per-part candidates; threads 0..D-1, every one gets the result.
template <int D>
MKV_DEV int h2o_victim(const SeqDesc &sd, int h, AppendLds<D> &L) {
  const int c = threadIdx.x, lane = c & 63, w = c >> 6;
  const uint32_t *vb = reinterpret_cast<const uint32_t *>(sd.vbest) + (size_t)h * sd.vparts * 4;
  unsigned long long best = ~0ull;
  int bslot = -1;
  for (int p = c; p < sd.vparts; p += D) {
    const uint4 e = gld16(vb + 4 * p);
    const unsigned long long key = (unsigned long long)e.x | ((unsigned long long)e.y << 32);
    if (key < best) {
      best = key;
      bslot = (int)e.z;
    }
  }
  const unsigned long long wm = wave_min_u64(best);
  if (lane == 0) L.vkey[w] = wm;
  __syncthreads();
  unsigned long long all = L.vkey[0];
#pragma unroll
  for (int i = 1; i < D / 64; ++i) all = L.vkey[i] < all ? L.vkey[i] : all;
  // keys carry the position, so at most one thread holds the lowest
  if (all != ~0ull && best == all) L.vslot = bslot;
  if (c == 0 && all == ~0ull) L.vslot = -1;
  __syncthreads();
  return L.vslot;
}

// Append the new token of (seq, h) by threads 0..D-1 of the workgroup (every barrier below is
// reached by exactly those threads).
template <int D>
MKV_DEV void append_pair(const SeqDesc &sd, int32_t *st, int seq, int h, int Hkv, const uint16_t *__restrict__ k,
                         const uint16_t *__restrict__ v, const float *__restrict__ cbtab, AppendLds<D> &L) {
  float *s_abs = L.abs, *s_cbt = L.cbt;
  uint8_t *s_code = L.code;
  int *s_tmp = L.tmp;
  uint32_t *s_blk = L.blk;
  const int c = threadIdx.x;
  // reads that need only the work item or the descriptor are issued first
  const uint32_t kb = k[((size_t)seq * Hkv + h) * D + c];
  const uint32_t vb = v[((size_t)seq * Hkv + h) * D + c];
  const float2 ti = sd.method == KVQ ? kvq_key_tau(sd, h, c, D) : make_float2(0.f, 0.f);
  const int count = st[ST_COUNT], pos = st[ST_NEXT_POS], kfill = st[ST_KOUT_FILL];
  for (int i = c; i < kCbTableFloats; i += D) s_cbt[i] = cbtab[i];
  // H2O: an eviction decided by the last attention pass frees its slot for this token (-1: none)
  const int victim = sd.method == H2O ? h2o_victim<D>(sd, h, L) : -1;
  const int slot = sd.method == H2O ? (victim >= 0 ? victim : st[ST_FREE_SLOT]) : count;
  // a full region (reachable only by replaying a captured decode step past max_new_tokens) drops
  // the token instead of writing past the region; the decision is the same for every thread
  if (slot >= sd.cap || (sd.method == KVQ && sd.bp > 0 && kfill + D > sd.pool_cap)) return;
  __syncthreads();  // every thread has read the state before thread 0 updates it
  switch (sd.method) {
    case FP16: {
      (reinterpret_cast<uint16_t *>(sd.k) + h * stride_rows(sd, D))[(size_t)count * D + c] = (uint16_t)kb;
      (reinterpret_cast<uint16_t *>(sd.v) + h * stride_rows(sd, D))[(size_t)count * D + c] = (uint16_t)vb;
      if (c == 0) st[ST_COUNT] = count + 1;
      break;
    }
    case H2O: {
      // into the victim's slot, else at the end
      const int new_count = victim >= 0 ? count : count + 1;
      (reinterpret_cast<uint16_t *>(sd.k) + h * stride_rows(sd, D))[(size_t)slot * D + c] = (uint16_t)kb;
      (reinterpret_cast<uint16_t *>(sd.v) + h * stride_rows(sd, D))[(size_t)slot * D + c] = (uint16_t)vb;
      __syncthreads();
      if (c == 0) {
        (reinterpret_cast<int32_t *>(sd.pos) + h * stride_slots(sd))[slot] = pos;
        (reinterpret_cast<float *>(sd.score) + h * stride_slots(sd))[slot] = 0.f;
        st[ST_COUNT] = new_count;
        st[ST_FREE_SLOT] = new_count;
      }
      break;
    }
    case ROCKET: {
      (reinterpret_cast<uint16_t *>(sd.k) + h * stride_rows(sd, D))[(size_t)count * D + c] = (uint16_t)kb;
      (reinterpret_cast<uint16_t *>(sd.v) + h * stride_rows(sd, D))[(size_t)count * D + c] = (uint16_t)vb;
      (reinterpret_cast<uint16_t *>(sd.kcm) + h * stride_kcm(sd, D))[(size_t)c * sd.cstride + count] = (uint16_t)kb;
      if (c == 0) {
        (reinterpret_cast<int32_t *>(sd.pos) + h * stride_slots(sd))[count] = pos;
        st[ST_COUNT] = count + 1;
      }
      break;
    }
    case UQ: {
      const int vcode = uq_value_token<D>(sd, h, count, vb);
      // the value code goes into its 4-token block: zero for the block's first token, otherwise
      // the stored block
      const int j = count & 3, words = D / 2;
      const uint32_t *blk = reinterpret_cast<const uint32_t *>(reinterpret_cast<const uint8_t *>(sd.vc) +
                                                               h * stride_codes(sd) + (size_t)(count / 4) * 4 * sd.rowbytes);
      for (int w = c; w < words; w += D) s_blk[w] = j == 0 ? 0u : gld(blk + w);
      __syncthreads();
      or_uq_code(s_blk, c, j, vcode, D);
      __syncthreads();
      store_block<D>(reinterpret_cast<uint8_t *>(sd.vc), (int)stride_codes(sd), h, count & ~3, sd.rowbytes, s_blk, words);
      uint16_t *res = reinterpret_cast<uint16_t *>(sd.kres) + (size_t)h * 64 * D;
      res[(size_t)(count & 63) * D + c] = (uint16_t)kb;
      if ((count & 63) == 63) {
        // the block is complete: thread c quantizes channel c of the 64 residual rows it wrote
        __syncthreads();
        uq_key_block<D>(sd, h, count >> 6, [&](int t) { return (uint32_t)res[(size_t)t * D + c]; });
      }
      if (c == 0) st[ST_COUNT] = count + 1;
      break;
    }
    case KVQ: {
      bool outl;
      const int code = kvq_key_code(sd, ti, kb, s_cbt, &outl);
      uint8_t *row = reinterpret_cast<uint8_t *>(sd.kc) + h * stride_codes(sd) + (size_t)count * sd.rowbytes;
      pack_row<D>(code, sd.bits, s_code, row);
      int total;
      const int r = flag_rank<D>(outl, s_tmp, &total);
      const int fill = kfill;
      uint32_t *ko = reinterpret_cast<uint32_t *>(sd.kout) + h * stride_kout(sd);
      if (outl) ko[fill + r] = outlier_entry(kb, count, code, c);
      const int vcode = kvq_value_token<D>(sd, h, count, vb, s_cbt, s_abs, &L.scale, s_tmp);
      // the value code goes into its 4-token block: the block's first token writes the whole
      // block (other tokens' codes zero); later tokens OR their bits into the stored words
      const int j = count & 3, words = D * sd.bits / 8;
      if (j == 0) {
        for (int w = c; w < words; w += D) s_blk[w] = 0u;
        __syncthreads();
        or_quad_code(s_blk, c, j, vcode, sd.bits);
        __syncthreads();
        store_quad(sd, h, count & ~3, s_blk, D);
      } else {
        uint32_t *blk = reinterpret_cast<uint32_t *>(reinterpret_cast<uint8_t *>(sd.vc) + h * stride_codes(sd) +
                                                     (size_t)(count / 4) * 4 * sd.rowbytes);
        const int bit = sd.bits * (4 * c + j);
        atomicOr(blk + (bit >> 5), (uint32_t)vcode << (bit & 31));
        const int spill = (bit & 31) + sd.bits - 32;
        if (spill > 0) atomicOr(blk + (bit >> 5) + 1, (uint32_t)vcode >> (sd.bits - spill));
      }
      __syncthreads();
      if (c == 0) {
        (reinterpret_cast<uint32_t *>(sd.krow) + h * stride_krow(sd))[count + 1] = (uint32_t)(fill + total);
        st[ST_KOUT_FILL] = fill + total;
        st[ST_COUNT] = count + 1;
      }
      break;
    }
    default:
      break;
  }
  if (c == 0) st[ST_NEXT_POS] = pos + 1;
}

// One workgroup of D threads per (sequence, kv head).
template <int D>
__global__ __launch_bounds__(128) void k_append_decode(const SeqDesc *__restrict__ seqs, int32_t *state,
                                                      const uint16_t *__restrict__ k,
                                                      const uint16_t *__restrict__ v,
                                                      const float *__restrict__ cbtab, int Hkv) {
  __shared__ AppendLds<D> L;
  const int seq = blockIdx.x / Hkv, h = blockIdx.x % Hkv;
  append_pair<D>(seqs[seq], state + ((size_t)seq * Hkv + h) * ST_WORDS, seq, h, Hkv, k, v, cbtab, L);
}

// The decode step's first two launches when RocketKV sequences are present.
//
// k_append_score, workgroups of kScoreThreads threads over a work list (int4: seq, kv head,
// part, parts): part -1 appends the token of a non-RocketKV pair on its first D threads (the
// other waves leave at once; a barrier waits only for waves that have not ended).  A RocketKV pair
// has ceil(cap / kScoreTokens) parts: part 0 appends its token (rows, channel-major copy,
// position) and every part picks the channels and scores its kScoreTokens tokens, the new one
// from the key it holds in LDS.  The state of a RocketKV pair is left to the selecting launch.
//
// k_rocket_select, one workgroup of kTopkThreads threads per RocketKV pair (int2: seq, kv head):
// the top-k of the scores, then the pair's state (count, next position, selection count).
template <int D, int G>
__global__ __launch_bounds__(kScoreThreads) void k_append_score(const SeqDesc *__restrict__ seqs, int32_t *state,
                                                                const int4 *__restrict__ items,
                                                                const uint16_t *__restrict__ k,
                                                                const uint16_t *__restrict__ v,
                                                                const uint16_t *__restrict__ q,
                                                                const float *__restrict__ cbtab, int Hkv) {
  __shared__ union {
    AppendLds<D> a;
    ChanLds<D, kScoreThreads> c;
  } L;
  const int4 it = items[blockIdx.x];
  const int seq = it.x, h = it.y, part = it.z, c = threadIdx.x;
  const SeqDesc &sd = seqs[seq];
  int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  if (part < 0) {
    if (c >= D) return;
    append_pair<D>(sd, st, seq, h, Hkv, k, v, cbtab, L.a);
    return;
  }
  // the query channels first: their address needs only the work item
  uint16_t qr[G];
  load_qcol<D, G>(q + ((size_t)seq * Hkv * G + h * G) * D, qr);
  const int count = st[ST_COUNT];
  // a full region (reachable only by replaying a captured decode step past max_new_tokens) drops
  // the token, as the separate append does
  const bool room = count < sd.cap;
  if (room && c < D) {
    const uint16_t kb = k[((size_t)seq * Hkv + h) * D + c];
    L.c.knew[c] = kb;
    if (part == 0) {
      const uint16_t vb = v[((size_t)seq * Hkv + h) * D + c];
      (reinterpret_cast<uint16_t *>(sd.k) + h * stride_rows(sd, D))[(size_t)count * D + c] = kb;
      (reinterpret_cast<uint16_t *>(sd.v) + h * stride_rows(sd, D))[(size_t)count * D + c] = vb;
      (reinterpret_cast<uint16_t *>(sd.kcm) + h * stride_kcm(sd, D))[(size_t)c * sd.cstride + count] = kb;
      if (c == 0) (reinterpret_cast<int32_t *>(sd.pos) + h * stride_slots(sd))[count] = st[ST_NEXT_POS];
    }
  }
  score_part<D, G>(sd, h, room ? count + 1 : count, part, room, qr, L.c);
}

template <int D>
__global__ __launch_bounds__(kTopkThreads) void k_rocket_select(const SeqDesc *__restrict__ seqs, int32_t *state,
                                                                const int2 *__restrict__ pairs, int Hkv) {
  __shared__ SelLds L;
  const int2 pr = pairs[blockIdx.x];
  const int seq = pr.x, h = pr.y, tid = threadIdx.x;
  const SeqDesc &sd = seqs[seq];
  int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  const int count = st[ST_COUNT], pos = st[ST_NEXT_POS];
  const bool room = count < sd.cap;
  const int n = room ? count + 1 : count, k = sd.topk;
  int32_t *sel = reinterpret_cast<int32_t *>(sd.sel) + h * stride_sel(sd);
  if (k >= n) {
    for (int j = tid; j < n; j += kTopkThreads) sel[j] = j;
  } else {
    const uint32_t *akeys = reinterpret_cast<const uint32_t *>(sd.akeys) + h * stride_slots(sd);
    select_keys<kTopkThreads>(n, k, [&](int j) { return gld(akeys + j); }, sel, L);
  }
  __syncthreads();  // every thread has read the state
  if (tid == 0) {
    st[ST_SEL_COUNT] = min(k, n);
    if (room) {
      st[ST_COUNT] = count + 1;
      st[ST_NEXT_POS] = pos + 1;
    }
  }
}

// ---- prefill -----------------------------------------------------------------------------------

// Copy prompt rows [n0][Hkv][D] (input layout) into per-head rows [Hkv][n0 or cap][D].
template <int D>
__global__ void k_prefill_copy(const uint16_t *__restrict__ k, const uint16_t *__restrict__ v,
                               uint16_t *dk, uint16_t *dv, int64_t head_stride, int n0, int Hkv) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;   // one 16-byte chunk
  const int64_t total = (int64_t)n0 * Hkv * (D / 8);
  if (i >= total) return;
  const int ch = (int)(i % (D / 8));
  const int h = (int)((i / (D / 8)) % Hkv);
  const int64_t t = i / ((D / 8) * Hkv);
  const uint4 a = reinterpret_cast<const uint4 *>(k)[i];
  const uint4 b = reinterpret_cast<const uint4 *>(v)[i];
  *reinterpret_cast<uint4 *>(dk + h * head_stride + t * D + ch * 8) = a;
  *reinterpret_cast<uint4 *>(dv + h * head_stride + t * D + ch * 8) = b;
}

// UQ prompt values: one workgroup per (4-token block, kv head).
template <int D>
__global__ __launch_bounds__(128) void k_prefill_uq_values(const SeqDesc *__restrict__ seqs, int seq,
                                                          const uint16_t *__restrict__ v, int Hkv, int n0) {
  __shared__ uint32_t s_blk[D / 2];
  const SeqDesc &sd = seqs[seq];
  const int q = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
  for (int w = c; w < D / 2; w += D) s_blk[w] = 0;
  __syncthreads();
  for (int j = 0; j < 4 && 4 * q + j < n0; ++j) {
    const int t = 4 * q + j;
    const int code = uq_value_token<D>(sd, h, t, v[((size_t)t * Hkv + h) * D + c]);
    or_uq_code(s_blk, c, j, code, D);
  }
  __syncthreads();
  store_block<D>(reinterpret_cast<uint8_t *>(sd.vc), (int)stride_codes(sd), h, 4 * q, sd.rowbytes, s_blk, D / 2);
}

template <int D>
__global__ __launch_bounds__(128) void k_prefill_uq_keys(const SeqDesc *__restrict__ seqs, int seq,
                                                        const uint16_t *__restrict__ k, int Hkv, int n0) {
  const SeqDesc &sd = seqs[seq];
  const int blk = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
  const int nfull = n0 / 64;
  if (blk < nfull) {
    uq_key_block<D>(sd, h, blk, [&](int t) { return (uint32_t)k[((size_t)(blk * 64 + t) * Hkv + h) * D + c]; });
  } else {
    uint16_t *res = reinterpret_cast<uint16_t *>(sd.kres) + (size_t)h * 64 * D;
    for (int t = nfull * 64; t < n0; ++t) res[(size_t)(t & 63) * D + c] = k[((size_t)t * Hkv + h) * D + c];
  }
}

// KVQ key thresholds: the n_o-th largest |k| (0-based) of every channel over the prompt, by a
// two-pass radix select on the 15-bit fp16 magnitude.  A workgroup takes 64 channels of one kv
// head: lane l of every wave owns channel c0 + l (one coalesced 128-byte load per token), the 8
// waves take every eighth token, kCalibBatch tokens' loads in flight at a time, and count into
// one 256-bin histogram per channel by LDS atomics (rows padded so that the lanes' bins spread
// over the banks); thread c < 64 then finds its channel's digit.
constexpr int kCalibThreads = 512;
constexpr int kCalibBatch = 16;
template <int D>
__global__ __launch_bounds__(kCalibThreads) void k_kvq_calibrate(const SeqDesc *__restrict__ seqs, int seq,
                                                                 const uint16_t *__restrict__ k, int Hkv, int n0) {
  __shared__ uint32_t hist[64][257];
  __shared__ uint32_t s_sel[64], s_rem[64];
  const SeqDesc &sd = seqs[seq];
  const int h = blockIdx.x, c0 = 64 * blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int NW = kCalibThreads / 64;
  const int want = sd.bp > 0 ? sd.n_o : 0;  // 0-based rank from the top
  if (want >= n0) {  // fewer prompt tokens than the rank: no threshold (every key is an inlier)
    if (threadIdx.x < 64)
      (reinterpret_cast<float2 *>(sd.kmeta) + (size_t)h * D)[c0 + threadIdx.x] = make_float2(0.f, 0.f);
    return;
  }
  if (threadIdx.x < 64) s_rem[threadIdx.x] = (uint32_t)want + 1;  // 1-based rank
  const uint16_t *kc = k + (size_t)h * D + c0 + lane;
  const size_t tstride = (size_t)Hkv * D;
  for (int pass = 0; pass < 2; ++pass) {
    for (int e = threadIdx.x; e < 64 * 257; e += kCalibThreads) (&hist[0][0])[e] = 0u;
    __syncthreads();
    const uint32_t sel = pass == 0 ? 0u : s_sel[lane];
    for (int t0 = wave; t0 < n0; t0 += NW * kCalibBatch) {
      uint32_t key[kCalibBatch];
#pragma unroll
      for (int b = 0; b < kCalibBatch; ++b)
        key[b] = (uint32_t)gld(kc + (size_t)min(t0 + b * NW, n0 - 1) * tstride) & 0x7FFFu;
#pragma unroll
      for (int b = 0; b < kCalibBatch; ++b) {
        if (t0 + b * NW >= n0) break;
        if (pass == 0) atomicAdd(&hist[lane][key[b] >> 8], 1u);
        else if ((key[b] >> 8) == sel) atomicAdd(&hist[lane][key[b] & 255u], 1u);
      }
    }
    __syncthreads();
    if (threadIdx.x < 64) {
      const int c = threadIdx.x;
      const uint32_t remaining = s_rem[c];
      uint32_t cum = 0;
      int dg = 0;
      for (int bb = 255; bb >= 0; --bb) {
        if (cum + hist[c][bb] >= remaining) {
          dg = bb;
          break;
        }
        cum += hist[c][bb];
      }
      s_rem[c] = remaining - cum;
      if (pass == 0) {
        s_sel[c] = (uint32_t)dg;
      } else {
        const float tau = h2f((s_sel[c] << 8) | (uint32_t)dg);
        const float inv = tau > 0.f ? __fdiv_rn(1.0f, tau) : 0.f;
        (reinterpret_cast<float2 *>(sd.kmeta) + (size_t)h * D)[c0 + c] = make_float2(tau, inv);
      }
    }
    __syncthreads();
  }
}

// KVQ prompt keys, pass 1 (write codes, count outliers per token into krow[t+1]) or pass 2
// (write the outlier entries at their CSR offsets).
template <int D>
__global__ __launch_bounds__(128) void k_kvq_keys(const SeqDesc *__restrict__ seqs, int seq,
                                                 const uint16_t *__restrict__ k, const float *__restrict__ cbtab,
                                                 int Hkv, int pass) {
  __shared__ uint8_t s_code[D];
  __shared__ int s_tmp[4];
  const SeqDesc &sd = seqs[seq];
  const int t = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
  const uint32_t kb = k[((size_t)t * Hkv + h) * D + c];
  bool outl;
  const int code = kvq_key_code(sd, kvq_key_tau(sd, h, c, D), kb, cbtab, &outl);
  uint32_t *krow = reinterpret_cast<uint32_t *>(sd.krow) + h * stride_krow(sd);
  if (pass == 0) {
    uint8_t *row = reinterpret_cast<uint8_t *>(sd.kc) + h * stride_codes(sd) + (size_t)t * sd.rowbytes;
    pack_row<D>(code, sd.bits, s_code, row);
    int total;
    flag_rank<D>(outl, s_tmp, &total);
    if (c == 0) krow[t + 1] = (uint32_t)total;
  } else {
    int total;
    const int r = flag_rank<D>(outl, s_tmp, &total);
    if (outl) (reinterpret_cast<uint32_t *>(sd.kout) + h * stride_kout(sd))[krow[t] + r] = outlier_entry(kb, t, code, c);
  }
}

// In-place inclusive scan of krow[1..n0] (per-token outlier counts) per kv head.
__global__ __launch_bounds__(256) void k_kvq_scan(const SeqDesc *__restrict__ seqs, int seq, int32_t *state,
                                                  int Hkv, int n0) {
  __shared__ int s_tmp[4];
  const SeqDesc &sd = seqs[seq];
  const int h = blockIdx.x;
  uint32_t *krow = reinterpret_cast<uint32_t *>(sd.krow) + h * stride_krow(sd);
  int run = 0;
  for (int a = 0; a < n0; a += 256) {
    const int i = a + (int)threadIdx.x;
    const int x = (i < n0) ? (int)krow[i + 1] : 0;
    int total;
    const int ex = block_exclusive_scan<256>(x, s_tmp, &total);
    if (i < n0) krow[i + 1] = (uint32_t)(run + ex + x);
    run += total;
  }
  if (threadIdx.x == 0) {
    krow[0] = 0;
    state[((size_t)seq * Hkv + h) * ST_WORDS + ST_KOUT_FILL] = run;
  }
}

// KVQ prompt values: one workgroup per (4-token block, kv head) quantizes the block's tokens and
// writes the block.
template <int D>
__global__ __launch_bounds__(128) void k_prefill_kvq_values(const SeqDesc *__restrict__ seqs, int seq,
                                                           const uint16_t *__restrict__ v,
                                                           const float *__restrict__ cbtab, int Hkv, int n0) {
  __shared__ float s_abs[D];
  __shared__ float s_scale;
  __shared__ int s_tmp[4];
  __shared__ uint32_t s_blk[D / 2];
  const SeqDesc &sd = seqs[seq];
  const int q = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
  const int words = D * sd.bits / 8;
  for (int w = c; w < words; w += D) s_blk[w] = 0;
  __syncthreads();
  for (int j = 0; j < 4 && 4 * q + j < n0; ++j) {
    const int t = 4 * q + j;
    const int code = kvq_value_token<D>(sd, h, t, v[((size_t)t * Hkv + h) * D + c], cbtab, s_abs, &s_scale, s_tmp);
    or_quad_code(s_blk, c, j, code, sd.bits);
  }
  __syncthreads();
  store_quad(sd, h, 4 * q, s_blk, D);
}

__global__ void k_prefill_state(const SeqDesc *__restrict__ seqs, int seq, int32_t *state, int Hkv) {
  const SeqDesc &sd = seqs[seq];
  const int h = threadIdx.x;
  if (h >= Hkv) return;
  int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  const bool staged = sd.method == H2O || sd.method == ROCKET;
  st[ST_COUNT] = staged ? 0 : sd.n0;
  st[ST_NEXT_POS] = sd.n0;
  st[ST_FREE_SLOT] = 0;
  st[ST_KEPT] = sd.n0;
}

__global__ void k_init_state(int32_t *state, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) state[i] = 0;
}

template <int D>
hipError_t append_decode_impl(const Dev &dv, const Shape &sh, const uint16_t *k, const uint16_t *v,
                              hipStream_t st, LaunchEv ev) {
  hipExtLaunchKernelGGL(k_append_decode<D>, dim3(sh.S * sh.Hkv), dim3(D), 0, st, ev.start, ev.stop, 0, dv.seqs,
                        dv.state, k, v, dv.cbtab, sh.Hkv);
  return hipGetLastError();
}

template <int D, int G>
hipError_t append_select_impl(const Dev &dv, const Shape &sh, const uint16_t *k, const uint16_t *v,
                              const uint16_t *q, hipStream_t st, LaunchEv ev_score, LaunchEv ev_select) {
  hipExtLaunchKernelGGL((k_append_score<D, G>), dim3(dv.n_prep), dim3(kScoreThreads), 0, st, ev_score.start,
                        ev_score.stop, 0, dv.seqs, dv.state, dv.prep, k, v, q, dv.cbtab, sh.Hkv);
  hipExtLaunchKernelGGL(k_rocket_select<D>, dim3(dv.n_rk_pairs), dim3(kTopkThreads), 0, st, ev_select.start,
                        ev_select.stop, 0, dv.seqs, dv.state, dv.rk_pairs, sh.Hkv);
  return hipGetLastError();
}

template <int D>
hipError_t prefill_impl(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq, const uint16_t *k,
                        const uint16_t *v, hipStream_t st) {
  const int n0 = hs.n0, Hkv = sh.Hkv;
  hipLaunchKernelGGL(k_prefill_state, dim3(1), dim3(64 * ((Hkv + 63) / 64)), 0, st, dv.seqs, seq, dv.state, Hkv);
  switch (hs.method) {
    case FP16:
    case H2O:
    case ROCKET: {
      const bool staged = hs.method != FP16;
      uint16_t *dk = reinterpret_cast<uint16_t *>(staged ? hs.stage_k : hs.k);
      uint16_t *dvp = reinterpret_cast<uint16_t *>(staged ? hs.stage_v : hs.v);
      const int64_t hstride = staged ? stride_stage(hs, D) : stride_rows(hs, D);
      const int64_t chunks = (int64_t)n0 * Hkv * (D / 8);
      hipLaunchKernelGGL(k_prefill_copy<D>, dim3((unsigned)((chunks + 255) / 256)), dim3(256), 0, st, k, v,
                         dk, dvp, hstride, n0, Hkv);
      break;
    }
    case UQ:
      hipLaunchKernelGGL(k_prefill_uq_values<D>, dim3((n0 + 3) / 4, Hkv), dim3(D), 0, st, dv.seqs, seq, v, Hkv, n0);
      hipLaunchKernelGGL(k_prefill_uq_keys<D>, dim3(n0 / 64 + 1, Hkv), dim3(D), 0, st, dv.seqs, seq, k, Hkv, n0);
      break;
    case KVQ:
      hipLaunchKernelGGL(k_kvq_calibrate<D>, dim3(Hkv, D / 64), dim3(kCalibThreads), 0, st, dv.seqs, seq, k, Hkv, n0);
      hipLaunchKernelGGL(k_kvq_keys<D>, dim3(n0, Hkv), dim3(D), 0, st, dv.seqs, seq, k, dv.cbtab, Hkv, 0);
      hipLaunchKernelGGL(k_kvq_scan, dim3(Hkv), dim3(256), 0, st, dv.seqs, seq, dv.state, Hkv, n0);
      hipLaunchKernelGGL(k_kvq_keys<D>, dim3(n0, Hkv), dim3(D), 0, st, dv.seqs, seq, k, dv.cbtab, Hkv, 1);
      hipLaunchKernelGGL(k_prefill_kvq_values<D>, dim3((n0 + 3) / 4, Hkv), dim3(D), 0, st, dv.seqs, seq, v, dv.cbtab,
                         Hkv, n0);
      break;
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_append_decode(const Dev &dv, const Shape &sh, const uint16_t *k, const uint16_t *v,
                                hipStream_t st, LaunchEv ev) {
  return sh.D == 64 ? append_decode_impl<64>(dv, sh, k, v, st, ev) : append_decode_impl<128>(dv, sh, k, v, st, ev);
}

hipError_t launch_append_select(const Dev &dv, const Shape &sh, const uint16_t *k, const uint16_t *v,
                                const uint16_t *q, hipStream_t st, LaunchEv ev_score, LaunchEv ev_select) {
  switch (sh.D * 16 + sh.G) {
    case 64 * 16 + 1: return append_select_impl<64, 1>(dv, sh, k, v, q, st, ev_score, ev_select);
    case 64 * 16 + 2: return append_select_impl<64, 2>(dv, sh, k, v, q, st, ev_score, ev_select);
    case 64 * 16 + 4: return append_select_impl<64, 4>(dv, sh, k, v, q, st, ev_score, ev_select);
    case 64 * 16 + 8: return append_select_impl<64, 8>(dv, sh, k, v, q, st, ev_score, ev_select);
    case 128 * 16 + 1: return append_select_impl<128, 1>(dv, sh, k, v, q, st, ev_score, ev_select);
    case 128 * 16 + 2: return append_select_impl<128, 2>(dv, sh, k, v, q, st, ev_score, ev_select);
    case 128 * 16 + 4: return append_select_impl<128, 4>(dv, sh, k, v, q, st, ev_score, ev_select);
    case 128 * 16 + 8: return append_select_impl<128, 8>(dv, sh, k, v, q, st, ev_score, ev_select);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_prefill_seq(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq, const uint16_t *k,
                              const uint16_t *v, hipStream_t st) {
  return sh.D == 64 ? prefill_impl<64>(dv, sh, hs, seq, k, v, st) : prefill_impl<128>(dv, sh, hs, seq, k, v, st);
}

hipError_t launch_init_state(const Dev &dv, const Shape &sh, hipStream_t st) {
  const int n = sh.S * sh.Hkv * ST_WORDS;
  hipLaunchKernelGGL(k_init_state, dim3((n + 255) / 256), dim3(256), 0, st, dv.state, n);
  return hipGetLastError();
}

}  // namespace mkv
