// Split-K decode attention over a mixed-configuration KV cache, and the combine pass.
//
// Every configuration's decode step ends in softmax attention over the tokens its cache keeps
// (MetaKV Section 2.1): all tokens with dequantized values (uniform / KVQuant), the retained
// set (H2O) or the selected set (RocketKV).  One launch covers all sequences: each workgroup
// takes one tile = (sequence, kv head, token range) and runs the loop for that sequence's
// method.
//
// Tile work: 4 waves split the tile's tokens into contiguous ranges.  Within a wave, D/8 lanes
// share a token (8 channels each: one 16-byte fp16 load per row, or the matching packed-code
// bytes), so one wave load reads whole rows of 64/(D/8) consecutive tokens.  Each lane group
// issues the loads of U tokens before computing any of them (32 tokens per wave in flight), then
// reduces q . k over the group with DPP row ops, updates the wave-uniform running maximum once
// per batch, and accumulates p . v in registers.  Logits use the base-2 exponent (scaled by
// log2(e) / sqrt(d) after the reduction).
#include "kernels_common.h"

namespace mkv {

namespace {

typedef _Float16 h2v __attribute__((ext_vector_type(2)));

MKV_DEV float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(h2v, a), __builtin_bit_cast(h2v, b), c, false);
}

template <int D, int G>
struct Geo {
  static constexpr int LPT = D / 8;      // lanes per token
  static constexpr int TPW = 64 / LPT;   // tokens per wave load
  static constexpr int BT = G > 4 ? 16 : 32;  // tokens per wave batch (all loads issued first)
  static constexpr int U = BT / TPW;     // wave loads in flight per batch
};

template <int G>
struct Qs {
  uint32_t h[G][4];  // fp16 pairs of channels c0..c0+7, unscaled
  float f[G][8];     // the same in fp32
};

MKV_DEV U4 ld16(const void *p) { return gld16u(p); }

// ---- per-method loaders ------------------------------------------------------------------------
// fetch(t, raw): the loads of token t that depend only on t;  fetch2(raw): loads that depend on
// fetch's results;  dot(raw, q, part): this lane's partial q . k for every head (unscaled);
// pv(raw, p, o): o += p * v for this lane's 8 channels.

template <int D, int G>
struct LdRows {  // fp16 rows, token t = slot t (FP16, H2O)
  const uint16_t *K, *V;
  int c0;
  struct Raw { U4 k, v; };
  MKV_DEV void prep(int, const Qs<G> &) {}
  MKV_DEV void rescale(int, float) {}
  MKV_DEV void finish(float (&)[G][8]) const {}
  MKV_DEV int slot(const Raw &, int t) const { return t; }
  MKV_DEV void fetch(int t, Raw &r) const {
    r.k = ld16(K + (size_t)t * D + c0);
    r.v = ld16(V + (size_t)t * D + c0);
  }
  MKV_DEV void fetch2(Raw &) const {}
  MKV_DEV void dot(const Raw &r, const Qs<G> &q, float (&part)[G]) const {
#pragma unroll
    for (int g = 0; g < G; ++g)
      part[g] = dot2(q.h[g][3], r.k.w, dot2(q.h[g][2], r.k.z, dot2(q.h[g][1], r.k.y, dot2(q.h[g][0], r.k.x, 0.f))));
  }
  MKV_DEV void pv(const Raw &r, const float (&p)[G], float (&o)[G][8]) const {
    float vf[8];
    unpack8(r.v, vf);
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] = fmaf(p[g], vf[i], o[g][i]);
  }
};

template <int D, int G>
struct LdGather {  // RocketKV: token t of the tile is the t-th selected slot
  const uint16_t *K, *V;
  const int32_t *sel;
  int c0;
  struct Raw { U4 k, v; int s; };
  MKV_DEV void prep(int, const Qs<G> &) {}
  MKV_DEV void rescale(int, float) {}
  MKV_DEV void finish(float (&)[G][8]) const {}
  MKV_DEV int slot(const Raw &r, int) const { return r.s; }
  MKV_DEV void fetch(int t, Raw &r) const { r.s = gld(sel + t); }
  MKV_DEV void fetch2(Raw &r) const {
    r.k = ld16(K + (size_t)r.s * D + c0);
    r.v = ld16(V + (size_t)r.s * D + c0);
  }
  MKV_DEV void dot(const Raw &r, const Qs<G> &q, float (&part)[G]) const {
#pragma unroll
    for (int g = 0; g < G; ++g)
      part[g] = dot2(q.h[g][3], r.k.w, dot2(q.h[g][2], r.k.z, dot2(q.h[g][1], r.k.y, dot2(q.h[g][0], r.k.x, 0.f))));
  }
  MKV_DEV void pv(const Raw &r, const float (&p)[G], float (&o)[G][8]) const {
    float vf[8];
    unpack8(r.v, vf);
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] = fmaf(p[g], vf[i], o[g][i]);
  }
};

// Uniform 4-bit: k = mn_c + code * st_c per (64-token block, channel), so q . k = sum q mn +
// sum (q st) code with both per-block factors prepared once per block; v = mn_t + code * st_t
// per (token, 64 channels), so p v = p mn + (p st) code, with sum p mn kept per head (`om`).
template <int D, int G>
struct LdUQ {
  const uint8_t *kc, *vc;
  const float2 *kmeta, *vmeta;
  const uint16_t *kres;
  int c0, full, cur_blk;
  float qs[G][8], qm[G];
  float om[G];  // sum over tokens of p * mn, rescaled with o and added to it at the end
  struct Raw { uint32_t kw, vw, k0, k1, k2, k3; float vmn, vst; bool quant; };
  MKV_DEV void rescale(int g, float corr) { om[g] *= corr; }
  MKV_DEV void finish(float (&o)[G][8]) const {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] += om[g];
  }
  MKV_DEV void prep(int base, const Qs<G> &q) {
    const int blk = base >> 6;
    if (blk == cur_blk) return;
    cur_blk = blk;
    if (blk * 64 < full) {
#pragma unroll
      for (int g = 0; g < G; ++g) qm[g] = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float *mp = reinterpret_cast<const float *>(kmeta + (size_t)blk * D + c0 + i);
        const float mn = gld(mp), stp = gld(mp + 1);
#pragma unroll
        for (int g = 0; g < G; ++g) {
          qs[g][i] = q.f[g][i] * stp;
          qm[g] = fmaf(q.f[g][i], mn, qm[g]);
        }
      }
    }
  }
  MKV_DEV int slot(const Raw &, int t) const { return t; }
  MKV_DEV void fetch(int t, Raw &r) const {
    r.quant = t < full;
    r.kw = 0;
    r.k0 = r.k1 = r.k2 = r.k3 = 0;
    if (r.quant) {
      r.kw = gld(reinterpret_cast<const uint32_t *>(kc + (size_t)t * (D / 2) + c0 / 2));
    } else {
      const uint32_t *kr = reinterpret_cast<const uint32_t *>(kres + (size_t)(t & 63) * D + c0);
      r.k0 = gld(kr);
      r.k1 = gld(kr + 1);
      r.k2 = gld(kr + 2);
      r.k3 = gld(kr + 3);
    }
    r.vw = gld(reinterpret_cast<const uint32_t *>(vc + (size_t)t * (D / 2) + c0 / 2));
    const float *mp = reinterpret_cast<const float *>(vmeta + (size_t)t * (D / 64) + c0 / 64);
    r.vmn = gld(mp);
    r.vst = gld(mp + 1);
  }
  MKV_DEV void fetch2(Raw &) const {}
  MKV_DEV void dot(const Raw &r, const Qs<G> &q, float (&part)[G]) const {
    if (r.quant) {
      float cf[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) cf[i] = (float)((r.kw >> (4 * i)) & 15u);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float acc = qm[g];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc = fmaf(qs[g][i], cf[i], acc);
        part[g] = acc;
      }
    } else {
#pragma unroll
      for (int g = 0; g < G; ++g)
        part[g] = dot2(q.h[g][3], r.k3, dot2(q.h[g][2], r.k2, dot2(q.h[g][1], r.k1, dot2(q.h[g][0], r.k0, 0.f))));
    }
  }
  MKV_DEV void pv(const Raw &r, const float (&p)[G], float (&o)[G][8]) {
    float cf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) cf[i] = (float)((r.vw >> (4 * i)) & 15u);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      om[g] = fmaf(p[g], r.vmn, om[g]);
      const float ps = p[g] * r.vst;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] = fmaf(ps, cf[i], o[g][i]);
    }
  }
};

// KVQuant-style: codebooks in LDS; the per-channel key threshold is folded into q (q' = q tau),
// so a non-outlier key contributes q' cb[code]; outliers replace their channel's value.  The
// per-token value scale multiplies the dequantized row.
template <int D, int G, int BITS>
struct LdKVQ {
  static constexpr int bits = BITS;
  const uint8_t *kc, *vc;
  const uint32_t *krow, *kout, *vout;
  const float *vs;
  const float *cbk, *cbv;   // LDS
  const float *qlds;        // LDS [G][D]: unscaled q, for outlier corrections
  int c0, rowbytes, nov;
  float qp[G][8];
  struct Raw { uint32_t kw, vw; float sv; uint32_t ka, kb, e0, e1, vo; int t; };
  MKV_DEV void prep(int, const Qs<G> &) {}
  MKV_DEV void rescale(int, float) {}
  MKV_DEV void finish(float (&)[G][8]) const {}
  MKV_DEV int slot(const Raw &, int t) const { return t; }
  MKV_DEV uint32_t codes_word(const uint8_t *row) const {
    if (bits == 4) return gld(reinterpret_cast<const uint32_t *>(row + c0 / 2));
    if (bits == 2) return gld(reinterpret_cast<const uint16_t *>(row + c0 / 4));
    return (uint32_t)gld(reinterpret_cast<const uint16_t *>(row + c0 / 4)) | ((uint32_t)gld(row + D / 4 + c0 / 8) << 16);
  }
  MKV_DEV int code_at(uint32_t w, int i) const {
    if (bits == 4) return (w >> (4 * i)) & 15u;
    if (bits == 2) return (w >> (2 * i)) & 3u;
    return ((w >> (2 * i)) & 3u) | (((w >> (16 + i)) & 1u) << 2);
  }
  MKV_DEV void fetch(int t, Raw &r) const {
    r.kw = codes_word(kc + (size_t)t * rowbytes);
    r.vw = codes_word(vc + (size_t)t * rowbytes);
    r.sv = gld(vs + t);
    r.ka = gld(krow + t);
    r.kb = gld(krow + t + 1);
    r.vo = gld(vout + (size_t)t * nov);
    r.t = t;
  }
  MKV_DEV void fetch2(Raw &r) const {
    r.e0 = r.ka < r.kb ? gld(kout + r.ka) : kNoOutlier;
    r.e1 = r.ka + 1 < r.kb ? gld(kout + r.ka + 1) : kNoOutlier;
  }
  // correction of one key outlier entry: q . (x - tau cb[code]) on its channel
  MKV_DEV void k_fix(uint32_t ent, uint32_t kw, float (&part)[G]) const {
    const int ch = (int)(ent & 0xFFu);
    if (ch < c0 || ch >= c0 + 8) return;
    const float x = h2f(ent >> 16);
    const float cb = cbk[code_at(kw, ch - c0)];
#pragma unroll
    for (int g = 0; g < G; ++g) part[g] += qlds[g * D + ch] * x - qlds[G * D + g * D + ch] * cb;
  }
  MKV_DEV void dot(const Raw &r, const Qs<G> &, float (&part)[G]) const {
    float kf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) kf[i] = cbk[code_at(r.kw, i)];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc = fmaf(qp[g][i], kf[i], acc);
      part[g] = acc;
    }
    if (r.e0 != kNoOutlier) k_fix(r.e0, r.kw, part);
    if (r.e1 != kNoOutlier) k_fix(r.e1, r.kw, part);
    for (uint32_t e = r.ka + 2; e < r.kb; ++e) k_fix(gld(kout + e), r.kw, part);
  }
  MKV_DEV void pv(const Raw &r, const float (&p)[G], float (&o)[G][8]) const {
    float vf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) vf[i] = cbv[code_at(r.vw, i)] * r.sv;
    // value outliers replace their channel (the first slot comes with the row; more are rare)
    for (int j = 0; j < nov; ++j) {
      const uint32_t ent = j == 0 ? r.vo : gld(vout + (size_t)r.t * nov + j);
      if (ent == kNoOutlier) break;
      const int ch = (int)(ent & 0xFFu) - c0;
      const float x = h2f(ent >> 16);
#pragma unroll
      for (int i = 0; i < 8; ++i) vf[i] = (ch == i) ? x : vf[i];
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] = fmaf(p[g], vf[i], o[g][i]);
  }
};

// Run one wave over tokens [a, b) of its tile, 32 tokens per batch.
template <int D, int G, class L>
MKV_DEV void wave_attend(L &ld, int a, int b, const Qs<G> &q, float qscale, float (&m_run)[G], float (&l)[G],
                         float (&o)[G][8], int grp, int sub, float *logit_out) {
  constexpr int LPT = Geo<D, G>::LPT, TPW = Geo<D, G>::TPW, U = Geo<D, G>::U;
  for (int base = a; base < b; base += U * TPW) {
    ld.prep(base, q);
    // every lane loads; a lane past the end of the range re-reads the range's last token, whose
    // weight below is exactly 0 (no divergent branches around the loads)
    typename L::Raw raw[U];
#pragma unroll
    for (int u = 0; u < U; ++u) ld.fetch(min(base + u * TPW + grp, b - 1), raw[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) ld.fetch2(raw[u]);
    float s[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool valid = base + u * TPW + grp < b;
      float part[G];
      ld.dot(raw[u], q, part);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float x = group_sum<LPT>(part[g]) * qscale;
        s[u][g] = valid ? x : -INFINITY;
      }
    }
    if (logit_out != nullptr && sub == 0) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int t = base + u * TPW + grp;
        if (t < b) {
          const int sl = ld.slot(raw[u], t);
#pragma unroll
          for (int g = 0; g < G; ++g) gst(logit_out + (size_t)sl * G + g, s[u][g]);
        }
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = s[0][g];
#pragma unroll
      for (int u = 1; u < U; ++u) mx = fmaxf(mx, s[u][g]);
#pragma unroll
      for (int m = LPT; m < 64; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m));
      if (mx > m_run[g]) {
        const float corr = fexp2(m_run[g] - mx);
        l[g] *= corr;
        ld.rescale(g, corr);
#pragma unroll
        for (int i = 0; i < 8; ++i) o[g][i] *= corr;
        m_run[g] = mx;
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float p[G];
#pragma unroll
      for (int g = 0; g < G; ++g) {
        p[g] = s[u][g] == -INFINITY ? 0.f : fexp2(s[u][g] - m_run[g]);
        l[g] += p[g];
      }
      ld.pv(raw[u], p, o);
    }
  }
}

template <int D, int G>
__global__ __launch_bounds__(kTileThreads) void k_attn_partial(
    const SeqDesc *__restrict__ seqs, const int32_t *__restrict__ state, const int4 *__restrict__ tiles,
    const uint16_t *__restrict__ q, float *__restrict__ partials, const float *__restrict__ cbtab,
    int Hkv, float qscale) {
  constexpr int LPT = Geo<D, G>::LPT, NW = kTileThreads / 64;
  __shared__ float s_cb[32];
  __shared__ float s_q[2 * G * D];            // KVQ: q and q * tau for outlier corrections
  __shared__ float s_red[NW][G][D + 2];

  const int4 tile = tiles[blockIdx.x];
  const int seq = tile.x, h = tile.y;
  const SeqDesc &sd = seqs[seq];
  const int method = sd.method;
  const int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  const int n_act = (method == ROCKET) ? st[ST_SEL_COUNT] : st[ST_COUNT];
  const int t0 = tile.z, t1 = min(tile.w, n_act);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / LPT, sub = lane % LPT, c0 = sub * 8;
  const int Hq = Hkv * G;

  Qs<G> qv;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const U4 u = ld16(q + ((size_t)seq * Hq + h * G + g) * D + c0);
    qv.h[g][0] = u.x; qv.h[g][1] = u.y; qv.h[g][2] = u.z; qv.h[g][3] = u.w;
    unpack8(u, qv.f[g]);
  }

  float m_run[G], l[G], o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m_run[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[g][i] = 0.f;
  }

  // contiguous token range per wave, a multiple of 32 tokens (one batch)
  const int end = max(t1, t0);
  const int span = ((end - t0 + NW - 1) / NW + 31) & ~31;
  const int a = min(t0 + wave * span, end);
  const int b = min(a + span, end);

  if (method == KVQ) {
    const int nc = 1 << sd.bits;
    const float *cb = cbtab + cb_offset(sd.bits);
    if (threadIdx.x < nc) s_cb[threadIdx.x] = cb[threadIdx.x];
    if (threadIdx.x < nc) s_cb[16 + threadIdx.x] = cb[nc + threadIdx.x];
    const float2 *tt = reinterpret_cast<const float2 *>(sd.kmeta) + (size_t)h * D;
    for (int e = threadIdx.x; e < G * D; e += kTileThreads) {
      const int g = e / D, c = e % D;
      const float qx = h2f(q[((size_t)seq * Hq + h * G + g) * D + c]);
      s_q[e] = qx;
      s_q[G * D + e] = qx * tt[c].x;
    }
  }
  __syncthreads();

  if (method == FP16 || method == H2O) {
    LdRows<D, G> ld{reinterpret_cast<const uint16_t *>(sd.k) + h * stride_rows(sd, D),
                    reinterpret_cast<const uint16_t *>(sd.v) + h * stride_rows(sd, D), c0};
    float *lg = (method == H2O) ? reinterpret_cast<float *>(sd.logits) + h * stride_logits(sd, G) : nullptr;
    wave_attend<D, G>(ld, a, b, qv, qscale, m_run, l, o, grp, sub, lg);
  } else if (method == ROCKET) {
    LdGather<D, G> ld{reinterpret_cast<const uint16_t *>(sd.k) + h * stride_rows(sd, D),
                      reinterpret_cast<const uint16_t *>(sd.v) + h * stride_rows(sd, D),
                      reinterpret_cast<const int32_t *>(sd.sel) + h * stride_sel(sd), c0};
    wave_attend<D, G>(ld, a, b, qv, qscale, m_run, l, o, grp, sub, nullptr);
  } else if (method == UQ) {
    LdUQ<D, G> ld;
    ld.kc = reinterpret_cast<const uint8_t *>(sd.kc) + h * stride_codes(sd);
    ld.vc = reinterpret_cast<const uint8_t *>(sd.vc) + h * stride_codes(sd);
    ld.kmeta = reinterpret_cast<const float2 *>(sd.kmeta) + h * stride_uq_kmeta(sd, D);
    ld.vmeta = reinterpret_cast<const float2 *>(sd.vmeta) + h * stride_uq_vmeta(sd, D);
    ld.kres = reinterpret_cast<const uint16_t *>(sd.kres) + (size_t)h * 64 * D;
    ld.c0 = c0;
    ld.full = (st[ST_COUNT] / 64) * 64;
    ld.cur_blk = -1;
#pragma unroll
    for (int g = 0; g < G; ++g) ld.om[g] = 0.f;
    wave_attend<D, G>(ld, a, b, qv, qscale, m_run, l, o, grp, sub, nullptr);
    ld.finish(o);
  } else if (method == KVQ) {
    auto run = [&](auto bits_tag) {
      constexpr int BITS = decltype(bits_tag)::value;
      LdKVQ<D, G, BITS> ld;
      ld.kc = reinterpret_cast<const uint8_t *>(sd.kc) + h * stride_codes(sd);
      ld.vc = reinterpret_cast<const uint8_t *>(sd.vc) + h * stride_codes(sd);
      ld.krow = reinterpret_cast<const uint32_t *>(sd.krow) + h * stride_krow(sd);
      ld.kout = reinterpret_cast<const uint32_t *>(sd.kout) + h * stride_kout(sd);
      ld.vout = reinterpret_cast<const uint32_t *>(sd.vout) + h * stride_vout(sd);
      ld.vs = reinterpret_cast<const float *>(sd.vmeta) + h * stride_slots(sd);
      ld.cbk = s_cb;
      ld.cbv = s_cb + 16;
      ld.qlds = s_q;
      ld.c0 = c0;
      ld.rowbytes = sd.rowbytes;
      ld.nov = sd.nov_slots;
#pragma unroll
      for (int g = 0; g < G; ++g)
#pragma unroll
        for (int i = 0; i < 8; ++i) ld.qp[g][i] = s_q[G * D + g * D + c0 + i];
      wave_attend<D, G>(ld, a, b, qv, qscale, m_run, l, o, grp, sub, nullptr);
    };
    if (sd.bits == 4) run(std::integral_constant<int, 4>{});
    else if (sd.bits == 3) run(std::integral_constant<int, 3>{});
    else run(std::integral_constant<int, 2>{});
  }

  // reduce over the lane groups of the wave (they share m_run), then across waves via LDS
#pragma unroll
  for (int g = 0; g < G; ++g) {
#pragma unroll
    for (int m = LPT; m < 64; m <<= 1) {
      l[g] += __shfl_xor(l[g], m);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] += __shfl_xor(o[g][i], m);
    }
  }
  // l was accumulated once per lane of a group; every lane of a group holds the same l
  if (grp == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int i = 0; i < 8; ++i) s_red[wave][g][2 + c0 + i] = o[g][i];
      if (sub == 0) {
        s_red[wave][g][0] = m_run[g];
        s_red[wave][g][1] = l[g];
      }
    }
  }
  __syncthreads();
  float *dst = partials + (size_t)blockIdx.x * G * (D + 2);
  for (int e = threadIdx.x; e < G * (D + 2); e += kTileThreads) {
    const int g = e / (D + 2), c = e % (D + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, s_red[w][g][0]);
    float val;
    if (M == -INFINITY) {
      val = (c == 0) ? -INFINITY : 0.f;
    } else if (c == 0) {
      val = M;
    } else {
      val = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w)
        if (s_red[w][g][0] != -INFINITY) val += s_red[w][g][c] * exp2f(s_red[w][g][0] - M);
    }
    dst[e] = val;
  }
}

// Log-sum-exp merge of one (sequence, kv head)'s tiles; H2O also adds every query head's
// probability to each retained token's accumulated score.
constexpr int kMaxTilesPerPair = 64;

template <int D, int G>
__global__ __launch_bounds__(256) void k_attn_combine(const SeqDesc *__restrict__ seqs,
                                                      int32_t *__restrict__ state,
                                                      const float *__restrict__ partials,
                                                      float *__restrict__ out, int Hkv) {
  __shared__ float sm[kMaxTilesPerPair][G];
  __shared__ float sl[kMaxTilesPerPair][G];
  __shared__ float sM[G], sL[G];
  const int seq = blockIdx.x / Hkv, h = blockIdx.x % Hkv;
  const SeqDesc &sd = seqs[seq];
  const int first = sd.tile_first + h * sd.tile_count, nt = sd.tile_count;
  const float *P = partials + (size_t)first * G * (D + 2);
  for (int e = threadIdx.x; e < nt * G; e += 256) {
    const int t = e / G, g = e % G;
    sm[t][g] = P[((size_t)t * G + g) * (D + 2)];
    sl[t][g] = P[((size_t)t * G + g) * (D + 2) + 1];
  }
  __syncthreads();
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    float M = -INFINITY;
    for (int t = 0; t < nt; ++t) M = fmaxf(M, sm[t][g]);
    float L = 0.f;
    for (int t = 0; t < nt; ++t)
      if (sm[t][g] != -INFINITY) L += sl[t][g] * exp2f(sm[t][g] - M);
    sM[g] = M;
    sL[g] = L;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < nt * G; e += 256) {
    const int t = e / G, g = e % G;
    sm[t][g] = sm[t][g] == -INFINITY ? 0.f : exp2f(sm[t][g] - sM[g]) / sL[g];
  }
  __syncthreads();
  const int Hq = Hkv * G;
  for (int e = threadIdx.x; e < G * D; e += 256) {
    const int g = e / D, c = e % D;
    float acc = 0.f;
    const float *pp = P + (size_t)g * (D + 2) + 2 + c;
#pragma unroll 8
    for (int t = 0; t < nt; ++t) acc = fmaf(pp[(size_t)t * G * (D + 2)], sm[t][g], acc);
    out[((size_t)seq * Hq + h * G + g) * D + c] = acc;
  }
  if (sd.method == H2O) {
    // accumulate, and find the eviction candidate (lowest score among positions older than the
    // R most recent, lower position on a tie) for the eviction call to apply
    int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
    const int count = st[ST_COUNT];
    const int limit = st[ST_NEXT_POS] - 1 - sd.R + 1;
    const float *lg = reinterpret_cast<const float *>(sd.logits) + h * stride_logits(sd, G);
    float *score = reinterpret_cast<float *>(sd.score) + h * stride_slots(sd);
    const int32_t *pos = reinterpret_cast<const int32_t *>(sd.pos) + h * stride_slots(sd);
    float invL[G], M[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      invL[g] = 1.f / sL[g];
      M[g] = sM[g];
    }
    unsigned long long best = ~0ull;
    int best_slot = -1;
    for (int j = threadIdx.x; j < count; j += 256) {
      float acc = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) acc += exp2f(gld(lg + (size_t)j * G + g) - M[g]) * invL[g];
      const float sc = gld(score + j) + acc;
      gst(score + j, sc);
      const int pj = gld(pos + j);
      const unsigned long long key =
          ((unsigned long long)__builtin_bit_cast(uint32_t, sc) << 32) | (unsigned long long)(uint32_t)pj;
      if (pj < limit && key < best) {
        best = key;
        best_slot = j;
      }
    }
    if (count > sd.B) {
      __shared__ unsigned long long s_best[4];
      unsigned long long wb = best;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) {
        const unsigned long long x = __shfl_xor(wb, m);
        wb = x < wb ? x : wb;
      }
      if ((threadIdx.x & 63) == 0) s_best[threadIdx.x >> 6] = wb;
      __syncthreads();
      unsigned long long all = s_best[0];
      for (int w = 1; w < 4; ++w) all = s_best[w] < all ? s_best[w] : all;
      if (best_slot >= 0 && best == all) st[ST_VICTIM] = best_slot;
    }
  }
}

template <int D, int G>
hipError_t partial_impl(const Dev &dv, const Shape &sh, const uint16_t *q, hipStream_t st) {
  const float qscale = kLog2e / sqrtf((float)D);
  hipLaunchKernelGGL((k_attn_partial<D, G>), dim3(dv.n_tiles), dim3(kTileThreads), 0, st, dv.seqs,
                     dv.state, dv.tiles, q, dv.partials, dv.cbtab, sh.Hkv, qscale);
  return hipGetLastError();
}

template <int D, int G>
hipError_t combine_impl(const Dev &dv, const Shape &sh, float *out, hipStream_t st) {
  hipLaunchKernelGGL((k_attn_combine<D, G>), dim3(sh.S * sh.Hkv), dim3(256), 0, st, dv.seqs, dv.state,
                     dv.partials, out, sh.Hkv);
  return hipGetLastError();
}

}  // namespace

#define MKV_DISPATCH_DG(FN, ...)                                              \
  switch (sh.D * 16 + sh.G) {                                                 \
    case 64 * 16 + 1: return FN<64, 1>(__VA_ARGS__);                          \
    case 64 * 16 + 2: return FN<64, 2>(__VA_ARGS__);                          \
    case 64 * 16 + 4: return FN<64, 4>(__VA_ARGS__);                          \
    case 64 * 16 + 8: return FN<64, 8>(__VA_ARGS__);                          \
    case 128 * 16 + 1: return FN<128, 1>(__VA_ARGS__);                        \
    case 128 * 16 + 2: return FN<128, 2>(__VA_ARGS__);                        \
    case 128 * 16 + 4: return FN<128, 4>(__VA_ARGS__);                        \
    case 128 * 16 + 8: return FN<128, 8>(__VA_ARGS__);                        \
    default: return hipErrorInvalidValue;                                     \
  }

hipError_t launch_attention_partial(const Dev &dv, const Shape &sh, const uint16_t *q, hipStream_t st) {
  MKV_DISPATCH_DG(partial_impl, dv, sh, q, st)
}

hipError_t launch_attention_combine(const Dev &dv, const Shape &sh, float *out, hipStream_t st) {
  MKV_DISPATCH_DG(combine_impl, dv, sh, out, st)
}

}  // namespace mkv
