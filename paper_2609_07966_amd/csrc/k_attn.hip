// Split-K decode attention over a mixed-configuration KV cache, and the combine pass.
//
// Every configuration's decode step ends in softmax attention over the tokens its cache keeps
// (MetaKV Section 2.1): all tokens with dequantized values (uniform / KVQuant), the retained
// set (H2O) or the selected set (RocketKV).  One launch covers all sequences: each workgroup
// takes one tile = (sequence, kv head, token range) and runs the loop for that sequence's method;
// the 4 waves of a workgroup split the tile's tokens into contiguous ranges.
//
// Matrix path (fp16 rows, gathered rows, KVQuant): a wave handles 16 tokens per step with
// v_mfma_f32_16x16x16_f16.  q.k is S^T = K Q^T (tokens x query heads; channels permuted so a
// lane reads 32 contiguous channels of one token), and its result layout is exactly the operand
// layout of P^T in O^T = V^T P^T (channels x query heads), so probabilities feed the second
// product without moving.  KVQuant codes become packed fp16 pairs by one LDS table lookup per
// two codes (codebook entries are fp16 values); its key thresholds are folded into q and its
// value scales into p, both of which are fp32: their fp16 rounding residual rides in the spare
// columns G..2G-1 of the same product and is added back after it.  Outliers are sparse
// corrections, applied without LDS atomics (which the LDS executes one lane at a time): a
// batch's key outliers are loaded by the whole wave at once and gathered per token by lane
// shuffles; value outliers accumulate in LDS rows private to each lane and are folded into the
// output at the end.
//
// Vector path (uniform 4-bit): D/8 lanes share a token (8 channels each) and reduce q.k with DPP
// row ops; per-block key scales are folded into q once per 64-token block.
//
// Logits use the base-2 exponent (scaled by log2(e)/sqrt(d) after the dot product); each lane
// group issues the loads of 32 tokens per wave before computing any of them.
#include "kernels_common.h"

namespace mkv {

namespace {

typedef _Float16 h2v __attribute__((ext_vector_type(2)));
typedef _Float16 h4v __attribute__((ext_vector_type(4)));
typedef float f4v __attribute__((ext_vector_type(4)));

MKV_DEV float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(h2v, a), __builtin_bit_cast(h2v, b), c, false);
}

MKV_DEV h4v mk_h4(uint32_t lo, uint32_t hi) {
  return __builtin_bit_cast(h4v, ((uint64_t)hi << 32) | (uint64_t)lo);
}
MKV_DEV f4v mfma16(h4v a, h4v b, f4v c) { return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0); }
// low halves of a and b packed (a in bits 0..15), and the high halves
MKV_DEV uint32_t pk_lo(uint32_t a, uint32_t b) { return __builtin_amdgcn_perm(b, a, 0x05040100u); }
MKV_DEV uint32_t pk_hi(uint32_t a, uint32_t b) { return __builtin_amdgcn_perm(b, a, 0x07060302u); }
MKV_DEV uint32_t f16bits(float x) { return (uint32_t)__builtin_bit_cast(unsigned short, (_Float16)x); }
MKV_DEV uint32_t pk_f16(float lo, float hi) { return f16bits(lo) | (f16bits(hi) << 16); }

// ================================================================================================
// Matrix path
// ================================================================================================
// Lane roles (lr = lane % 16, lq = lane / 16):
//   q.k operand A  token row lr, channels CPL*lq + 4m + j (m = MFMA index, j = element)
//   q.k operand B  query head lr, same channels
//   S              token rows 4*lq + j, query head lr
//   p.v operand A  channel VPL*lr + m, tokens 4*lq + j
//   O^T            channel VPL*(4*lq + i) + m, query head lr
// Where q or p carry an fp16 rounding residual, the residual of head g sits in column 2G-1-g,
// so one DPP mirror (quad, half-row or row) adds it to column g.
template <int D>
struct MG {
  static constexpr int NM = D / 16;   // MFMAs per 16-token step, for q.k and for p.v
  static constexpr int CPL = D / 4;   // key channels per lane
  static constexpr int VPL = D / 16;  // value channels per lane
  static constexpr int NS = 2;        // 16-token steps per batch
};

template <int G>
MKV_DEV float mirror_cols(float x) {
  if constexpr (G == 1) return dpp<0xB1>(x);        // quad_perm [1,0,3,2]
  else if constexpr (G == 2) return dpp<0x1B>(x);   // quad_perm [3,2,1,0]
  else if constexpr (G == 4) return dpp<0x141>(x);  // row_half_mirror
  else return dpp<0x140>(x);                        // row_mirror
}

// q.k operand B per MFMA (see the kernel for its columns).
template <int D>
struct QB {
  h4v b[MG<D>::NM];
};

// fp16 rows.  Gather: token t of the tile is the t-th selected slot (RocketKV).
template <int D, int G, bool GATHER>
struct MRows {
  static constexpr int NM = MG<D>::NM, CPL = MG<D>::CPL, VPL = MG<D>::VPL;
  static constexpr bool kSplit = false;   // q and p enter as single fp16 parts
  static constexpr bool kScaled = false;  // logits still need the log2(e)/sqrt(d) factor
  const uint16_t *K, *V;
  const int32_t *sel;
  int lr, lq;
  struct Raw {
    uint32_t kw[CPL / 2];
    uint32_t vw[4][VPL / 2];
    int ks, vs[4];
  };
  struct Batch {};
  // Gather: the slots of the next batch, loaded one batch ahead so that row loads never wait
  // for their index loads
  struct Carry {
    int ks[MG<D>::NS], vs[MG<D>::NS][4];
  };
  MKV_DEV int slot_of(int t) const { return GATHER ? gld(sel + t) : t; }
  MKV_DEV void carry(int base, int b, Carry &cy) const {
    if (!GATHER) return;
#pragma unroll
    for (int s = 0; s < MG<D>::NS; ++s) {
      cy.ks[s] = gld(sel + min(base + 16 * s + lr, b - 1));
#pragma unroll
      for (int j = 0; j < 4; ++j) cy.vs[s][j] = gld(sel + min(base + 16 * s + 4 * lq + j, b - 1));
    }
  }
  MKV_DEV void load_rows(Raw &r) const {
    const uint32_t *kp = reinterpret_cast<const uint32_t *>(K + (size_t)r.ks * D + CPL * lq);
#pragma unroll
    for (int i = 0; i < CPL / 2; ++i) r.kw[i] = gld(kp + i);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t *vp = reinterpret_cast<const uint32_t *>(V + (size_t)r.vs[j] * D + VPL * lr);
#pragma unroll
      for (int i = 0; i < VPL / 2; ++i) r.vw[j][i] = gld(vp + i);
    }
  }
  // step s: FULL: all 16 tokens of the step exist; otherwise indices past the end re-read the
  // last one
  template <bool FULL>
  MKV_DEV void fetch(int base, int b, int s, const Carry &cy, Raw &r) const {
    if (GATHER) {
      r.ks = cy.ks[s];
#pragma unroll
      for (int j = 0; j < 4; ++j) r.vs[j] = cy.vs[s][j];
    } else {
      r.ks = FULL ? base + lr : min(base + lr, b - 1);
#pragma unroll
      for (int j = 0; j < 4; ++j) r.vs[j] = FULL ? base + 4 * lq + j : min(base + 4 * lq + j, b - 1);
    }
    load_rows(r);
  }
  MKV_DEV void batch_fetch(const Carry &, Batch &) const {}
  MKV_DEV void batch_fix(const Batch &) const {}
  MKV_DEV int slot(const Raw &r, int j) const { return r.vs[j]; }
  MKV_DEV void qk(const Raw &r, const QB<D> &qb, f4v &S) const {
#pragma unroll
    for (int m = 0; m < NM; ++m) S = mfma16(mk_h4(r.kw[2 * m], r.kw[2 * m + 1]), qb.b[m], S);
  }
  MKV_DEV void kfix(int, float (&)[4]) const {}
  MKV_DEV float vscale(const Raw &, int) const { return 1.f; }
  MKV_DEV void vfix(const Raw &, const float (&)[4], const float (&)[4], int) const {}
  MKV_DEV void track_max(float) {}
  MKV_DEV void pv(const Raw &r, const float (&pp)[4], f4v (&O)[NM]) const {
    const h4v P = mk_h4(pk_f16(pp[0], pp[1]), pk_f16(pp[2], pp[3]));
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      const int w = m / 2;
      const uint32_t x01 = (m & 1) ? pk_hi(r.vw[0][w], r.vw[1][w]) : pk_lo(r.vw[0][w], r.vw[1][w]);
      const uint32_t x23 = (m & 1) ? pk_hi(r.vw[2][w], r.vw[3][w]) : pk_lo(r.vw[2][w], r.vw[3][w]);
      O[m] = mfma16(mk_h4(x01, x23), P, O[m]);
    }
  }
};

// KVQuant-style b-bit codes.  Key codes: code c of a row at bit b*c, so channels (2p, 2p+1)
// form a 2b-bit field p.  Value codes: 4-token blocks with code (channel c, token j) at bit
// b*(4c + j), so the tokens (0,1) and (2,3) of a channel form two 2b-bit fields.  A field
// indexes a table of packed fp16 pairs (cb[first code], cb[second code]).
template <int D, int G, int BITS>
struct MKVQ {
  static constexpr int NM = MG<D>::NM, CPL = MG<D>::CPL, VPL = MG<D>::VPL;
  static constexpr bool kSplit = true;   // fp16 residuals of q' and p in columns G..2G-1
  static constexpr bool kScaled = true;  // q' carries log2(e)/sqrt(d)
  static constexpr int SEG = CPL * BITS;  // bits per lane segment (keys; values alike)
  // words per segment: a segment starts at bit SEG * lane_index, which is word aligned unless
  // SEG = 48 (d = 64, 3 bits), where it starts at bit 0 or 16 of a word and still spans 2 words
  static constexpr int NW = (SEG + 31) / 32;
  static constexpr int FMASK = (1 << (2 * BITS)) - 1;
  const uint8_t *kc, *vc;
  const uint32_t *krow, *kout, *vout;
  const float *vsc;
  const uint32_t *lutk, *lutv;    // LDS pair tables
  const float *cbk, *cbv;         // LDS codebooks
  const float *qq;                // LDS [D][2G]: scaled q of heads 0..G-1, then scaled q tau
  float *vcorr;                   // LDS [D]: this lane's value-outlier terms (head lr), relative to vref
  float *kcorr;                   // LDS [G][32]: this wave's key-outlier logit terms of the batch
  int lr, lq, rowbytes, nov, cap;
  int prole;                      // p operand: 0 fp16 part, 1 residual, 2 zero
  // The value-outlier terms of head lr are kept relative to a reference max vref <= m_run that
  // moves only when m_run exceeds it by more than 8 (so the terms are rarely rescaled); a term
  // computed against m_run is multiplied by vscl = 2^(m_run - vref) <= 2^8.
  float vref, vscl;
  struct Raw {
    uint32_t kw[NW], vw[NW];
    float sv[4];
    uint32_t vo[4];
    int t0;
  };
  struct Batch {
    uint32_t kr, ent;
  };
  // The key outliers of a batch's slots [base, min(base + 32, b)) are one contiguous range of
  // the pool: lane l <= 32 holds the CSR word of slot base + l (clamped to b; CSR words past the
  // count are never read), loaded one batch ahead.
  struct Carry {
    uint32_t kr;
  };
  MKV_DEV void carry(int base, int b, Carry &cy) const {
    cy.kr = gld(krow + min(base + min((int)(threadIdx.x & 63), 32), b));
  }
  // load a segment and shift it to start at bit 0 of w[0]
  MKV_DEV void seg(const uint8_t *base, int bitoff, uint32_t (&w)[NW]) const {
    const uint32_t *p = reinterpret_cast<const uint32_t *>(base) + (bitoff >> 5);
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] = gld(p + i);
    if (SEG % 32 != 0) {
      const int sh = bitoff & 31;
      w[0] = __builtin_amdgcn_alignbit(w[1], w[0], sh);
      w[1] >>= sh;
    }
  }
  // the 2b-bit field f of a segment (compile-time position once unrolled)
  MKV_DEV uint32_t field(const uint32_t (&w)[NW], int f) const {
    const int bit = 2 * BITS * f, i = bit >> 5, s = bit & 31;
    if (s + 2 * BITS <= 32) return (w[i] >> s) & FMASK;
    return __builtin_amdgcn_alignbit(w[i + 1], w[i], s) & FMASK;
  }
  // this lane's 4 tokens form one 4-token block (tile and wave ranges start at multiples of 32);
  // past the end, the last block is re-read, whose slots all lie below the slot capacity (a
  // multiple of 4)
  template <bool FULL>
  MKV_DEV void fetch(int base, int b, int, const Carry &, Raw &r) const {
    const int tk = FULL ? base + lr : min(base + lr, b - 1);
    seg(kc + (size_t)tk * rowbytes, SEG * lq, r.kw);
    const int t0 = FULL ? base + 4 * lq : min(base + 4 * lq, (b - 1) & ~3);
    r.t0 = t0;
    seg(vc + (size_t)t0 * rowbytes, SEG * lr, r.vw);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      r.sv[j] = gld(vsc + t0 + j);
      r.vo[j] = gld(vout + t0 + j);  // entry 0 of each token (slot-major entries)
    }
  }
  // lane l takes entry l of the batch's key-outlier range
  MKV_DEV void batch_fetch(const Carry &cy, Batch &bt) const {
    bt.kr = cy.kr;
    const uint32_t e0 = __builtin_amdgcn_readlane(cy.kr, 0), e1 = __builtin_amdgcn_readlane(cy.kr, 32);
    const uint32_t e = e0 + (threadIdx.x & 63);
    bt.ent = e < e1 ? gld(kout + e) : kNoOutlier;
  }
  // Lane t < 32 sums, per head, q x - q' cb[code] over the outliers of slot base + t (each
  // replaces its channel) and writes the sums to kcorr[head][t].
  MKV_DEV void batch_fix(const Batch &bt) const {
    const int lane = threadIdx.x & 63;
    const uint32_t e0 = __builtin_amdgcn_readlane(bt.kr, 0);
    const int k0 = (int)(bt.kr - e0);
    const int k1 = (int)((uint32_t)__shfl_down((int)bt.kr, 1) - e0);
    const int cnt = lane < 32 ? k1 - k0 : 0;
    float acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = 0.f;
    for (int i = 0; __any(i < cnt); ++i) {
      const int src = k0 + i;
      // entries past the 64 loaded by the wave (more than 64 in one batch) come from memory
      uint32_t ent = (uint32_t)__shfl((int)bt.ent, min(src, 63));
      if (i < cnt && src >= 64) ent = gld(kout + e0 + src);
      if (i < cnt) {
        const int ch = outlier_ch(ent);
        const float x = h2f(ent >> 16), c = cbk[outlier_code(ent)];
#pragma unroll
        for (int g = 0; g < G; ++g) acc[g] += qq[ch * 2 * G + g] * x - qq[ch * 2 * G + G + g] * c;
      }
    }
    if (lane < 32) {
#pragma unroll
      for (int g = 0; g < G; ++g) kcorr[g * 32 + lane] = acc[g];
    }
  }
  MKV_DEV int slot(const Raw &r, int j) const { return r.t0 + j; }
  MKV_DEV void qk(const Raw &r, const QB<D> &qb, f4v &S) const {
#pragma unroll
    for (int m = 0; m < NM; ++m)
      S = mfma16(mk_h4(lutk[field(r.kw, 2 * m)], lutk[field(r.kw, 2 * m + 1)]), qb.b[m], S);
  }
  // step s of the batch: this lane's tokens 16 s + 4 lq + j, head lr
  MKV_DEV void kfix(int s, float (&x)[4]) const {
    if (lr >= G) return;
    const float4 c = *reinterpret_cast<const float4 *>(kcorr + lr * 32 + 16 * s + 4 * lq);
    x[0] += c.x;
    x[1] += c.y;
    x[2] += c.z;
    x[3] += c.w;
  }
  MKV_DEV float vscale(const Raw &r, int j) const { return r.sv[j]; }
  // value outliers replace their channel: p x - p' cb[code] accumulates in this lane's LDS row
  // (an absent or masked entry adds 0 to channel 0)
  MKV_DEV void vfix(const Raw &r, const float (&p)[4], const float (&pp)[4], int valid_mask) const {
    if (lr >= G) return;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t ent = r.vo[j];
      const bool ok = ((valid_mask >> j) & 1) && ent != kNoOutlier;
      const float val = (p[j] * h2f(ent >> 16) - pp[j] * cbv[outlier_code(ent)]) * vscl;
      vcorr[ok ? outlier_ch(ent) : 0] += ok ? val : 0.f;
    }
    if (nov > 1) {  // further entries (outlier budgets above one per token)
      for (int j = 0; j < 4; ++j) {
        if (!((valid_mask >> j) & 1) || r.vo[j] == kNoOutlier) continue;
        for (int i = 1; i < nov; ++i) {
          const uint32_t ent = gld(vout + (size_t)i * cap + r.t0 + j);
          if (ent == kNoOutlier) break;
          vcorr[outlier_ch(ent)] += (p[j] * h2f(ent >> 16) - pp[j] * cbv[outlier_code(ent)]) * vscl;
        }
      }
    }
  }
  MKV_DEV void track_max(float m_run) {
    if (m_run - vref > 8.f) {
      if (lr < G && vref != -INFINITY) {
        const float f = fexp2(vref - m_run);
        float4 *row = reinterpret_cast<float4 *>(vcorr);
        for (int c = 0; c < D / 4; ++c) {
          float4 v = row[c];
          v.x *= f;
          v.y *= f;
          v.z *= f;
          v.w *= f;
          row[c] = v;
        }
      }
      vref = m_run;
    }
    vscl = fexp2(m_run - vref);
  }
  // factor that brings the terms to the final m_run (0 when there are none)
  MKV_DEV float vfactor(float m_run) const { return vref == -INFINITY ? 0.f : fexp2(vref - m_run); }
  MKV_DEV void pv(const Raw &r, const float (&pp)[4], f4v (&O)[NM]) const {
    uint32_t w[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const float a = pp[2 * i], b = pp[2 * i + 1];
      const float ah = (float)(_Float16)a, bh = (float)(_Float16)b;
      w[i] = prole == 0 ? pk_f16(ah, bh) : prole == 1 ? pk_f16(a - ah, b - bh) : 0u;
    }
    const h4v P = mk_h4(w[0], w[1]);
#pragma unroll
    for (int m = 0; m < NM; ++m)
      O[m] = mfma16(mk_h4(lutv[field(r.vw, 2 * m)], lutv[field(r.vw, 2 * m + 1)]), P, O[m]);
  }
};

// One 32-token batch of a wave.  FULL: all 32 tokens exist (no clamping, no masks).
template <bool FULL, int D, int G, class L>
MKV_DEV void mfma_batch(L &ld, int base, int b, typename L::Carry &cy, const QB<D> &qb, float qscale,
                        float &m_run, float &l_part, f4v (&O)[MG<D>::NM], float *logit_out) {
  constexpr int NS = MG<D>::NS;
  const int lane = threadIdx.x & 63, lr = lane & 15, lq = lane >> 4;
  typename L::Raw raw[NS];
  typename L::Batch bt;
  // issue order: loads that depend on the carried indices first, then this batch's rows or
  // codes, then the next batch's indices
  ld.batch_fetch(cy, bt);
#pragma unroll
  for (int s = 0; s < NS; ++s) ld.template fetch<FULL>(base + 16 * s, b, s, cy, raw[s]);
  ld.carry(base + 16 * NS, b, cy);
  ld.batch_fix(bt);
  float sc[NS][4];
  float mx = -INFINITY;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    f4v S = {0.f, 0.f, 0.f, 0.f};
    ld.qk(raw[s], qb, S);
    float x[4] = {S[0], S[1], S[2], S[3]};
    ld.kfix(s, x);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (L::kSplit) x[j] += mirror_cols<G>(x[j]);
      float v = L::kScaled ? x[j] : x[j] * qscale;
      if (!FULL) v = base + 16 * s + 4 * lq + j < b ? v : -INFINITY;
      sc[s][j] = v;
      mx = fmaxf(mx, v);
    }
  }
  if (logit_out != nullptr && lr < G) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (FULL || sc[s][j] != -INFINITY) gst(logit_out + (size_t)ld.slot(raw[s], j) * G + lr, sc[s][j]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const bool up = mx > m_run;
  if (__any(up)) {  // wave-uniform: rescale with factor 1 for the heads whose max held
    const float corr = up ? fexp2(m_run - mx) : 1.f;
    l_part *= corr;
#pragma unroll
    for (int m = 0; m < MG<D>::NM; ++m) O[m] *= corr;
    if (up) {
      m_run = mx;
      ld.track_max(m_run);
    }
  }
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    float p[4], pp[4];
    int valid_mask = 0xF;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      p[j] = fexp2(sc[s][j] - m_run);  // 0 for a masked token
      l_part += p[j];
      pp[j] = p[j] * ld.vscale(raw[s], j);
      if (!FULL) {
        // slots past the count may hold any bits: their scale must not reach the product
        const bool ok = sc[s][j] != -INFINITY;
        pp[j] = ok ? pp[j] : 0.f;
        valid_mask &= ~((ok ? 0 : 1) << j);
      }
    }
    ld.vfix(raw[s], p, pp, valid_mask);
    ld.pv(raw[s], pp, O);
  }
}

// One wave over tokens [a, b) of its tile.  m_run / l_part belong to this lane's query head
// (column lr); O holds this lane's part of O^T.
template <int D, int G, class L>
MKV_DEV void wave_mfma(L &ld, int a, int b, const QB<D> &qb, float qscale, float &m_run, float &l_part,
                       f4v (&O)[MG<D>::NM], float *logit_out) {
  if (a >= b) return;
  typename L::Carry cy;
  ld.carry(a, b, cy);
  for (int base = a; base < b; base += 16 * MG<D>::NS) {
    if (base + 16 * MG<D>::NS <= b)
      mfma_batch<true, D, G>(ld, base, b, cy, qb, qscale, m_run, l_part, O, logit_out);
    else
      mfma_batch<false, D, G>(ld, base, b, cy, qb, qscale, m_run, l_part, O, logit_out);
  }
}

// ================================================================================================
// Vector path (uniform 4-bit)
// ================================================================================================
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

// Run one wave over tokens [a, b) of its tile.
template <int D, int G, class L>
MKV_DEV void wave_attend(L &ld, int a, int b, const Qs<G> &q, float qscale, float (&m_run)[G], float (&l)[G],
                         float (&o)[G][8], int grp) {
  constexpr int LPT = Geo<D, G>::LPT, TPW = Geo<D, G>::TPW, U = Geo<D, G>::U;
  for (int base = a; base < b; base += U * TPW) {
    ld.prep(base, q);
    // every lane loads; a lane past the end of the range re-reads the range's last token, whose
    // weight below is exactly 0 (no divergent branches around the loads)
    typename L::Raw raw[U];
#pragma unroll
    for (int u = 0; u < U; ++u) ld.fetch(min(base + u * TPW + grp, b - 1), raw[u]);
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

// ================================================================================================
// The partial kernels: one over the tiles of matrix-path sequences, one over the uniform 4-bit
// ones (kept apart so that neither's register budget limits the other's occupancy).
// ================================================================================================
// Contiguous token range [a, b) of this wave within its tile, a multiple of 32 tokens.
struct WaveRange {
  int a, b;
};
MKV_DEV WaveRange wave_range(int t0, int t1, int wave, int nw) {
  const int end = max(t1, t0);
  const int span = ((end - t0 + nw - 1) / nw + 31) & ~31;
  const int a = min(t0 + wave * span, end);
  return {a, min(a + span, end)};
}

// Merge the waves' (max, sum, o) into the tile's partial.  Wave w's values sit at
// red + w * wstride as [G][D + 2].
template <int D, int G, int NW>
MKV_DEV void merge_waves(const float *red, int wstride, float *dst) {
  auto at = [&](int w, int g, int c) { return red[w * wstride + g * (D + 2) + c]; };
  for (int e = threadIdx.x; e < G * (D + 2); e += kTileThreads) {
    const int g = e / (D + 2), c = e % (D + 2);
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < NW; ++w) M = fmaxf(M, at(w, g, 0));
    float val;
    if (M == -INFINITY) {
      val = (c == 0) ? -INFINITY : 0.f;
    } else if (c == 0) {
      val = M;
    } else {
      val = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        if (at(w, g, 0) == -INFINITY) continue;
        val += at(w, g, c) * exp2f(at(w, g, 0) - M);
      }
    }
    dst[e] = val;
  }
}

template <int D, int G>
__global__ __launch_bounds__(kTileThreads) void k_attn_partial_mx(
    const SeqDesc *__restrict__ seqs, const int32_t *__restrict__ state, const int4 *__restrict__ tiles,
    const uint16_t *__restrict__ q, float *__restrict__ partials, const float *__restrict__ cbtab,
    int Hkv, float qscale, int tile_base) {
  constexpr int NW = kTileThreads / 64, NM = MG<D>::NM, CPL = MG<D>::CPL, VPL = MG<D>::VPL;
  // per wave: KVQuant value-outlier terms, one row of D per (lane quad, head) while the wave
  // runs; then the wave's (max, sum, o) for the merge
  constexpr int kWaveFloats = 4 * G * D;
  static_assert(kWaveFloats >= G * (D + 2), "wave region too small");
  __shared__ __attribute__((aligned(16))) float s_wave[NW][kWaveFloats];
  __shared__ float s_q[D][2 * G];            // KVQuant: scaled q of each head, then scaled q * tau
  __shared__ uint32_t s_lut[2][256];         // KVQuant: key and value pair tables
  __shared__ float s_cb[2][16];              // KVQuant: codebooks
  __shared__ __attribute__((aligned(16))) float s_kc[NW][G][32];  // KVQuant key-outlier logit terms

  const int tid = tile_base + blockIdx.x;
  const int4 tile = tiles[tid];
  const int seq = tile.x, h = tile.y;
  const SeqDesc &sd = seqs[seq];
  const int method = sd.method;
  const int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  const int n_act = (method == ROCKET) ? st[ST_SEL_COUNT] : st[ST_COUNT];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int Hq = Hkv * G;
  const uint16_t *qh = q + ((size_t)seq * Hq + h * G) * D;
  const WaveRange wr = wave_range(tile.z, min(tile.w, n_act), wave, NW);
  const int lr = lane & 15, lq = lane >> 4;
  const bool kvq = method == KVQ;
  if (kvq) {
    // codebook tables and q, q * tau for this kv head
    const int bits = sd.bits, nc = 1 << bits;
    const float *cb = cbtab + cb_offset(bits);
    if (threadIdx.x < 32) {
      const int which = threadIdx.x >> 4, i = threadIdx.x & 15;
      s_cb[which][i] = i < nc ? cb[which * nc + i] : 0.f;
    }
    for (int e = threadIdx.x; e < 2 * (1 << (2 * bits)); e += kTileThreads) {
      const int which = e >> (2 * bits), f = e & ((1 << (2 * bits)) - 1);
      const float *c = cb + which * nc;
      s_lut[which][f] = pk_f16(c[f & (nc - 1)], c[f >> bits]);  // first, second code of the field
    }
    const float *tau = reinterpret_cast<const float *>(sd.kmeta) + (size_t)h * D * 2;
    for (int e = threadIdx.x; e < G * D; e += kTileThreads) {
      const int g = e / D, c = e % D;
      const float qx = h2f(qh[(size_t)g * D + c]) * qscale;
      s_q[c][g] = qx;
      s_q[c][G + g] = qx * gld(tau + 2 * c);
    }
    float4 *vz = reinterpret_cast<float4 *>(&s_wave[wave][0]);
    for (int e = lane; e < kWaveFloats / 4; e += 64) vz[e] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  __syncthreads();
  // q.k operand B: query head lr, channels CPL*lq + 4m .. +3 (KVQuant: fp16 part of the scaled
  // q' in columns g < G, its residual in columns 2G-1-g)
  QB<D> qb;
#pragma unroll
  for (int m = 0; m < NM; ++m) {
    uint32_t w[2] = {0u, 0u};
    const int c = CPL * lq + 4 * m;
    if (kvq) {
      if (lr < 2 * G) {
        const int g = lr < G ? lr : 2 * G - 1 - lr;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const float x0 = s_q[c + 2 * j][G + g], x1 = s_q[c + 2 * j + 1][G + g];
          const float h0 = (float)(_Float16)x0, h1 = (float)(_Float16)x1;
          w[j] = lr < G ? pk_f16(h0, h1) : pk_f16(x0 - h0, x1 - h1);
        }
      }
    } else if (lr < G) {
      const uint32_t *qp = reinterpret_cast<const uint32_t *>(qh + (size_t)lr * D + c);
      w[0] = gld(qp);
      w[1] = gld(qp + 1);
    }
    qb.b[m] = mk_h4(w[0], w[1]);
  }
  float m_run = -INFINITY, l_part = 0.f;
  f4v O[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) O[m] = f4v{0.f, 0.f, 0.f, 0.f};
  if (method == FP16 || method == H2O) {
    MRows<D, G, false> ld;
    ld.K = reinterpret_cast<const uint16_t *>(sd.k) + h * stride_rows(sd, D);
    ld.V = reinterpret_cast<const uint16_t *>(sd.v) + h * stride_rows(sd, D);
    ld.sel = nullptr;
    ld.lr = lr;
    ld.lq = lq;
    float *lg = (method == H2O) ? reinterpret_cast<float *>(sd.logits) + h * stride_logits(sd, G) : nullptr;
    wave_mfma<D, G>(ld, wr.a, wr.b, qb, qscale, m_run, l_part, O, lg);
  } else if (method == ROCKET) {
    MRows<D, G, true> ld;
    ld.K = reinterpret_cast<const uint16_t *>(sd.k) + h * stride_rows(sd, D);
    ld.V = reinterpret_cast<const uint16_t *>(sd.v) + h * stride_rows(sd, D);
    ld.sel = reinterpret_cast<const int32_t *>(sd.sel) + h * stride_sel(sd);
    ld.lr = lr;
    ld.lq = lq;
    wave_mfma<D, G>(ld, wr.a, wr.b, qb, qscale, m_run, l_part, O, nullptr);
  } else if (kvq) {
    auto run = [&](auto bits_tag) {
      constexpr int BITS = decltype(bits_tag)::value;
      MKVQ<D, G, BITS> ld;
      ld.kc = reinterpret_cast<const uint8_t *>(sd.kc) + h * stride_codes(sd);
      ld.vc = reinterpret_cast<const uint8_t *>(sd.vc) + h * stride_codes(sd);
      ld.krow = reinterpret_cast<const uint32_t *>(sd.krow) + h * stride_krow(sd);
      ld.kout = reinterpret_cast<const uint32_t *>(sd.kout) + h * stride_kout(sd);
      ld.vout = reinterpret_cast<const uint32_t *>(sd.vout) + h * stride_vout(sd);
      ld.vsc = reinterpret_cast<const float *>(sd.vmeta) + h * stride_slots(sd);
      ld.lutk = s_lut[0];
      ld.lutv = s_lut[1];
      ld.cbk = s_cb[0];
      ld.cbv = s_cb[1];
      ld.qq = &s_q[0][0];
      ld.kcorr = &s_kc[wave][0][0];
      ld.vcorr = &s_wave[wave][(lq * G + (lr < G ? lr : 0)) * D];
      ld.lr = lr;
      ld.lq = lq;
      ld.rowbytes = sd.rowbytes;
      ld.nov = sd.nov_slots;
      ld.cap = sd.cap;
      ld.prole = lr < G ? 0 : lr < 2 * G ? 1 : 2;
      ld.vref = -INFINITY;
      ld.vscl = 1.f;
      wave_mfma<D, G>(ld, wr.a, wr.b, qb, qscale, m_run, l_part, O, nullptr);
      // fold the value-outlier rows of head lr (one per lane quad) into this lane's channels
      if (lr < G) {
        const float f = ld.vfactor(m_run);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int m = 0; m < NM; ++m) {
            const int c = VPL * (4 * lq + i) + m;
            float v = 0.f;
#pragma unroll
            for (int k = 0; k < 4; ++k) v += s_wave[wave][(k * G + lr) * D + c];
            O[m][i] += v * f;
          }
        }
      }
    };
    if (sd.bits == 4) run(std::integral_constant<int, 4>{});
    else if (sd.bits == 3) run(std::integral_constant<int, 3>{});
    else run(std::integral_constant<int, 2>{});
  }
  // KVQuant: column 2G-1-lr holds the products of head lr's p residual
  if (kvq) {
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) O[m][i] += mirror_cols<G>(O[m][i]);
  }
  // the 4 quads of a query head hold disjoint tokens
  l_part += __shfl_xor(l_part, 16);
  l_part += __shfl_xor(l_part, 32);
  // this wave's (max, sum, o) over its own region (the outlier rows were folded above; a wave's
  // LDS accesses complete in order)
  float(*red)[D + 2] = reinterpret_cast<float(*)[D + 2]>(&s_wave[wave][0]);
  if (lr < G) {
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[lr][2 + VPL * (4 * lq + i) + m] = O[m][i];
    if (lq == 0) {
      red[lr][0] = m_run;
      red[lr][1] = l_part;
    }
  }
  __syncthreads();
  merge_waves<D, G, NW>(&s_wave[0][0], kWaveFloats, partials + (size_t)tid * G * (D + 2));
}

template <int D, int G>
__global__ __launch_bounds__(kTileThreads) void k_attn_partial_uq(
    const SeqDesc *__restrict__ seqs, const int32_t *__restrict__ state, const int4 *__restrict__ tiles,
    const uint16_t *__restrict__ q, float *__restrict__ partials, int Hkv, float qscale, int tile_base) {
  constexpr int NW = kTileThreads / 64, LPT = Geo<D, G>::LPT;
  __shared__ float s_red[NW][G][D + 2];
  const int tid = tile_base + blockIdx.x;
  const int4 tile = tiles[tid];
  const int seq = tile.x, h = tile.y;
  const SeqDesc &sd = seqs[seq];
  const int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint16_t *qh = q + ((size_t)seq * Hkv * G + h * G) * D;
  const WaveRange wr = wave_range(tile.z, min(tile.w, st[ST_COUNT]), wave, NW);
  const int grp = lane / LPT, sub = lane % LPT, c0 = sub * 8;
  Qs<G> qv;
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const U4 u = gld16u(qh + (size_t)g * D + c0);
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
  wave_attend<D, G>(ld, wr.a, wr.b, qv, qscale, m_run, l, o, grp);
  ld.finish(o);
  // reduce over the lane groups of the wave (they share m_run)
#pragma unroll
  for (int g = 0; g < G; ++g) {
#pragma unroll
    for (int m = LPT; m < 64; m <<= 1) {
      l[g] += __shfl_xor(l[g], m);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] += __shfl_xor(o[g][i], m);
    }
  }
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
  merge_waves<D, G, NW>(&s_red[0][0][0], G * (D + 2), partials + (size_t)tid * G * (D + 2));
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
hipError_t partial_impl(const Dev &dv, const Shape &sh, const uint16_t *q, int part, hipStream_t st) {
  const float qscale = kLog2e / sqrtf((float)D);
  const int n_mx = dv.n_tiles - dv.n_tiles_uq;
  if (part == 0 && n_mx > 0)
    hipLaunchKernelGGL((k_attn_partial_mx<D, G>), dim3(n_mx), dim3(kTileThreads), 0, st, dv.seqs, dv.state,
                       dv.tiles, q, dv.partials, dv.cbtab, sh.Hkv, qscale, 0);
  if (part == 1 && dv.n_tiles_uq > 0)
    hipLaunchKernelGGL((k_attn_partial_uq<D, G>), dim3(dv.n_tiles_uq), dim3(kTileThreads), 0, st, dv.seqs,
                       dv.state, dv.tiles, q, dv.partials, sh.Hkv, qscale, n_mx);
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

hipError_t launch_attention_partial(const Dev &dv, const Shape &sh, const uint16_t *q, int part, hipStream_t st) {
  MKV_DISPATCH_DG(partial_impl, dv, sh, q, part, st)
}

hipError_t launch_attention_combine(const Dev &dv, const Shape &sh, float *out, hipStream_t st) {
  MKV_DISPATCH_DG(combine_impl, dv, sh, out, st)
}

}  // namespace mkv
