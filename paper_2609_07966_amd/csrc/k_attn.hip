// Split-K decode attention over a mixed-configuration KV cache, and the combine pass.
//
// Every configuration's decode step ends in softmax attention over the tokens its cache keeps
// (MetaKV Section 2.1): all tokens with dequantized values (uniform / KVQuant), the retained
// set (H2O) or the selected set (RocketKV).  One launch covers all sequences: each workgroup
// takes one tile = (sequence, kv head, token range) and runs the loop for that sequence's method;
// the 4 waves of a workgroup split the tile's tokens into contiguous ranges.  Tiles launch in an
// order chosen on the host (quantized tiles early, RocketKV's last), so a tile writes its partial
// to the slot its sequence, kv head and range give, not to its launch index.
//
// Matrix path (fp16 rows, gathered rows, KVQuant): a wave handles 16 tokens per step with
// v_mfma_f32_16x16x16_f16.  q.k is S^T = K Q^T (tokens x query heads; channels permuted so a
// lane reads 32 contiguous channels of one token), and its result layout is exactly the operand
// layout of P^T in O^T = V^T P^T (channels x query heads), so probabilities feed the second
// product without moving.  KVQuant codes become packed fp16 pairs by one LDS table lookup per
// two codes (codebook entries are fp16 values); its key thresholds are folded into q and its
// value scales into p, both of which are fp32: their fp16 rounding residual rides in the spare
// columns G..2G-1 of the same product and is added back after it.  Outliers are sparse
// corrections: the logit terms of a batch's key outliers are computed by the whole wave at once,
// one entry per lane, into LDS and summed per token by the token's lane (LDS atomics measured
// slower there); value outliers add p (x - s cb[code]) to the wave's per-head LDS rows by LDS
// atomics (private rows per lane with read-modify-write measured slower there), folded into the
// output at the end.
//
// Uniform 4-bit tiles run the same matrix loop: 4-bit codes become exact fp16 integers (one
// and-or and one packed subtraction per pair), each 64-token block's key steps are folded into q
// (computed once per channel and head across the wave and staged in LDS), each token's value
// steps into p, and the minima enter as per-head bias terms.
//
// Logits use the base-2 exponent (scaled by log2(e)/sqrt(d)).  fp16-row tiles keep the loads of
// the next 16 tokens in flight while computing the current 16; the other paths issue the loads
// of a 32-token batch before computing any of it.
#include <mutex>

#include "kernels_common.h"

// Split-K workspace of mkv_decode_attention_noalloc, for callers that cannot allocate: the
// partial (max, sum, output) of every attention tile lives here instead of in the cache arena.
// Each GPU the library runs on holds one copy until the process ends; every call on a GPU shares
// it, so calls that overlap on one GPU race.  Nothing in it needs clearing between calls: each
// tile writes its whole partial before the combine pass reads it.
static __device__ __align__(256) float scratch[mkv::kStaticScratchBytes / sizeof(float)];

namespace mkv {

namespace {
constexpr int kMaxDevices = 64;
std::once_flag g_scratch_once[kMaxDevices];
hipError_t g_scratch_err[kMaxDevices];
float *g_scratch_ptr[kMaxDevices];
}  // namespace

hipError_t static_scratch(float **ptr, size_t *bytes) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  // the array's device address on this device, looked up once with the device current (in host
  // code the name `scratch` is only a host-side stand-in and must never reach a kernel)
  std::call_once(g_scratch_once[dev], [dev] {
    void *p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch_ptr[dev] = static_cast<float *>(p);
  });
  if (g_scratch_err[dev] != hipSuccess) return g_scratch_err[dev];
  *ptr = g_scratch_ptr[dev];
  *bytes = kStaticScratchBytes;
  return hipSuccess;
}

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
MKV_DEV uint32_t pk_f16(float lo, float hi) { return __builtin_bit_cast(uint32_t, h2v{(_Float16)lo, (_Float16)hi}); }

// ================================================================================================
// Matrix path
// ================================================================================================
// Lane roles (lr = lane % 16, lq = lane / 16):
//   q.k operand A  token row lr, channels CPL*lq + 4m + j (m = MFMA index, j = element); fp16
//                  rows instead take channels 32*(m/2) + 8*lq + 4*(m%2) + j, so that the four
//                  lanes of a row read one contiguous 64-byte piece per load
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
  static constexpr int NS = MG<D>::NS;
  static constexpr bool kSplit = false;   // q and p enter as single fp16 parts
  static constexpr bool kScaled = false;  // logits still need the log2(e)/sqrt(d) factor
  const uint16_t *K, *V;
  const int32_t *sel;
  int lr, lq;
  struct Raw {
    uint32_t kw[CPL / 2];
    uint32_t vw[4][VPL / 2];
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
  MKV_DEV void load_rows(int ks, const int (&vs)[4], Raw &r) const {
    // 16-byte pieces at channels 32 i + 8 lq (i < D / 32)
    const uint32_t *kp = reinterpret_cast<const uint32_t *>(K + (size_t)ks * D + 8 * lq);
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
      for (int w = 0; w < 4; ++w) r.kw[4 * i + w] = gld(kp + 16 * i + w);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t *vp = reinterpret_cast<const uint32_t *>(V + (size_t)vs[j] * D + VPL * lr);
#pragma unroll
      for (int i = 0; i < VPL / 2; ++i) r.vw[j][i] = gld(vp + i);
    }
  }
  // slots of the step at `base` (indices past the end re-read the last token)
  MKV_DEV void index(int base, int b, int &ks, int (&vs)[4]) const {
    ks = slot_of(min(base + lr, b - 1));
#pragma unroll
    for (int j = 0; j < 4; ++j) vs[j] = slot_of(min(base + 4 * lq + j, b - 1));
  }
  // step s: FULL: all 16 tokens of the step exist; otherwise indices past the end re-read the
  // last one
  template <bool FULL>
  MKV_DEV void fetch(int base, int b, int s, const Carry &cy, Raw &r) const {
    int ks, vs[4];
    if (GATHER) {
      ks = cy.ks[s];
#pragma unroll
      for (int j = 0; j < 4; ++j) vs[j] = cy.vs[s][j];
    } else {
      ks = FULL ? base + lr : min(base + lr, b - 1);
#pragma unroll
      for (int j = 0; j < 4; ++j) vs[j] = FULL ? base + 4 * lq + j : min(base + 4 * lq + j, b - 1);
    }
    load_rows(ks, vs, r);
  }
  MKV_DEV void batch_fetch(const Carry &, Batch &) const {}
  MKV_DEV void batch_fix(const Batch &) const {}
  // slot of this lane's token j of the step at `base` (rows only: the logit store of H2O)
  MKV_DEV int slot(int base, const Raw &, int j) const { return base + 4 * lq + j; }
  MKV_DEV void qk(const Raw &r, const QB<D> &qb, f4v &S) const {
#pragma unroll
    for (int m = 0; m < NM; ++m) S = mfma16(mk_h4(r.kw[2 * m], r.kw[2 * m + 1]), qb.b[m], S);
  }
  MKV_DEV void kfix(int, float (&)[4]) const {}
  MKV_DEV float vscale(const Raw &, int) const { return 1.f; }
  MKV_DEV void vfix(const Raw &, const float (&)[4], const float (&)[4], int) const {}
  MKV_DEV void prep(int, QB<D> &) {}
  MKV_DEV void rescale(float) const {}
  MKV_DEV void pv(const Raw &r, const float (&)[4], const float (&pp)[4], int, f4v (&O)[NM]) const {
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
// form a 2b-bit field p and channels 4m..4m+3 (one matrix operand) a 4b-bit one.  Value codes:
// 4-token blocks with code (channel c, token j) at bit b*(4c + j), so a channel's 4 tokens (one
// matrix operand) form a 4b-bit field.  At 2 bits that field is one byte and indexes a table of
// packed fp16 quads; at 3 and 4 bits it is two 2b-bit fields indexing a table of packed fp16
// pairs (cb[first code], cb[second code]).  The tables are built on the host at cache creation.
template <int D, int G, int BITS>
struct MKVQ {
  static constexpr int NM = MG<D>::NM, CPL = MG<D>::CPL, VPL = MG<D>::VPL;
  static constexpr int NS = 2;           // 32-token batches (the key-outlier tags are slot mod 32)
  static constexpr bool kSplit = true;   // fp16 residual of q' in columns G..2G-1
  static constexpr bool kScaled = true;  // q' carries log2(e)/sqrt(d)
  static constexpr int SEG = CPL * BITS;  // bits per lane segment (keys; values alike)
  // words per segment: a segment starts at bit SEG * lane_index, which is word aligned unless
  // SEG = 48 (d = 64, 3 bits), where it starts at bit 0 or 16 of a word and still spans 2 words
  static constexpr int NW = (SEG + 31) / 32;
  static constexpr int FMASK = (1 << (2 * BITS)) - 1;
  // LDS row strides of the value-outlier sums and the key-outlier slot sums, padded so that the
  // heads' rows start in different banks (the same channel or slot of G heads is touched at once)
  static constexpr int VS = D + 4, KCS = 36;
  const uint8_t *kc, *vc;
  const uint32_t *krow, *kout, *vdel;
  const float *vsc;
  const uint32_t *lutk, *lutv;    // LDS tables: quads (2 words per entry) at 2 bits, else pairs
  const float *cbk;               // LDS key codebook
  const float *qq;                // LDS [D][2G]: scaled q of heads 0..G-1, then scaled q tau
  float *vacc;                    // LDS [G][VS]: this wave's value-outlier terms
  float *kterm;                   // LDS [64][G]: this wave's per-entry key-outlier logit terms
  float *kcorr;                   // LDS [G + 1][KCS]: this wave's key-outlier logit terms of the
                                  // batch (row G stays zero)
  int lr, lq, rowbytes, nov, cap;
  struct Raw {
    uint32_t kw[NW], vw[NW];
    float sv[4];
    uint32_t vd[4];
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
  // operand m of a segment: 4 codes as 4 fp16 codebook values
  MKV_DEV h4v operand(const uint32_t *lut, const uint32_t (&w)[NW], int m) const {
    if constexpr (BITS == 2) {
      const uint32_t q = (w[m >> 2] >> (8 * (m & 3))) & 0xFFu;
      const uint2 e = *reinterpret_cast<const uint2 *>(lut + 2 * q);
      return mk_h4(e.x, e.y);
    } else {
      return mk_h4(lut[field(w, 2 * m)], lut[field(w, 2 * m + 1)]);
    }
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
    const U4 s = gld16u(vsc + t0);
    r.sv[0] = __builtin_bit_cast(float, s.x);
    r.sv[1] = __builtin_bit_cast(float, s.y);
    r.sv[2] = __builtin_bit_cast(float, s.z);
    r.sv[3] = __builtin_bit_cast(float, s.w);
    const U4 e = gld16u(vdel + t0);  // entry 0 of each token (slot-major entries)
    r.vd[0] = e.x;
    r.vd[1] = e.y;
    r.vd[2] = e.z;
    r.vd[3] = e.w;
  }
  // lane l takes entry l of the batch's key-outlier range
  MKV_DEV void batch_fetch(const Carry &cy, Batch &bt) const {
    bt.kr = cy.kr;
    const uint32_t e0 = __builtin_amdgcn_readlane(cy.kr, 0), e1 = __builtin_amdgcn_readlane(cy.kr, 32);
    const uint32_t e = e0 + (threadIdx.x & 63);
    bt.ent = e < e1 ? gld(kout + e) : kNoOutlier;
  }
  // Per head, the logit correction q x - q' cb[code] of every key outlier of the batch (each
  // replaces its channel), summed per slot: lane e computes the terms of entry e of the batch's
  // range (64 entries per round) into LDS, then lane t < 32 adds those of its slot's entries
  // [k0, k1) (the CSR range; LDS atomics measured slower here) and writes the sums to kcorr.
  MKV_DEV void batch_fix(const Batch &bt) const {
    const int lane = threadIdx.x & 63;
    const uint32_t e0 = __builtin_amdgcn_readlane(bt.kr, 0), e1 = __builtin_amdgcn_readlane(bt.kr, 32);
    const int total = (int)(e1 - e0);  // wave-uniform
    const int k0 = (int)(bt.kr - e0);
    const int next = (int)((uint32_t)__shfl_down((int)bt.kr, 1) - e0);
    const int k1 = lane < 32 ? next : k0;
    float acc[G];
#pragma unroll
    for (int g = 0; g < G; ++g) acc[g] = 0.f;
    for (int r0 = 0; r0 < total; r0 += 64) {
      const bool on = r0 + lane < total;
      uint32_t ent = bt.ent;
      if (r0 > 0) ent = on ? gld(kout + e0 + r0 + lane) : kNoOutlier;
      const int ch = on ? min(outlier_ch(ent), D - 1) : 0;
      const float x = on ? h2f(ent >> 16) : 0.f, c = on ? cbk[outlier_code(ent)] : 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) kterm[lane * G + g] = qq[ch * 2 * G + g] * x - qq[ch * 2 * G + G + g] * c;
      const int a = max(k0 - r0, 0), b = min(k1 - r0, 64);
      for (int i = a; i < b; i += 4) {
        float t[4][G];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int g = 0; g < G; ++g) t[u][g] = kterm[min(i + u, 63) * G + g];
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int g = 0; g < G; ++g) acc[g] += i + u < b ? t[u][g] : 0.f;
      }
    }
    if (lane < 32) {
#pragma unroll
      for (int g = 0; g < G; ++g) kcorr[g * KCS + lane] = acc[g];
    }
  }
  MKV_DEV int slot(int, const Raw &r, int j) const { return r.t0 + j; }
  MKV_DEV void qk(const Raw &r, const QB<D> &qb, f4v &S) const {
#pragma unroll
    for (int m = 0; m < NM; ++m) S = mfma16(operand(lutk, r.kw, m), qb.b[m], S);
  }
  // step s of the batch: this lane's tokens 16 s + 4 lq + j, head lr (columns lr >= G read the
  // zero row)
  MKV_DEV void kfix(int s, float (&x)[4]) const {
    const float4 c = *reinterpret_cast<const float4 *>(kcorr + min(lr, G) * KCS + 16 * s + 4 * lq);
    x[0] += c.x;
    x[1] += c.y;
    x[2] += c.z;
    x[3] += c.w;
  }
  MKV_DEV float vscale(const Raw &r, int j) const { return r.sv[j]; }
  // value outliers replace their channel: p (x - s cb[code]) goes to the channel's LDS sum.  The
  // append stores that difference d = x - s cb[code] per outlier as a float32 whose 7 lowest
  // mantissa bits hold the channel (a relative change of d below 2^-16); 0.0 marks no outlier
  // and adds nothing to channel 0.
  MKV_DEV void vfix(const Raw &r, const float (&p)[4], const float (&)[4], int valid_mask) const {
    if (lr >= G) return;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t ent = r.vd[j];
      const bool ok = (valid_mask >> j) & 1;
      atomicAdd(vacc + lr * VS + (ok ? (int)(ent & 127u) : 0), ok ? p[j] * __builtin_bit_cast(float, ent) : 0.f);
    }
    if (nov > 1) {  // further entries (outlier budgets above one per token)
      for (int j = 0; j < 4; ++j) {
        if (!((valid_mask >> j) & 1)) continue;
        for (int i = 1; i < nov; ++i) {
          const uint32_t ent = gld(vdel + (size_t)i * cap + r.t0 + j);
          if (ent == 0u) break;
          atomicAdd(vacc + lr * VS + (int)(ent & 127u), p[j] * __builtin_bit_cast(float, ent));
        }
      }
    }
  }
  MKV_DEV void prep(int, QB<D> &) {}
  // a rescale of the running sums rescales the value-outlier terms with them (each lane quad
  // takes a quarter of its head's row)
  MKV_DEV void rescale(float corr) const {
    if (lr >= G) return;
    float4 *row = reinterpret_cast<float4 *>(vacc + lr * VS + lq * (D / 4));
#pragma unroll
    for (int c = 0; c < D / 16; ++c) {
      float4 v = row[c];
      v.x *= corr;
      v.y *= corr;
      v.z *= corr;
      v.w *= corr;
      row[c] = v;
    }
  }
  MKV_DEV void pv(const Raw &r, const float (&)[4], const float (&pp)[4], int, f4v (&O)[NM]) const {
    const h4v P = lr < G ? mk_h4(pk_f16(pp[0], pp[1]), pk_f16(pp[2], pp[3])) : mk_h4(0u, 0u);
#pragma unroll
    for (int m = 0; m < NM; ++m) O[m] = mfma16(operand(lutv, r.vw, m), P, O[m]);
  }
};

// (x & mask) | bits in one instruction (the compiler splits it in two when both are literals)
MKV_DEV uint32_t and_or(uint32_t x, uint32_t mask, uint32_t bits) {
  uint32_t r;
  asm("v_and_or_b32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "s"(mask), "v"(bits));
  return r;
}

// the 4-bit nibbles k and k + 4 of w as a packed pair of fp16 integers: one and-or sets each
// nibble into the mantissa of an fp16 base (1024 for a nibble at the foot of its 16-bit half, 64
// for one 4 bits up; nibbles 2, 3, 6 and 7 after a shift by 8), then one packed fp16 subtraction
// removes the base (both exact)
MKV_DEV uint32_t nib_pair(uint32_t w, int k) {
  const uint32_t x = k >= 2 ? w >> 8 : w;
  const bool up = k & 1;
  const h2v v = __builtin_bit_cast(h2v, and_or(x, up ? 0x00F000F0u : 0x000F000Fu, up ? 0x54005400u : 0x64006400u));
  const _Float16 base = up ? (_Float16)64.0f : (_Float16)1024.0f;
  const h2v off = {base, base};
  return __builtin_bit_cast(uint32_t, v - off);
}

// Uniform 4-bit (64-token key blocks with per-channel min and step; per-token value groups of
// 64 channels with min and step).  Codes n enter the matrix cores as exact fp16 integers:
// q.k = sum q'' n + sum q mn with q'' = q st, and p.v = sum p' n + sum p mn with p' = p st,
// the second terms kept per head (keys: per block; values: per value group).  A lane's 8 key channels of one code
// word enter in the order {0,4,1,5} and {2,6,3,7} (two nibble pairs per and-or); value codes
// are stored in the operand order (uq_vbit).  RES: the current incomplete block, whose keys
// are fp16 rows (same channel order, q'' = q).
template <int D, int G, bool RES>
struct MUQ {
  static constexpr int NM = MG<D>::NM, CPL = MG<D>::CPL;
  static constexpr int NGRP = D / 64;     // value groups
  static constexpr int KW = RES ? CPL / 2 : CPL / 8;  // key words per lane and step
  static constexpr int NS = RES ? 1 : 2;  // the fp16 block (at most 63 tokens) in 16-token batches
  static constexpr bool kSplit = true;    // fp16 residual of q'' in columns G..2G-1
  static constexpr bool kScaled = true;   // q'' carries log2(e)/sqrt(d)
  const uint8_t *kc, *vc;
  const float *kmeta, *vmeta;             // float2 pairs (min, step)
  const uint16_t *kres;
  const float *qs;                        // LDS [D][2G]: scaled q in columns 0..G-1
  float2 *vm;                             // LDS [32 * NGRP]: this wave's batch of value (min, step)
  float *km;                              // LDS [D][2]: this wave's key block (min, step) pairs
  static constexpr int SROW = D + 4;      // staging row stride (halves): rows start 2 banks apart
  _Float16 *stg;                          // LDS [2G][SROW]: this wave's q'' staging rows
  int lr, lq, prole, cur_blk;
  int next_blk;                           // the block whose (min, step) pairs `next_km` holds
  U4 next_km;                             // lanes l < D / 2: channels 2l, 2l + 1 of that block
  float kbias;                            // sum q mn of head lr for the current block
  float om[NGRP];                         // sum p mn of head lr per value group
  struct Raw {
    uint32_t kw[KW];
    uint32_t vw[NM / 2];
    int t0;  // first slot of this lane's 4-token value block
  };
  struct Batch {
    float mn, st;
  };
  struct Carry {};
  MKV_DEV void carry(int, int, Carry &) const {}
  // the batch's value (min, step) pairs, one per lane (slot base + l / NGRP, group l % NGRP),
  // staged in LDS for the p.v step (slots past the end re-read the last one)
  int bbase, bend;
  MKV_DEV void batch_fetch(const Carry &, Batch &bt) const {
    const int l = threadIdx.x & 63;
    const int t = min(bbase + l / NGRP, bend - 1);
    const float *mp = vmeta + ((size_t)t * NGRP + l % NGRP) * 2;
    bt.mn = l < 16 * NS * NGRP ? gld(mp) : 0.f;
    bt.st = l < 16 * NS * NGRP ? gld(mp + 1) : 0.f;
  }
  MKV_DEV void batch_fix(const Batch &bt) const {
    const int l = threadIdx.x & 63;
    if (l < 16 * NS * NGRP) vm[l] = make_float2(bt.mn, bt.st);
  }
  MKV_DEV int slot(int, const Raw &, int) const { return 0; }
  // offset, from the lane's first key channel CPL*lq, of element j of key operand m
  static constexpr int kofs(int m, int j) { return 8 * (m >> 1) + ((m & 1) ? 2 : 0) + ((j & 1) ? 4 : 0) + (j >> 1); }
  // rebuild the key operand B (and sum q mn) when the batch enters a new block
  MKV_DEV void prep(int base, QB<D> &qb) {
    bbase = base;
    const int blk = RES ? -2 : base >> 6;
    if (blk == cur_blk) return;
    cur_blk = blk;
    if (!RES) {
      // stage the block's (min, step) pairs, lane l taking channels 2l and 2l + 1 (loaded one
      // block ahead, the first on demand), then load the next block's (the last complete block
      // of the range at most)
      const int l = threadIdx.x & 63;
      if (l < D / 2) {
        const U4 u = next_blk == blk ? next_km : gld16u(kmeta + ((size_t)blk * D + 2 * l) * 2);
        next_blk = min(blk + 1, (bend - 1) >> 6);
        next_km = gld16u(kmeta + ((size_t)next_blk * D + 2 * l) * 2);
        float4 *dst = reinterpret_cast<float4 *>(km + 4 * l);
        *dst = make_float4(__builtin_bit_cast(float, u.x), __builtin_bit_cast(float, u.y),
                           __builtin_bit_cast(float, u.z), __builtin_bit_cast(float, u.w));
      }
    }
    if (!RES) {
      // q'' = q st of every (channel, head) computed once: lane l takes head l % G and channels
      // l / G + (64 / G) i, writes the fp16 part and the residual of each into the wave's
      // staging rows (row g: head g's parts, row 2G-1-g: its residuals; each row in operand
      // order, so that lane quad lq reads operand m as 4 halves at CPL lq + 4m), and sums
      // q mn over its channels; the sums of a head meet by xor shuffles among the lanes of the
      // same l % G, which include lane lr = g of every quad
      constexpr int LPH = 64 / G, NCH = D / LPH;  // lanes per head, channels per lane
      const int l = threadIdx.x & 63, g = l % G, k0 = l / G;
      float bias = 0.f;
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int c = k0 + LPH * i;
        const float q = qs[c * 2 * G + g];
        const float2 ms = *reinterpret_cast<const float2 *>(km + 2 * c);
        const float x = q * ms.y;
        bias += q * ms.x;
        const float hv = (float)(_Float16)x;
        const _Float16 rv = (_Float16)(x - hv);
        // operand position of channel c: quad c / CPL, then (m, j) with kofs(m, j) = c % CPL
        const int d = c % CPL;
        const int pos = (c / CPL) * CPL + 4 * (2 * (d >> 3) + ((d >> 1) & 1)) + 2 * (d & 1) + ((d >> 2) & 1);
        stg[g * SROW + pos] = (_Float16)hv;
        stg[(2 * G - 1 - g) * SROW + pos] = rv;
      }
#pragma unroll
      for (int o = G; o < 64; o *= 2) bias += __shfl_xor(bias, o);
      kbias = lr < G ? bias : 0.f;
      const _Float16 *row = stg + min(lr, 2 * G - 1) * SROW + CPL * lq;
#pragma unroll
      for (int m = 0; m < NM; ++m) {
        const h4v v = *reinterpret_cast<const h4v *>(row + 4 * m);
        qb.b[m] = lr < 2 * G ? v : mk_h4(0u, 0u);
      }
      return;
    }
    // the fp16 block (prepared once per range): q'' = q, in the lane's own column (the head
    // whose part it carries; columns >= 2G: any head, the operand is zero)
    const int g = lr < G ? lr : lr < 2 * G ? 2 * G - 1 - lr : 0;
    const float *qrow = qs + CPL * lq * 2 * G + g;  // q of channel CPL*lq + d at qrow[d * 2G]
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      uint32_t w[2];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        float hv[2], rv[2];
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          const float x = qrow[kofs(m, 2 * h2 + e) * 2 * G];
          hv[e] = (float)(_Float16)x;
          rv[e] = (float)(_Float16)(x - hv[e]);
        }
        const uint32_t ph = pk_f16(hv[0], hv[1]), pr = pk_f16(rv[0], rv[1]);
        w[h2] = prole == 0 ? ph : prole == 1 ? pr : 0u;
      }
      qb.b[m] = mk_h4(w[0], w[1]);
    }
    kbias = 0.f;
  }
  template <bool FULL>
  MKV_DEV void fetch(int base, int b, int, const Carry &, Raw &r) const {
    const int tk = FULL ? base + lr : min(base + lr, b - 1);
    if (RES) {
      const uint32_t *kp = reinterpret_cast<const uint32_t *>(kres + (size_t)(tk & 63) * D + CPL * lq);
#pragma unroll
      for (int i = 0; i < KW; ++i) r.kw[i] = gld(kp + i);
    } else {
      const uint32_t *kp = reinterpret_cast<const uint32_t *>(kc + (size_t)tk * (D / 2) + CPL * lq / 2);
#pragma unroll
      for (int i = 0; i < KW; ++i) r.kw[i] = gld(kp + i);
    }
    // the 4-token value block of this lane's tokens (past the end: the last block, whose slots
    // all lie below the capacity, a multiple of 4)
    const int t0 = FULL ? base + 4 * lq : min(base + 4 * lq, (b - 1) & ~3);
    r.t0 = t0;
    const uint32_t *vp = reinterpret_cast<const uint32_t *>(vc + (size_t)t0 * (D / 2) + lr * (D / 8));
#pragma unroll
    for (int i = 0; i < NM / 2; ++i) r.vw[i] = gld(vp + i);
  }
  MKV_DEV void qk(const Raw &r, const QB<D> &qb, f4v &S) const {
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      h4v a;
      if (RES) {
        const int u = m >> 1, o = (m & 1) ? 1 : 0;
        const uint32_t wa = r.kw[4 * u + o], wb = r.kw[4 * u + 2 + o];  // channel pairs (0|2, 1|3), (4|6, 5|7)
        a = mk_h4(pk_lo(wa, wb), pk_hi(wa, wb));
      } else {
        const uint32_t w = r.kw[m >> 1];
        a = (m & 1) ? mk_h4(nib_pair(w, 2), nib_pair(w, 3)) : mk_h4(nib_pair(w, 0), nib_pair(w, 1));
      }
      S = mfma16(a, qb.b[m], S);
    }
  }
  MKV_DEV void kfix(int, float (&x)[4]) const {
#pragma unroll
    for (int j = 0; j < 4; ++j) x[j] += kbias;
  }
  MKV_DEV float vscale(const Raw &, int) const { return 1.f; }
  MKV_DEV void vfix(const Raw &, const float (&)[4], const float (&)[4], int) const {}
  MKV_DEV void rescale(float corr) {
#pragma unroll
    for (int gr = 0; gr < NGRP; ++gr) om[gr] *= corr;
  }
  MKV_DEV void pv(const Raw &r, const float (&p)[4], const float (&)[4], int valid_mask, f4v (&O)[NM]) {
    // this lane's 4 slots r.t0 .. r.t0 + 3 within the staged batch (clamped like the loads)
    const int k0 = min(r.t0 - bbase, 16 * NS - 4);
#pragma unroll
    for (int gr = 0; gr < NGRP; ++gr) {
      float pp[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        // slots past the count may hold any bits: masked tokens contribute nothing
        const bool ok = (valid_mask >> j) & 1;
        const float2 ms = vm[(k0 + j) * NGRP + gr];
        pp[j] = ok ? p[j] * ms.y : 0.f;
        om[gr] += ok ? p[j] * ms.x : 0.f;
      }
      const h4v P = lr < G ? mk_h4(pk_f16(pp[0], pp[1]), pk_f16(pp[2], pp[3])) : mk_h4(0u, 0u);
#pragma unroll
      for (int m = 4 * gr; m < 4 * gr + 4 && m < NM; ++m) {
        const uint32_t w = r.vw[m >> 1];
        const h4v a = (m & 1) ? mk_h4(nib_pair(w, 2), nib_pair(w, 3)) : mk_h4(nib_pair(w, 0), nib_pair(w, 1));
        O[m] = mfma16(a, P, O[m]);
      }
    }
  }
};

// The running max of head lr moves only when a logit exceeds it by more than kLazyMax (log2
// units): between moves the probabilities 2^(s - m_run) stay below 2^kLazyMax, well inside fp16
// and float32, and most steps skip the cross-lane max and the rescale altogether.  The max that
// is kept is a reference for the sums, not the exact maximum; the merges of waves and tiles
// rescale by the references' differences, so the results are the same.
constexpr float kLazyMax = 8.f;

// Move head lr's reference to the wave-wide max of this step's logits (lane max `mx`) and
// rescale the sums; called wave-uniformly.
template <class L, int NM>
MKV_DEV void rescale_to(L &ld, float mx, float &m_run, float &l_part, f4v (&O)[NM]) {
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const bool up = mx > m_run;
  const float corr = up ? fexp2(m_run - mx) : 1.f;  // factor 1 for the heads whose max held
  l_part *= corr;
#pragma unroll
  for (int m = 0; m < NM; ++m) O[m] *= corr;
  ld.rescale(corr);
  if (up) m_run = mx;
}

// One 16-token step of fp16 rows (the loads of the next step are already in flight).
template <int D, int G, bool GATHER>
MKV_DEV void rows_step(const MRows<D, G, GATHER> &ld, const typename MRows<D, G, GATHER>::Raw &r, int base, int b,
                       const QB<D> &qb, float qscale, float &m_run, float &l_part, f4v (&O)[MG<D>::NM],
                       float *logit_out) {
  const int lane = threadIdx.x & 63, lr = lane & 15, lq = lane >> 4;
  f4v S = {0.f, 0.f, 0.f, 0.f};
  ld.qk(r, qb, S);
  float sc[4];
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    sc[j] = base + 4 * lq + j < b ? S[j] * qscale : -INFINITY;
    mx = fmaxf(mx, sc[j]);
  }
  if (logit_out != nullptr && lr < G) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (sc[j] != -INFINITY) gst(logit_out + (size_t)(base + 4 * lq + j) * G + lr, sc[j]);
  }
  if (__any(mx > m_run + kLazyMax)) rescale_to(ld, mx, m_run, l_part, O);
  float pp[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    pp[j] = fexp2(sc[j] - m_run);  // 0 for a masked token
    l_part += pp[j];
  }
  ld.pv(r, pp, pp, 0xF, O);
}

// fp16 rows (FP16, H2O; gathered for RocketKV) over tokens [a, b) in 16-token steps, the row
// loads of step i + 1 issued before step i is computed (and, when gathering, the slot indices
// one step further ahead).
template <int D, int G, bool GATHER>
MKV_DEV void wave_rows(const MRows<D, G, GATHER> &ld, int a, int b, const QB<D> &qb, float qscale, float &m_run,
                       float &l_part, f4v (&O)[MG<D>::NM], float *logit_out) {
  if (a >= b) return;
  typename MRows<D, G, GATHER>::Raw r0, r1;
  int ks, vs[4];
  ld.index(a, b, ks, vs);
  ld.load_rows(ks, vs, r0);
  ld.index(a + 16, b, ks, vs);
  for (int base = a; base < b; base += 32) {
    const bool more1 = base + 16 < b;
    if (more1) {
      ld.load_rows(ks, vs, r1);
      ld.index(base + 32, b, ks, vs);
    }
    rows_step(ld, r0, base, b, qb, qscale, m_run, l_part, O, logit_out);
    if (!more1) break;
    if (base + 32 < b) {
      ld.load_rows(ks, vs, r0);
      ld.index(base + 48, b, ks, vs);
    }
    rows_step(ld, r1, base + 16, b, qb, qscale, m_run, l_part, O, logit_out);
  }
}

// One 32-token batch of a wave.  FULL: all 32 tokens exist (no clamping, no masks).
template <bool FULL, int D, int G, class L>
MKV_DEV void mfma_batch(L &ld, int base, int b, typename L::Carry &cy, QB<D> &qb, float qscale,
                        float &m_run, float &l_part, f4v (&O)[MG<D>::NM], float *logit_out) {
  constexpr int NS = L::NS;
  const int lane = threadIdx.x & 63, lr = lane & 15, lq = lane >> 4;
  typename L::Raw raw[NS];
  typename L::Batch bt;
  ld.prep(base, qb);
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
        if (FULL || sc[s][j] != -INFINITY) gst(logit_out + (size_t)ld.slot(base + 16 * s, raw[s], j) * G + lr, sc[s][j]);
  }
  if (__any(mx > m_run + kLazyMax)) rescale_to(ld, mx, m_run, l_part, O);
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
    ld.pv(raw[s], p, pp, valid_mask, O);
  }
}

// One wave over tokens [a, b) of its tile.  m_run / l_part belong to this lane's query head
// (column lr); O holds this lane's part of O^T.
template <int D, int G, class L>
MKV_DEV void wave_mfma(L &ld, int a, int b, QB<D> &qb, float qscale, float &m_run, float &l_part,
                       f4v (&O)[MG<D>::NM], float *logit_out) {
  if (a >= b) return;
  typename L::Carry cy;
  ld.carry(a, b, cy);
  for (int base = a; base < b; base += 16 * L::NS) {
    if (base + 16 * L::NS <= b)
      mfma_batch<true, D, G>(ld, base, b, cy, qb, qscale, m_run, l_part, O, logit_out);
    else
      mfma_batch<false, D, G>(ld, base, b, cy, qb, qscale, m_run, l_part, O, logit_out);
  }
}

// ================================================================================================
// The partial kernel: one launch over the tiles of every sequence, whatever its method.
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
        val += at(w, g, c) * fexp2(at(w, g, 0) - M);  // argument <= 0
      }
    }
    dst[e] = val;
  }
}

template <int D, int G>
__global__ __launch_bounds__(kTileThreads) void k_attn_partial_mx(
    const SeqDesc *__restrict__ seqs, const int32_t *__restrict__ state, const int4 *__restrict__ tiles,
    const uint16_t *__restrict__ q, float *__restrict__ partials, const float *__restrict__ cbtab,
    int Hkv, float qscale) {
  constexpr int NW = kTileThreads / 64, NM = MG<D>::NM, CPL = MG<D>::CPL, VPL = MG<D>::VPL;
  // per wave: KVQuant value-outlier terms [G][D] while the wave runs; then the wave's (max,
  // sum, o) for the merge
  constexpr int kWaveFloats = G * (D + 4);  // holds [G][D + 2] for the merge
  static_assert(2 * G * (D + 4) * 2 <= kWaveFloats * 4, "uniform 4-bit q'' staging fits the wave region");
  __shared__ __attribute__((aligned(16))) float s_wave[NW][kWaveFloats];
  __shared__ float s_q[D][2 * G];            // KVQuant: scaled q of each head, then scaled q * tau
  __shared__ __attribute__((aligned(16))) uint32_t s_lut[1024];  // KVQuant: key, then value table
  __shared__ float s_cbk[16];                // KVQuant: key codebook
  __shared__ __attribute__((aligned(16))) float s_kt[NW][64 * G];  // KVQuant per-entry key-outlier terms
  __shared__ __attribute__((aligned(16))) float s_kc[NW][G + 1][36];  // KVQuant key-outlier logit terms
  __shared__ float2 s_vm[NW][64];            // uniform 4-bit: a batch's value (min, step) pairs
  __shared__ __attribute__((aligned(16))) float s_km[NW][2 * D];  // uniform 4-bit: a key block's pairs

  const int tid = blockIdx.x;
  const int4 tile = tiles[tid];
  const int seq = tile.x, h = tile.y;
  const SeqDesc &sd = seqs[seq];
  const int method = sd.method;
  const int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  // both counts are read alongside the descriptor (not after it), then chosen by method
  const int n_cnt = st[ST_COUNT], n_sel = st[ST_SEL_COUNT];
  const int n_act = (method == ROCKET) ? n_sel : n_cnt;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int Hq = Hkv * G;
  const uint16_t *qh = q + ((size_t)seq * Hq + h * G) * D;
  const WaveRange wr = wave_range(tile.z, min(tile.w, n_act), wave, NW);
  const int lr = lane & 15, lq = lane >> 4;
  const bool kvq = method == KVQ;
  const bool uq = method == UQ;
  // Set-up: every global read of the tile's set-up is issued before any of it is used (the
  // reads are independent, so the tile waits for one round trip, not one per read).
  constexpr int kQI = (G * D + kTileThreads - 1) / kTileThreads;  // q elements per thread
  // both lookup tables of a codebook take at most 256 uint4 (the 2-bit quad tables)
  static_assert(kTileThreads >= 256, "one uint4 of the lookup tables per thread");
  if (uq || kvq) {
    uint16_t qv[kQI];
    float tv[kQI];
#pragma unroll
    for (int i = 0; i < kQI; ++i) {
      const int e = min((int)threadIdx.x + i * kTileThreads, G * D - 1);
      qv[i] = qh[(size_t)(e / D) * D + e % D];
    }
    uint4 lv = make_uint4(0u, 0u, 0u, 0u);
    int nlut = 0;
    float cbv = 0.f;
    if (kvq) {
      // tau per channel, the codebook's lookup tables (copied as built on the host) and the key
      // codebook
      const float *tau = reinterpret_cast<const float *>(sd.kmeta) + (size_t)h * D * 2;
#pragma unroll
      for (int i = 0; i < kQI; ++i) tv[i] = gld(tau + 2 * ((threadIdx.x + i * kTileThreads) % D));
      const int bits = sd.bits, nc = 1 << bits;
      const uint32_t *lut = reinterpret_cast<const uint32_t *>(cbtab + kLutBase) + lut_offset(bits);
      nlut = lut_half_words(bits) / 2;
      if ((int)threadIdx.x < nlut) lv = gld16(lut + 4 * threadIdx.x);
      if (threadIdx.x < 16 && (int)threadIdx.x < nc) cbv = cbtab[cb_offset(bits) + threadIdx.x];
      // cleared per-wave outlier rows
      float4 *vz = reinterpret_cast<float4 *>(&s_wave[wave][0]);
      for (int e = lane; e < kWaveFloats / 4; e += 64) vz[e] = make_float4(0.f, 0.f, 0.f, 0.f);
      float4 *kz = reinterpret_cast<float4 *>(&s_kc[wave][0][0]);
      for (int e = lane; e < (G + 1) * 36 / 4; e += 64) kz[e] = make_float4(0.f, 0.f, 0.f, 0.f);
      if ((int)threadIdx.x < nlut) reinterpret_cast<uint4 *>(s_lut)[threadIdx.x] = lv;
      if (threadIdx.x < 16) s_cbk[threadIdx.x] = cbv;
    }
    // q of each head (scaled), and for KVQuant q * tau
#pragma unroll
    for (int i = 0; i < kQI; ++i) {
      const int e = threadIdx.x + i * kTileThreads;
      if (e < G * D) {
        const int g = e / D, c = e % D;
        const float qx = h2f(qv[i]) * qscale;
        s_q[c][g] = qx;
        if (kvq) s_q[c][G + g] = qx * tv[i];
      }
    }
  }
  __syncthreads();
  // q.k operand B: query head lr, channels CPL*lq + 4m .. +3 (KVQuant: fp16 part of the scaled
  // q' in columns g < G, its residual in columns 2G-1-g)
  QB<D> qb;
  if (kvq) {
    const int g = lr < G ? lr : lr < 2 * G ? 2 * G - 1 - lr : 0;
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      const int c = CPL * lq + 4 * m;
      uint32_t w[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const float x0 = s_q[c + 2 * j][G + g], x1 = s_q[c + 2 * j + 1][G + g];
        const float h0 = (float)(_Float16)x0, h1 = (float)(_Float16)x1;
        w[j] = lr < G ? pk_f16(h0, h1) : lr < 2 * G ? pk_f16(x0 - h0, x1 - h1) : 0u;
      }
      qb.b[m] = mk_h4(w[0], w[1]);
    }
  } else {
    uint32_t w[NM][2];
#pragma unroll
    for (int m = 0; m < NM; ++m) {
      const int c = 32 * (m / 2) + 8 * lq + 4 * (m % 2);
      const uint32_t *qp = reinterpret_cast<const uint32_t *>(qh + (size_t)min(lr, G - 1) * D + c);
      w[m][0] = gld(qp);  // lanes lr >= G read head G - 1 and drop it
      w[m][1] = gld(qp + 1);
    }
#pragma unroll
    for (int m = 0; m < NM; ++m) qb.b[m] = lr < G ? mk_h4(w[m][0], w[m][1]) : mk_h4(0u, 0u);
  }
  float m_run = -INFINITY, l_part = 0.f;
  float uq_om[D / 64];  // uniform 4-bit: sum p mn per value group (summed over the lane quads)
  f4v O[NM];
#pragma unroll
  for (int m = 0; m < NM; ++m) O[m] = f4v{0.f, 0.f, 0.f, 0.f};
  auto run_uq = [&]() {
    // the complete 64-token blocks, then the incomplete block's fp16 keys (a batch never spans
    // both: ranges start at multiples of 32)
    const int full = (st[ST_COUNT] / 64) * 64;
    auto init = [&](auto &ld) {
      ld.kc = reinterpret_cast<const uint8_t *>(sd.kc) + h * stride_codes(sd);
      ld.vc = reinterpret_cast<const uint8_t *>(sd.vc) + h * stride_codes(sd);
      ld.kmeta = reinterpret_cast<const float *>(sd.kmeta) + h * stride_uq_kmeta(sd, D) * 2;
      ld.vmeta = reinterpret_cast<const float *>(sd.vmeta) + h * stride_uq_vmeta(sd, D) * 2;
      ld.kres = reinterpret_cast<const uint16_t *>(sd.kres) + (size_t)h * 64 * D;
      ld.qs = &s_q[0][0];
      ld.vm = s_vm[wave];
      ld.km = s_km[wave];
      ld.stg = reinterpret_cast<_Float16 *>(&s_wave[wave][0]);
      ld.lr = lr;
      ld.lq = lq;
      ld.prole = lr < G ? 0 : lr < 2 * G ? 1 : 2;
      ld.cur_blk = -1;
      ld.next_blk = -1;
      ld.kbias = 0.f;
    };
    MUQ<D, G, false> lq_;
    init(lq_);
    lq_.bend = min(wr.b, full);
#pragma unroll
    for (int gr = 0; gr < D / 64; ++gr) lq_.om[gr] = 0.f;
    wave_mfma<D, G>(lq_, wr.a, min(wr.b, full), qb, qscale, m_run, l_part, O, nullptr);
    MUQ<D, G, true> lr_;
    init(lr_);
    lr_.bend = wr.b;
#pragma unroll
    for (int gr = 0; gr < D / 64; ++gr) lr_.om[gr] = lq_.om[gr];
    wave_mfma<D, G>(lr_, max(wr.a, full), wr.b, qb, qscale, m_run, l_part, O, nullptr);
#pragma unroll
    for (int gr = 0; gr < D / 64; ++gr) {
      float v = lr_.om[gr];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      uq_om[gr] = v;
    }
  };
  if (uq) {
    run_uq();
  } else if (method == FP16 || method == H2O) {
    MRows<D, G, false> ld;
    ld.K = reinterpret_cast<const uint16_t *>(sd.k) + h * stride_rows(sd, D);
    ld.V = reinterpret_cast<const uint16_t *>(sd.v) + h * stride_rows(sd, D);
    ld.sel = nullptr;
    ld.lr = lr;
    ld.lq = lq;
    float *lg = (method == H2O) ? reinterpret_cast<float *>(sd.logits) + h * stride_logits(sd, G) : nullptr;
    wave_rows<D, G, false>(ld, wr.a, wr.b, qb, qscale, m_run, l_part, O, lg);
  } else if (method == ROCKET) {
    MRows<D, G, true> ld;
    ld.K = reinterpret_cast<const uint16_t *>(sd.k) + h * stride_rows(sd, D);
    ld.V = reinterpret_cast<const uint16_t *>(sd.v) + h * stride_rows(sd, D);
    ld.sel = reinterpret_cast<const int32_t *>(sd.sel) + h * stride_sel(sd);
    ld.lr = lr;
    ld.lq = lq;
    wave_rows<D, G, true>(ld, wr.a, wr.b, qb, qscale, m_run, l_part, O, nullptr);
  } else if (kvq) {
    auto run = [&](auto bits_tag) {
      constexpr int BITS = decltype(bits_tag)::value;
      MKVQ<D, G, BITS> ld;
      ld.kc = reinterpret_cast<const uint8_t *>(sd.kc) + h * stride_codes(sd);
      ld.vc = reinterpret_cast<const uint8_t *>(sd.vc) + h * stride_codes(sd);
      ld.krow = reinterpret_cast<const uint32_t *>(sd.krow) + h * stride_krow(sd);
      ld.kout = reinterpret_cast<const uint32_t *>(sd.kout) + h * stride_kout(sd);
      ld.vdel = reinterpret_cast<const uint32_t *>(sd.vdel) + h * stride_vout(sd);
      ld.vsc = reinterpret_cast<const float *>(sd.vmeta) + h * stride_slots(sd);
      ld.lutk = s_lut;
      ld.lutv = s_lut + lut_half_words(BITS);
      ld.cbk = s_cbk;
      ld.qq = &s_q[0][0];
      ld.kcorr = &s_kc[wave][0][0];
      ld.kterm = s_kt[wave];
      ld.vacc = &s_wave[wave][0];
      ld.lr = lr;
      ld.lq = lq;
      ld.rowbytes = sd.rowbytes;
      ld.nov = sd.nov_slots;
      ld.cap = sd.cap;
      wave_mfma<D, G>(ld, wr.a, wr.b, qb, qscale, m_run, l_part, O, nullptr);
      // fold the value-outlier terms of head lr into this lane's channels (the wave's LDS
      // accesses complete in order, so the merge may reuse the region afterwards)
      if (lr < G) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
#pragma unroll
          for (int m = 0; m < NM; ++m) O[m][i] += s_wave[wave][lr * (D + 4) + VPL * (4 * lq + i) + m];
        }
      }
    };
    if (sd.bits == 4) run(std::integral_constant<int, 4>{});
    else if (sd.bits == 3) run(std::integral_constant<int, 3>{});
    else run(std::integral_constant<int, 2>{});
  }
  if (uq) {
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i) O[m][i] += uq_om[m / 4];
  }
  // the 4 quads of a query head hold disjoint tokens
  l_part += __shfl_xor(l_part, 16);
  l_part += __shfl_xor(l_part, 32);
  // this wave's (max, sum, o) over its own region (the outlier terms were folded above)
  float(*red)[D + 2] = reinterpret_cast<float(*)[D + 2]>(&s_wave[wave][0]);
  if (lr < G) {
    // O^T row 4 lq + i of operand m: channel VPL (4 lq + i) + m; uniform 4-bit values use the
    // group-aligned order 64 (m / 4) + 4 (4 lq + i) + m % 4
#pragma unroll
    for (int m = 0; m < NM; ++m)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        red[lr][2 + (uq ? 64 * (m / 4) + 4 * (4 * lq + i) + (m & 3) : VPL * (4 * lq + i) + m)] = O[m][i];
    if (lq == 0) {
      red[lr][0] = m_run;
      red[lr][1] = l_part;
    }
  }
  __syncthreads();
  // the tile's partial slot (tiles launch in an order of their own)
  const int slot = sd.tile_first + h * sd.tile_count + tile.z / sd.chunk;
  merge_waves<D, G, NW>(&s_wave[0][0], kWaveFloats, partials + (size_t)slot * G * (D + 2));
}

// Log-sum-exp merge of one (sequence, kv head)'s tiles, and for H2O the score accumulation and the
// eviction candidates, over a work list (int4: seq, kv head, part, parts).  Part 0 merges the
// output.  An H2O kv head has one part per kCombineSlots slots: each adds every query head's
// probability to the accumulated score of its slots and writes its own eviction candidate, the
// lowest (score, position) key among the positions older than the R most recent (none while the
// head is within its budget); the next decode append takes the lowest candidate's slot.  512
// threads: a wave per query head reduces the tile maxima and sums while every thread's output
// values and slot data are already in flight, so a part waits for one round of loads.
constexpr int kMaxTilesPerPair = 64;
constexpr int kCombineThreads = 512;

template <int D, int G>
__global__ __launch_bounds__(kCombineThreads) void k_attn_combine(const SeqDesc *__restrict__ seqs,
                                                                  const int32_t *__restrict__ state,
                                                                  const int4 *__restrict__ items,
                                                                  const float *__restrict__ partials,
                                                                  float *__restrict__ out, int Hkv) {
  constexpr int NWC = kCombineThreads / 64;
  static_assert(G <= NWC, "a wave per query head");
  constexpr int kChunk = 32;  // tiles whose output loads a thread issues together
  constexpr int kU = kCombineSlots / kCombineThreads;  // H2O slots per thread
  static_assert(kU * kCombineThreads == kCombineSlots, "whole slots per thread");
  __shared__ float sW[kMaxTilesPerPair][G];  // tile weights 2^(m_t - M) / L
  __shared__ float sM[G], sL[G];
  __shared__ unsigned long long s_best[NWC];
  __shared__ int s_bslot[NWC];
  const int4 it = items[blockIdx.x];
  const int seq = it.x, h = it.y, part = it.z;
  const SeqDesc &sd = seqs[seq];
  const int first = sd.tile_first + h * sd.tile_count, nt = sd.tile_count;
  const float *P = partials + (size_t)first * G * (D + 2);
  const int wv = threadIdx.x >> 6, ln = threadIdx.x & 63;
  const bool merge = part == 0;
  const bool h2o = sd.method == H2O;
  const int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
  const float *lg = reinterpret_cast<const float *>(sd.logits) + h * stride_logits(sd, G);
  float *score = reinterpret_cast<float *>(sd.score) + h * stride_slots(sd);
  const int32_t *pos = reinterpret_cast<const int32_t *>(sd.pos) + h * stride_slots(sd);
  // loads in the order they are needed: tile maxima and sums (wave g, lane t: tile t, nt <= 64),
  // part 0's output values of the first kChunk tiles, then an H2O part's slot data (every slot
  // below the capacity is allocated, so these need not wait for the count)
  float tm = -INFINITY, tl = 0.f;
  if (wv < G && ln < nt) {
    tm = P[((size_t)ln * G + wv) * (D + 2)];
    tl = P[((size_t)ln * G + wv) * (D + 2) + 1];
  }
  constexpr int kE = (G * D + kCombineThreads - 1) / kCombineThreads;  // output elements per thread
  float o0[kE][kChunk];
  if (merge) {
#pragma unroll
    for (int i = 0; i < kE; ++i) {
      const int e = min((int)threadIdx.x + i * kCombineThreads, G * D - 1);
      const float *po = P + (size_t)(e / D) * (D + 2) + 2 + e % D;
#pragma unroll
      for (int u = 0; u < kChunk; ++u) o0[i][u] = po[(size_t)min(u, nt - 1) * G * (D + 2)];
    }
  }
  int count = 0, limit = 0;
  const int j0 = part * kCombineSlots + (int)threadIdx.x;
  float lgv[kU][G], scv[kU];
  int pv[kU];
  if (h2o) {
    count = st[ST_COUNT];
    limit = st[ST_NEXT_POS] - 1 - sd.R + 1;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int j = min(j0 + u * kCombineThreads, sd.cap - 1);
#pragma unroll
      for (int g = 0; g < G; ++g) lgv[u][g] = gld(lg + (size_t)j * G + g);
      scv[u] = gld(score + j);
      pv[u] = gld(pos + j);
    }
  }
  if (wv < G) {
    const float M = wave_max(tm);
    const float L = wave_sum_rows(tm != -INFINITY ? tl * fexp2(tm - M) : 0.f);  // arguments <= 0
    if (ln < nt) sW[ln][wv] = tm == -INFINITY ? 0.f : fexp2(tm - M) / L;
    if (ln == 0) {
      sM[wv] = M;
      sL[wv] = L;
    }
  }
  __syncthreads();
  if (merge) {
    const int Hq = Hkv * G;
#pragma unroll
    for (int i = 0; i < kE; ++i) {
      const int e = (int)threadIdx.x + i * kCombineThreads;
      if (e < G * D) {
        const int g = e / D, c = e % D;
        float acc = 0.f;
#pragma unroll
        for (int u = 0; u < kChunk; ++u)
          if (u < nt) acc = fmaf(o0[i][u], sW[u][g], acc);
        const float *po = P + (size_t)g * (D + 2) + 2 + c;
        for (int t0 = kChunk; t0 < nt; t0 += kChunk) {  // more than kChunk tiles
          float o[kChunk];
#pragma unroll
          for (int u = 0; u < kChunk; ++u) o[u] = po[(size_t)min(t0 + u, nt - 1) * G * (D + 2)];
#pragma unroll
          for (int u = 0; u < kChunk; ++u)
            if (t0 + u < nt) acc = fmaf(o[u], sW[t0 + u][g], acc);
        }
        out[((size_t)seq * Hq + h * G + g) * D + c] = acc;
      }
    }
  }
  if (h2o) {
    float invL[G], M[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      invL[g] = 1.f / sL[g];
      M[g] = sM[g];
    }
    unsigned long long best = ~0ull;
    int best_slot = -1;
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int j = j0 + u * kCombineThreads;
      float acc = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) acc += fexp2(lgv[u][g] - M[g]) * invL[g];  // arguments <= 0
      const float sc = scv[u] + acc;
      if (j < count) gst(score + j, sc);
      const unsigned long long key =
          ((unsigned long long)__builtin_bit_cast(uint32_t, sc) << 32) | (unsigned long long)(uint32_t)pv[u];
      if (j < count && pv[u] < limit && key < best) {
        best = key;
        best_slot = j;
      }
    }
    if (count <= sd.B) best = ~0ull;  // within the budget: no eviction
    const unsigned long long wb = wave_min_u64(best);
    if (ln == 0) s_best[wv] = wb;
    if (wb != ~0ull && best == wb) s_bslot[wv] = best_slot;  // keys carry the position: one lane
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long all = ~0ull;
      int slot = -1;
      for (int w = 0; w < NWC; ++w)
        if (s_best[w] < all) {
          all = s_best[w];
          slot = s_bslot[w];
        }
      uint32_t *vb = reinterpret_cast<uint32_t *>(sd.vbest) + ((size_t)h * sd.vparts + part) * 4;
      gst(vb, (uint32_t)all);
      gst(vb + 1, (uint32_t)(all >> 32));
      gst(vb + 2, (uint32_t)slot);
      gst(vb + 3, 0u);
    }
  }
}

template <int D, int G>
hipError_t partial_impl(const Dev &dv, const Shape &sh, const uint16_t *q, hipStream_t st, LaunchEv ev) {
  const float qscale = kLog2e / sqrtf((float)D);
  if (dv.n_tiles > 0)
    hipExtLaunchKernelGGL((k_attn_partial_mx<D, G>), dim3(dv.n_tiles), dim3(kTileThreads), 0, st, ev.start, ev.stop,
                          0, dv.seqs, dv.state, dv.tiles, q, dv.partials, dv.cbtab, sh.Hkv, qscale);
  return hipGetLastError();
}

template <int D, int G>
hipError_t combine_impl(const Dev &dv, const Shape &sh, float *out, hipStream_t st, LaunchEv ev) {
  hipExtLaunchKernelGGL((k_attn_combine<D, G>), dim3(dv.n_comb), dim3(kCombineThreads), 0, st, ev.start,
                        ev.stop, 0, dv.seqs, dv.state, dv.comb, dv.partials, out, sh.Hkv);
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

hipError_t launch_attention_partial(const Dev &dv, const Shape &sh, const uint16_t *q, hipStream_t st,
                                    LaunchEv ev) {
  MKV_DISPATCH_DG(partial_impl, dv, sh, q, st, ev)
}

hipError_t launch_attention_combine(const Dev &dv, const Shape &sh, float *out, hipStream_t st, LaunchEv ev) {
  MKV_DISPATCH_DG(combine_impl, dv, sh, out, st, ev)
}

}  // namespace mkv
