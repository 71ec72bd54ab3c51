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
// bytes), so a wave instruction reads whole rows of D/8 * 16 bytes for 64/(D/8) consecutive
// tokens.  q . k is reduced over the lane group with DPP row ops, the running maximum is kept
// wave-uniform so the rescale branch is uniform, and p . v accumulates in registers.  Logits
// use the base-2 exponent (q is pre-scaled by log2(e) / sqrt(d)).
#include "kernels_common.h"

namespace mkv {

namespace {

template <int D>
struct Geo {
  static constexpr int LPT = D / 8;      // lanes per token
  static constexpr int TPW = 64 / LPT;   // tokens per wave step
};

// ---- per-method token loaders: fill kf[8], vf[8] for channels c0..c0+7 of token t ----------

template <int D>
struct LoadFP16 {
  const uint16_t *K, *V;
  int c0;
  MKV_DEV void block(int) {}
  MKV_DEV int slot(int t) const { return t; }
  MKV_DEV void load(int t, float *kf, float *vf) const {
    const uint4 a = *reinterpret_cast<const uint4 *>(K + (size_t)t * D + c0);
    const uint4 b = *reinterpret_cast<const uint4 *>(V + (size_t)t * D + c0);
    unpack8(a, kf);
    unpack8(b, vf);
  }
};

template <int D>
struct LoadGather {  // RocketKV: token t of the tile is the t-th selected slot
  const uint16_t *K, *V;
  const int32_t *sel;
  int c0;
  MKV_DEV void block(int) {}
  MKV_DEV int slot(int t) const { return sel[t]; }
  MKV_DEV void load(int t, float *kf, float *vf) const {
    const int s = sel[t];
    const uint4 a = *reinterpret_cast<const uint4 *>(K + (size_t)s * D + c0);
    const uint4 b = *reinterpret_cast<const uint4 *>(V + (size_t)s * D + c0);
    unpack8(a, kf);
    unpack8(b, vf);
  }
};

template <int D>
struct LoadUQ {  // 4-bit uniform: keys per (64-token block, channel), values per (token, 64 channels)
  const uint8_t *kc, *vc;
  const float2 *kmeta, *vmeta;
  const uint16_t *kres;
  int c0, full;
  float kmn[8], kst[8];
  MKV_DEV void block(int blk) {
    if (blk * 64 < full) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float2 m = kmeta[(size_t)blk * D + c0 + i];
        kmn[i] = m.x;
        kst[i] = m.y;
      }
    }
  }
  MKV_DEV int slot(int t) const { return t; }
  MKV_DEV void load(int t, float *kf, float *vf) const {
    if (t < full) {
      const uint32_t w = *reinterpret_cast<const uint32_t *>(kc + (size_t)t * (D / 2) + c0 / 2);
#pragma unroll
      for (int i = 0; i < 8; ++i) kf[i] = fmaf((float)((w >> (4 * i)) & 15u), kst[i], kmn[i]);
    } else {
      const uint4 a = *reinterpret_cast<const uint4 *>(kres + (size_t)(t & 63) * D + c0);
      unpack8(a, kf);
    }
    const uint32_t w = *reinterpret_cast<const uint32_t *>(vc + (size_t)t * (D / 2) + c0 / 2);
    const float2 m = vmeta[(size_t)t * (D / 64) + c0 / 64];
#pragma unroll
    for (int i = 0; i < 8; ++i) vf[i] = fmaf((float)((w >> (4 * i)) & 15u), m.y, m.x);
  }
};

template <int D>
struct LoadKVQ {  // KVQuant-style: codebook in LDS, per-channel key threshold, per-token value scale
  const uint8_t *kc, *vc;
  const uint32_t *krow, *kout, *vout;
  const float *vs;
  const float *cbk, *cbv;  // LDS
  int c0, bits, rowbytes, nov;
  float tau[8];
  MKV_DEV void block(int) {}
  MKV_DEV int slot(int t) const { return t; }
  MKV_DEV void codes8(const uint8_t *row, int *code) const {
    if (bits == 4) {
      const uint32_t w = *reinterpret_cast<const uint32_t *>(row + c0 / 2);
#pragma unroll
      for (int i = 0; i < 8; ++i) code[i] = (w >> (4 * i)) & 15u;
    } else if (bits == 2) {
      const uint32_t w = *reinterpret_cast<const uint16_t *>(row + c0 / 4);
#pragma unroll
      for (int i = 0; i < 8; ++i) code[i] = (w >> (2 * i)) & 3u;
    } else {
      const uint32_t lo = *reinterpret_cast<const uint16_t *>(row + c0 / 4);
      const uint32_t hi = row[D / 4 + c0 / 8];
#pragma unroll
      for (int i = 0; i < 8; ++i) code[i] = ((lo >> (2 * i)) & 3u) | (((hi >> i) & 1u) << 2);
    }
  }
  MKV_DEV void load(int t, float *kf, float *vf) const {
    int ck[8], cv[8];
    codes8(kc + (size_t)t * rowbytes, ck);
    codes8(vc + (size_t)t * rowbytes, cv);
    const float s = vs[t];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      kf[i] = cbk[ck[i]] * tau[i];
      vf[i] = cbv[cv[i]] * s;
    }
    const uint32_t a = krow[t], b = krow[t + 1];
    for (uint32_t e = a; e < b; ++e) {
      const uint32_t ent = kout[e];
      const int ch = (int)(ent & 0xFFu) - c0;
      const float x = h2f(ent >> 16);
#pragma unroll
      for (int i = 0; i < 8; ++i) kf[i] = (ch == i) ? x : kf[i];
    }
    for (int j = 0; j < nov; ++j) {
      const uint32_t ent = vout[(size_t)t * nov + j];
      if (ent == kNoOutlier) break;
      const int ch = (int)(ent & 0xFFu) - c0;
      const float x = h2f(ent >> 16);
#pragma unroll
      for (int i = 0; i < 8; ++i) vf[i] = (ch == i) ? x : vf[i];
    }
  }
};

// Run one wave over tokens [a, b) of its tile.
template <int D, int G, class L>
MKV_DEV void wave_attend(L &ld, int a, int b, const float (&qf)[G][8], float (&m_run)[G],
                         float (&l)[G], float (&o)[G][8], int grp, int sub, float *logit_out) {
  constexpr int LPT = Geo<D>::LPT, TPW = Geo<D>::TPW;
  int cur_blk = -1;
  for (int base = a; base < b; base += TPW) {
    const int blk = base >> 6;
    if (blk != cur_blk) {
      ld.block(blk);
      cur_blk = blk;
    }
    const int t = base + grp;
    const bool valid = t < b;
    float kf[8], vf[8];
    if (valid) {
      ld.load(t, kf, vf);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) kf[i] = vf[i] = 0.f;
    }
    float s[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) acc = fmaf(qf[g][i], kf[i], acc);
      acc = group_sum<LPT>(acc);
      s[g] = valid ? acc : -INFINITY;
    }
    if (logit_out != nullptr && valid && sub == 0) {
      const int sl = ld.slot(t);
#pragma unroll
      for (int g = 0; g < G; ++g) logit_out[(size_t)sl * G + g] = s[g];
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = s[g];
#pragma unroll
      for (int m = LPT; m < 64; m <<= 1) mx = fmaxf(mx, __shfl_xor(mx, m));
      if (mx > m_run[g]) {
        const float corr = exp2f(m_run[g] - mx);
        l[g] *= corr;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[g][i] *= corr;
        m_run[g] = mx;
      }
      const float p = valid ? exp2f(s[g] - m_run[g]) : 0.f;
      l[g] += p;
#pragma unroll
      for (int i = 0; i < 8; ++i) o[g][i] = fmaf(p, vf[i], o[g][i]);
    }
  }
}

template <int D, int G>
__global__ __launch_bounds__(kTileThreads) void k_attn_partial(
    const SeqDesc *__restrict__ seqs, const int32_t *__restrict__ state, const int4 *__restrict__ tiles,
    const uint16_t *__restrict__ q, float *__restrict__ partials, const float *__restrict__ cbtab,
    int Hkv, float qscale) {
  constexpr int LPT = Geo<D>::LPT, NW = kTileThreads / 64;
  __shared__ float s_cb[32];
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

  float qf[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    const uint4 u = *reinterpret_cast<const uint4 *>(q + ((size_t)seq * Hq + h * G + g) * D + c0);
    unpack8(u, qf[g]);
#pragma unroll
    for (int i = 0; i < 8; ++i) qf[g][i] *= qscale;
  }

  float m_run[G], l[G], o[G][8];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m_run[g] = -INFINITY;
    l[g] = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) o[g][i] = 0.f;
  }

  // contiguous token range per wave, a multiple of 64 tokens so blocks never straddle waves
  const int end = max(t1, t0);
  const int span = ((end - t0 + NW - 1) / NW + 63) & ~63;
  const int a = min(t0 + wave * span, end);
  const int b = min(a + span, end);

  if (method == KVQ) {
    const int nc = 1 << sd.bits;
    const float *cb = cbtab + cb_offset(sd.bits);
    if (threadIdx.x < nc) s_cb[threadIdx.x] = cb[threadIdx.x];
    if (threadIdx.x < nc) s_cb[16 + threadIdx.x] = cb[nc + threadIdx.x];
  }
  __syncthreads();

  if (method == FP16 || method == H2O) {
    LoadFP16<D> ld{reinterpret_cast<const uint16_t *>(sd.k) + h * stride_rows(sd, D),
                   reinterpret_cast<const uint16_t *>(sd.v) + h * stride_rows(sd, D), c0};
    float *lg = (method == H2O) ? reinterpret_cast<float *>(sd.logits) + h * stride_logits(sd, G) : nullptr;
    wave_attend<D, G>(ld, a, b, qf, m_run, l, o, grp, sub, lg);
  } else if (method == ROCKET) {
    LoadGather<D> ld{reinterpret_cast<const uint16_t *>(sd.k) + h * stride_rows(sd, D),
                     reinterpret_cast<const uint16_t *>(sd.v) + h * stride_rows(sd, D),
                     reinterpret_cast<const int32_t *>(sd.sel) + h * stride_sel(sd), c0};
    wave_attend<D, G>(ld, a, b, qf, m_run, l, o, grp, sub, nullptr);
  } else if (method == UQ) {
    LoadUQ<D> ld;
    ld.kc = reinterpret_cast<const uint8_t *>(sd.kc) + h * stride_codes(sd);
    ld.vc = reinterpret_cast<const uint8_t *>(sd.vc) + h * stride_codes(sd);
    ld.kmeta = reinterpret_cast<const float2 *>(sd.kmeta) + h * stride_uq_kmeta(sd, D);
    ld.vmeta = reinterpret_cast<const float2 *>(sd.vmeta) + h * stride_uq_vmeta(sd, D);
    ld.kres = reinterpret_cast<const uint16_t *>(sd.kres) + (size_t)h * 64 * D;
    ld.c0 = c0;
    ld.full = (st[ST_COUNT] / 64) * 64;
    wave_attend<D, G>(ld, a, b, qf, m_run, l, o, grp, sub, nullptr);
  } else if (method == KVQ) {
    LoadKVQ<D> ld;
    ld.kc = reinterpret_cast<const uint8_t *>(sd.kc) + h * stride_codes(sd);
    ld.vc = reinterpret_cast<const uint8_t *>(sd.vc) + h * stride_codes(sd);
    ld.krow = reinterpret_cast<const uint32_t *>(sd.krow) + h * stride_krow(sd);
    ld.kout = reinterpret_cast<const uint32_t *>(sd.kout) + h * stride_kout(sd);
    ld.vout = reinterpret_cast<const uint32_t *>(sd.vout) + h * stride_vout(sd);
    ld.vs = reinterpret_cast<const float *>(sd.vmeta) + h * stride_slots(sd);
    ld.cbk = s_cb;
    ld.cbv = s_cb + 16;
    ld.c0 = c0;
    ld.bits = sd.bits;
    ld.rowbytes = sd.rowbytes;
    ld.nov = sd.nov_slots;
    const float2 *tt = reinterpret_cast<const float2 *>(sd.kmeta) + (size_t)h * D;
#pragma unroll
    for (int i = 0; i < 8; ++i) ld.tau[i] = tt[c0 + i].x;
    wave_attend<D, G>(ld, a, b, qf, m_run, l, o, grp, sub, nullptr);
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
      for (int w = 0; w < NW; ++w) val += s_red[w][g][c] * exp2f(s_red[w][g][0] - M);
    }
    dst[e] = val;
  }
}

template <int D, int G>
__global__ __launch_bounds__(256) void k_attn_combine(const SeqDesc *__restrict__ seqs,
                                                      const int32_t *__restrict__ state,
                                                      const float *__restrict__ partials,
                                                      float *__restrict__ out, int Hkv) {
  __shared__ float sM[G], sL[G];
  const int seq = blockIdx.x / Hkv, h = blockIdx.x % Hkv;
  const SeqDesc &sd = seqs[seq];
  const int first = sd.tile_first + h * sd.tile_count, nt = sd.tile_count;
  const float *P = partials + (size_t)first * G * (D + 2);
  if (threadIdx.x < G) {
    const int g = threadIdx.x;
    float M = -INFINITY;
    for (int t = 0; t < nt; ++t) M = fmaxf(M, P[((size_t)t * G + g) * (D + 2)]);
    float L = 0.f;
    for (int t = 0; t < nt; ++t) {
      const float m = P[((size_t)t * G + g) * (D + 2)];
      if (m != -INFINITY) L += P[((size_t)t * G + g) * (D + 2) + 1] * exp2f(m - M);
    }
    sM[g] = M;
    sL[g] = L;
  }
  __syncthreads();
  const int Hq = Hkv * G;
  for (int e = threadIdx.x; e < G * D; e += 256) {
    const int g = e / D, c = e % D;
    const float M = sM[g];
    float acc = 0.f;
    for (int t = 0; t < nt; ++t) {
      const float m = P[((size_t)t * G + g) * (D + 2)];
      if (m != -INFINITY) acc += P[((size_t)t * G + g) * (D + 2) + 2 + c] * exp2f(m - M);
    }
    out[((size_t)seq * Hq + h * G + g) * D + c] = acc / sL[g];
  }
  if (sd.method == H2O) {
    const int32_t *st = state + ((size_t)seq * Hkv + h) * ST_WORDS;
    const int count = st[ST_COUNT];
    const float *lg = reinterpret_cast<const float *>(sd.logits) + h * stride_logits(sd, G);
    float *score = reinterpret_cast<float *>(sd.score) + h * stride_slots(sd);
    float invL[G];
#pragma unroll
    for (int g = 0; g < G; ++g) invL[g] = 1.f / sL[g];
    for (int j = threadIdx.x; j < count; j += 256) {
      float acc = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) acc += exp2f(lg[(size_t)j * G + g] - sM[g]) * invL[g];
      score[j] += acc;
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
