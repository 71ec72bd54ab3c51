// Internal layout shared by the host library and the HIP kernels.
#pragma once

#include <vector>

#include <math.h>
#include <stdint.h>

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include "mkv.h"

namespace mkv {

// Record `msg` as this thread's mkv_last_error() text and return `s` (host code only).
mkv_status report_error(mkv_status s, const char *msg);

enum Method : int32_t { FP16 = 0, UQ = 1, KVQ = 2, H2O = 3, ROCKET = 4 };

// Per-(sequence, kv head) device state words.
enum StateWord : int32_t {
  ST_COUNT = 0,      // tokens held in the decode region (slots 0..count-1 are valid at attention time)
  ST_NEXT_POS = 1,   // position the next appended token gets
  ST_FREE_SLOT = 2,  // H2O: slot the next token is written to
  ST_KOUT_FILL = 3,  // KVQ: entries used in the key-outlier pool
  ST_SEL_COUNT = 4,  // ROCKET: tokens selected by the last top-k
  ST_KEPT = 5,       // tokens kept after prefill (H2O / ROCKET), prompt length otherwise
  ST_WORDS = 8
};

constexpr int kTileThreads = 256;
constexpr int kMaxG = 8;
constexpr uint32_t kNoOutlier = 0xFFFFFFFFu;  // fp16 bits 0xFFFF (a NaN) never occur in an entry

// KVQ outlier entry: the fp16 value in bits 16..31, the token's slot mod 32 in bits 11..15, the
// code stored at the outlier's channel in bits 7..10, the channel (d <= 128) in bits 0..6.
__host__ __device__ inline uint32_t outlier_pack(uint32_t bits16, int slot, int code, int ch) {
  return (bits16 << 16) | ((uint32_t)(slot & 31) << 11) | ((uint32_t)code << 7) | (uint32_t)ch;
}
__host__ __device__ inline int outlier_ch(uint32_t e) { return (int)(e & 127u); }
__host__ __device__ inline int outlier_code(uint32_t e) { return (int)((e >> 7) & 15u); }
__host__ __device__ inline int outlier_tag(uint32_t e) { return (int)((e >> 11) & 31u); }

// One sequence's configuration and region base pointers (kv head 0); every
// region is [Hkv][...] with the per-head stride given by the helpers below.
struct SeqDesc {
  int32_t method, bits, n0, cap;          // cap: decode-region slots per kv head
  int32_t B, R, T, topk;                  // H2O budget/recent; ROCKET keep/topk
  int32_t window, pool, nch, bp;          // ROCKET window/pool/channels; KVQ outlier bp
  int32_t n_o, n_ov, nov_slots, rowbytes; // KVQ outlier counts; packed code row bytes
  int32_t pool_cap, nblk, w_eff, chunk;   // KVQ outlier pool; UQ blocks; window rows; tile tokens
  int32_t tile_first, tile_count, q_off, cstride;  // partial tiles (per kv head); prompt-q row offset;
                                                   // ROCKET channel-major row stride (cap rounded to 8)
  int32_t vparts, spare0, spare1, spare2;  // H2O: eviction candidates per kv head (one per combine part)
  uint64_t k, v;            // fp16 [cap][d] rows (FP16 / H2O / ROCKET)
  uint64_t kc, vc;          // packed codes [cap][rowbytes] (UQ / KVQ)
  uint64_t kmeta, vmeta;    // UQ: float2 [nblk][d], float2 [cap][d/64]; KVQ: float2 tau/inv [d], float [cap]
  uint64_t kres;            // UQ: fp16 [64][d] residual key block
  uint64_t krow, kout, vout;// KVQ: u32 [cap+1] CSR, u32 [pool_cap], u32 [nov_slots][cap]
  uint64_t vdel;            // KVQ: u32 [nov_slots][cap] value-outlier differences for the attention
  uint64_t pos, score;      // H2O / ROCKET: int32 [cap], float [cap]
  uint64_t logits;          // H2O: float [cap][G] log2-domain logits of the last attention
  uint64_t vbest;           // H2O: [vparts] eviction candidates of the last attention pass, 16 bytes
                            // each: u64 key (score bits << 32 | position; ~0 = none), int32 slot
  uint64_t stage_k, stage_v;// H2O / ROCKET: fp16 [n0][d] prompt staging
  uint64_t kcm;             // ROCKET: fp16 [d][cap] channel-major keys
  uint64_t sel, akeys;      // ROCKET: int32 [topk] selected slots; u32 [cap] score keys
  uint64_t aux0, aux1;      // prefill scratch: H2O float [n0] scores, float2 [G][n0] row stats;
                            // ROCKET float [n0] votes, float2 [G*w][nchunk] partial row stats
};

struct Shape {
  int32_t S, Hq, Hkv, D, G, max_new;
};

// Per-kv-head strides (in elements of the region's type).
__host__ __device__ inline int64_t stride_rows(const SeqDesc &s, int D) { return (int64_t)s.cap * D; }
__host__ __device__ inline int64_t stride_codes(const SeqDesc &s) { return (int64_t)s.cap * s.rowbytes; }
__host__ __device__ inline int64_t stride_uq_kmeta(const SeqDesc &s, int D) { return (int64_t)s.nblk * D; }
__host__ __device__ inline int64_t stride_uq_vmeta(const SeqDesc &s, int D) { return (int64_t)s.cap * (D / 64); }
__host__ __device__ inline int64_t stride_krow(const SeqDesc &s) { return (int64_t)s.cap + 1; }
__host__ __device__ inline int64_t stride_kout(const SeqDesc &s) { return (int64_t)s.pool_cap; }
__host__ __device__ inline int64_t stride_vout(const SeqDesc &s) { return (int64_t)s.cap * s.nov_slots; }
__host__ __device__ inline int64_t stride_slots(const SeqDesc &s) { return (int64_t)s.cap; }
__host__ __device__ inline int64_t stride_logits(const SeqDesc &s, int G) { return (int64_t)s.cap * G; }
__host__ __device__ inline int64_t stride_stage(const SeqDesc &s, int D) { return (int64_t)s.n0 * D; }
__host__ __device__ inline int64_t stride_sel(const SeqDesc &s) { return (int64_t)(s.topk > 0 ? s.topk : 1); }
__host__ __device__ inline int64_t stride_kcm(const SeqDesc &s, int D) { return (int64_t)s.cstride * D; }

// UQ value codes sit in 4-token blocks of 2*D bytes laid out for the attention's matrix
// operands: 16 segments (one per operand row r) of D/16 codes x 4 tokens, 4 bits each.  Channel
// ch belongs to row r = (ch % 64) / 4 and operand m = 4 * (ch / 64) + ch % 4; within the segment
// operand m uses nibbles 2*(m%2) + {0, 4, 1, 5} of word m/2 for tokens 0..3 of the block.
// Returns the bit offset of (ch, token j of the block) within the block.
__host__ __device__ inline int uq_vbit(int ch, int j, int D) {
  const int r = (ch & 63) >> 2, m = 4 * (ch >> 6) + (ch & 3);
  const int nib = 2 * (m & 1) + ((j & 1) ? 4 : 0) + ((j >> 1) & 1);
  return r * D + (m >> 1) * 32 + 4 * nib;  // a segment holds D bits
}

// Codebook table: for b = 2, 3, 4: cbK[2^b], cbV[2^b], midK[2^b-1], midV[2^b-1].
__host__ __device__ inline int cb_offset(int bits) {
  // sizes: b=2: 4+4+3+3 = 14; b=3: 8+8+7+7 = 30; b=4: 16+16+15+15 = 62
  return bits == 2 ? 0 : bits == 3 ? 14 : 44;
}
constexpr int kCbTableFloats = 14 + 30 + 62;

// Lookup tables of the KVQ codebooks for the attention, built on the host at cache creation and
// stored after the codebook table (kLutBase floats into the same device region): for b = 2 one
// entry per byte of four codes, the four codebook values as packed fp16 (2 words, 256 entries);
// for b = 3 and 4 one entry per field of two codes, the two values as packed fp16 (2^(2b)
// entries).  Per b, the key table then the value table; lut_offset and lut_half_words in words.
constexpr int kLutBase = 112;
__host__ __device__ inline int lut_half_words(int bits) { return bits == 2 ? 512 : 1 << (2 * bits); }
__host__ __device__ inline int lut_offset(int bits) { return bits == 2 ? 0 : bits == 3 ? 1024 : 1152; }
constexpr int kLutWords = 1024 + 128 + 512;
constexpr int kCbRegionFloats = kLutBase + kLutWords;

// A KVQ value outlier as the attention reads it: d = x - s cb[code] (x the fp16 outlier, s the
// token's scale, cb[code] the codebook value its stored code stands for), float32 with the 7
// lowest mantissa bits replaced by the channel; 0 marks an empty slot.
__host__ __device__ inline uint32_t vdel_pack(float d, int ch) {
  return (__builtin_bit_cast(uint32_t, d) & ~127u) | (uint32_t)ch;
}

// Host: x rounded once, to nearest even, to the nearest fp16 value (finite |x| < 65520).
inline float round_to_half(double x) {
  if (x == 0.0 || !isfinite(x)) return (float)x;
  int e;
  frexp(x, &e);                                // |x| = m 2^e, m in [0.5, 1)
  const int qexp = (e - 1 >= -14 ? e - 1 : -14) - 10;  // quantum: 2^-10 of the leading bit, or 2^-24
  return (float)(nearbyint(ldexp(x, -qexp)) * ldexp(1.0, qexp));
}

// Tokens one RocketKV scoring workgroup of a decode step covers.
constexpr int kScoreTokensPerPart = 1024;
// H2O slots one combine workgroup scores (an H2O kv head has ceil(cap / kCombineSlots) parts).
constexpr int kCombineSlots = 2048;

// Kernel launchers (defined in the .hip files).  All enqueue on `st`.
struct Dev {
  const SeqDesc *seqs;   // device [S]
  int32_t *state;        // device [S][Hkv][ST_WORDS]
  const int4 *tiles;     // device [n_tiles]: seq, kv head, token begin, token end
  float *partials;       // device [n_tiles][G][D+2]
  const float *cbtab;    // device [kCbTableFloats]
  int n_tiles;
  int n_tiles_uq;        // tiles of uniform 4-bit sequences (reported, not used by the launches)
  int n_tiles_rk;        // the last n_tiles_rk tiles belong to RocketKV sequences
  const int4 *prep;      // device [n_prep]: a decode step's append / scoring work (seq, kv head,
                         // part or -1 for a plain append, parts)
  const int2 *rk_pairs;  // device [n_rk_pairs]: the RocketKV (seq, kv head) pairs
  const int4 *comb;      // device [n_comb]: combine work (seq, kv head, part, parts)
  int n_prep, n_rk_pairs, n_comb;
};

// Optional timing events of one launch: when set, they record the kernel's own start and end
// (hipExtLaunchKernelGGL), with no marker packets of their own around the launch.
struct LaunchEv {
  hipEvent_t start = nullptr, stop = nullptr;
};

// H2O pairs whose last attention pass chose a victim write the token into its slot.
hipError_t launch_append_decode(const Dev &dv, const Shape &sh, const uint16_t *k, const uint16_t *v,
                                hipStream_t st, LaunchEv ev = {});
hipError_t launch_prefill_seq(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq,
                              const uint16_t *k, const uint16_t *v, hipStream_t st);
hipError_t launch_attention_partial(const Dev &dv, const Shape &sh, const uint16_t *q, hipStream_t st,
                                    LaunchEv ev = {});
// The static split-K workspace of the current device (kStaticScratchBytes), its address looked up
// on the first call per device.
constexpr size_t kStaticScratchBytes = size_t(8) << 20;
hipError_t static_scratch(float **ptr, size_t *bytes);
// The attention tiles of a cache layout in launch order, and the sequences' descriptors (tile
// bookkeeping: tile_first, tile_count, chunk); host only, for checks of the layout rules.
mkv_status layout_tiles(const mkv_shape *shape, const mkv_config *cfg, const int32_t *prompt_len,
                        std::vector<int4> *tiles, std::vector<SeqDesc> *seqs);
hipError_t launch_attention_combine(const Dev &dv, const Shape &sh, float *out, hipStream_t st,
                                    LaunchEv ev = {});
hipError_t launch_topk(const Dev &dv, const Shape &sh, const uint16_t *q, int32_t *pos_out, int topk_max,
                       hipStream_t st, LaunchEv ev = {});
// The decode append of every sequence and the RocketKV top-k in two launches (the appends and the
// scores, spread over several workgroups per kv head; then the selection), with the effect of
// launch_append_decode followed by launch_topk without positions.
hipError_t launch_append_select(const Dev &dv, const Shape &sh, const uint16_t *k, const uint16_t *v,
                                const uint16_t *q, hipStream_t st, LaunchEv ev_score = {}, LaunchEv ev_select = {});
hipError_t launch_h2o_prefill_seq(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq,
                                  const uint16_t *q_rows, hipStream_t st);
hipError_t launch_snap_prefill_seq(const Dev &dv, const Shape &sh, const SeqDesc &hs, int seq,
                                   const uint16_t *q_window, hipStream_t st);
hipError_t launch_init_state(const Dev &dv, const Shape &sh, hipStream_t st);
// Streaming read of `bytes` (a multiple of `chunk`, itself a multiple of 16 KiB); sink: device
// uint32 [256], written only in the (practically never taken) branch that keeps the loads alive.
hipError_t launch_probe_read(const void *buf, size_t bytes, size_t chunk, uint32_t *sink, hipStream_t st);

}  // namespace mkv
