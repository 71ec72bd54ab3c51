// Host side of libmkv: argument validation, arena layout, call-order state machine, kernel
// launches, state export and kernel timing.  See include/mkv.h for the contract.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstddef>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "mkv.h"
#include "mkv_internal.h"

using namespace mkv;

namespace {

thread_local std::string g_err;

mkv_status fail(mkv_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

}  // namespace

namespace mkv {
mkv_status report_error(mkv_status s, const char *msg) { return fail(s, "%s", msg); }
}  // namespace mkv

namespace {

mkv_status hip_fail(hipError_t e, const char *what) {
  return fail(MKV_EHIP, "%s: %s", what, hipGetErrorString(e));
}

enum Phase { PH_CREATED, PH_PROMPT, PH_READY, PH_APPENDED, PH_SELECTED, PH_ATTENDED };

constexpr int kProfKinds = 5;

struct Layout {
  std::vector<SeqDesc> seqs;  // offsets (relative to the arena) in the pointer fields
  size_t off_seqs = 0, off_state = 0, off_tiles = 0, off_cbtab = 0, off_partials = 0, total = 0;
  size_t off_prep = 0, off_rk_pairs = 0, off_comb = 0;
  int n_tiles = 0, n_tiles_uq = 0, n_tiles_rk = 0;
  std::vector<int4> tiles;
  std::vector<int4> prep;      // decode-step append / scoring work list
  std::vector<int2> rk_pairs;  // RocketKV (seq, kv head) pairs
  std::vector<int4> comb;      // combine work list
};

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Every region pointer of a descriptor (arena offsets in the layout, device addresses once the
// arena is known); the descriptor is its integer fields followed by exactly these.
constexpr uint64_t SeqDesc::*kRegionFields[] = {
    &SeqDesc::k,      &SeqDesc::v,      &SeqDesc::kc,      &SeqDesc::vc,      &SeqDesc::kmeta, &SeqDesc::vmeta,
    &SeqDesc::kres,   &SeqDesc::krow,   &SeqDesc::kout,    &SeqDesc::vout,    &SeqDesc::vdel,  &SeqDesc::pos,
    &SeqDesc::score,  &SeqDesc::logits, &SeqDesc::vbest,   &SeqDesc::stage_k, &SeqDesc::stage_v,
    &SeqDesc::kcm,    &SeqDesc::sel,    &SeqDesc::akeys,   &SeqDesc::aux0,    &SeqDesc::aux1};
static_assert(offsetof(SeqDesc, k) + sizeof(kRegionFields) / sizeof(kRegionFields[0]) * sizeof(uint64_t) ==
                  sizeof(SeqDesc),
              "every region pointer of SeqDesc is relocated");

constexpr int kMaxTiles = 32;  // per (sequence, kv head); the combine kernel holds up to 64

// Bytes each token costs the attention pass.
double token_bytes(const SeqDesc &s, int D) {
  switch (s.method) {
    case UQ: return D + D / 64.0 * 8 + 8;
    case KVQ: return D * s.bits / 4.0 + 4 + 8 + 4;
    default: return 4.0 * D;
  }
}

// Tokens per attention tile for a tile of about `tile_bytes` (a multiple of 64: tiles of 32-token
// granularity, which filled the slots of small launches more finely, were measured slower on the
// FP16, uniform 4-bit, H2O and RocketKV per-configuration launches).
int tile_tokens(const SeqDesc &s, int D, double tile_bytes) {
  const int t = (int)(tile_bytes / token_bytes(s, D)) & ~63;
  return std::max(64, std::min(t, 4096));
}

// Tile size: large tiles amortise each workgroup's set-up, but a launch needs several
// workgroups per slot (256 CUs x 3 resident workgroups) to balance: about 4 rounds, within
// 64 to 192 KiB (measured best for batches of ~40 MB and ~600 MB per step); then adjusted to
// whole rounds (below).
constexpr int kTileSlots = 256 * 3;  // resident attention workgroups (3 per CU)
double tile_bytes_for(double total_bytes) {
  constexpr double kRounds = 4;
  return std::min(196608.0, std::max(65536.0, total_bytes / (kTileSlots * kRounds)));
}

mkv_status check_shape(const mkv_shape *sh) {
  if (!sh) return fail(MKV_EINVAL, "shape is NULL");
  if (sh->n_seqs < 1 || sh->n_kv_heads < 1 || sh->n_q_heads < 1 || sh->max_new_tokens < 0)
    return fail(MKV_EINVAL, "shape fields must be positive (max_new_tokens >= 0)");
  if (sh->n_q_heads % sh->n_kv_heads != 0) return fail(MKV_EINVAL, "n_q_heads %% n_kv_heads != 0");
  const int G = sh->n_q_heads / sh->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return fail(MKV_EUNSUPPORTED, "query heads per kv head must be 1, 2, 4 or 8 (got %d)", G);
  if (sh->head_dim != 64 && sh->head_dim != 128)
    return fail(MKV_EUNSUPPORTED, "head_dim must be 64 or 128 (got %d)", sh->head_dim);
  return MKV_OK;
}

// RocketKV's SnapKV budget: keep_tokens, or in ratio mode max(floor(n0 / keep_ratio), window).
int rocket_keep(const mkv_config &c, int n0) {
  return c.keep_ratio > 0 ? std::max(n0 / c.keep_ratio, c.window) : c.keep_tokens;
}

mkv_status check_config(const mkv_config &c, int n0, int D, int s) {
  if (n0 < 1) return fail(MKV_EINVAL, "seq %d: prompt_len must be >= 1", s);
  switch (c.method) {
    case MKV_FP16: return MKV_OK;
    case MKV_UQ:
      if (c.bits != 4) return fail(MKV_EUNSUPPORTED, "seq %d: uniform quantization supports bits=4", s);
      if (c.group != 64) return fail(MKV_EUNSUPPORTED, "seq %d: uniform quantization supports group=64", s);
      return MKV_OK;
    case MKV_KVQ:
      if (c.bits < 2 || c.bits > 4) return fail(MKV_EINVAL, "seq %d: KVQ bits must be 2, 3 or 4", s);
      if (c.outlier_bp < 0 || c.outlier_bp > 5000) return fail(MKV_EINVAL, "seq %d: outlier_bp in 0..5000", s);
      if (n0 > 65535) return fail(MKV_EUNSUPPORTED, "seq %d: KVQ prompt longer than 65535", s);
      return MKV_OK;
    case MKV_H2O: {
      if (c.budget_pct < 1 || c.budget_pct > 10000) return fail(MKV_EINVAL, "seq %d: budget_pct in 1..10000", s);
      const long long B = (long long)c.budget_pct * n0 / 100;
      if (B < 1) return fail(MKV_EINVAL, "seq %d: H2O budget is 0 tokens for prompt_len %d", s, n0);
      return MKV_OK;
    }
    case MKV_ROCKET:
      if (c.window < 1) return fail(MKV_EINVAL, "seq %d: window must be >= 1", s);
      if (c.keep_ratio < 0) return fail(MKV_EINVAL, "seq %d: keep_ratio must be >= 0", s);
      if (c.keep_ratio == 0 && c.keep_tokens < c.window) return fail(MKV_EINVAL, "seq %d: keep_tokens must be >= window", s);
      if (c.pool < 1 || (c.pool & 1) == 0) return fail(MKV_EINVAL, "seq %d: pool must be odd and >= 1", s);
      if (c.n_channels < 1 || c.n_channels > D) return fail(MKV_EINVAL, "seq %d: n_channels in 1..head_dim", s);
      if (c.topk < 0) return fail(MKV_EINVAL, "seq %d: topk must be >= 0", s);
      if (c.topk == 0 && rocket_keep(c, n0) / 2 < 1) return fail(MKV_EINVAL, "seq %d: the keep budget / 2 is 0", s);
      return MKV_OK;
    default:
      return fail(MKV_EINVAL, "seq %d: unknown method %d", s, c.method);
  }
}

mkv_status make_layout(const mkv_shape *shp, const mkv_config *cfg, const int32_t *plen, Layout *L) {
  mkv_status st = check_shape(shp);
  if (st != MKV_OK) return st;
  if (!cfg || !plen) return fail(MKV_EINVAL, "cfg and prompt_len must be non-NULL");
  const int S = shp->n_seqs, Hkv = shp->n_kv_heads, D = shp->head_dim, G = shp->n_q_heads / Hkv;
  const int mn = shp->max_new_tokens;
  for (int s = 0; s < S; ++s)
    if ((st = check_config(cfg[s], plen[s], D, s)) != MKV_OK) return st;

  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + std::max<size_t>(bytes, 1));
    return (uint64_t)o;
  };
  L->off_seqs = take(sizeof(SeqDesc) * S);
  L->off_state = take(sizeof(int32_t) * S * Hkv * ST_WORDS);
  L->off_cbtab = take(sizeof(float) * kCbRegionFloats);
  L->seqs.assign(S, SeqDesc{});
  int q_h2o = 0, q_rk = 0;
  for (int s = 0; s < S; ++s) {
    SeqDesc &d = L->seqs[s];
    const mkv_config &c = cfg[s];
    const int n0 = plen[s];
    d.method = c.method;
    d.n0 = n0;
    d.bits = c.bits;
    d.bp = c.outlier_bp;
    const size_t H = Hkv;
    switch (c.method) {
      case FP16:
        d.cap = n0 + mn;
        d.k = take(H * d.cap * D * 2);
        d.v = take(H * d.cap * D * 2);
        break;
      case UQ:
        d.cap = (n0 + mn + 3) & ~3;  // value codes are stored in 4-token blocks
        d.rowbytes = D / 2;
        d.nblk = d.cap / 64;
        d.kc = take(H * d.cap * d.rowbytes);
        d.vc = take(H * d.cap * d.rowbytes);
        d.kmeta = take(H * std::max(d.nblk, 1) * D * 8);
        d.vmeta = take(H * d.cap * (D / 64) * 8);
        d.kres = take(H * 64 * D * 2);
        break;
      case KVQ: {
        d.cap = (n0 + mn + 3) & ~3;  // value codes are stored in 4-token blocks
        d.rowbytes = D * c.bits / 8;
        d.n_o = (int)(((long long)n0 * c.outlier_bp + 5000) / 10000);
        d.n_ov = (int)(((long long)D * c.outlier_bp + 5000) / 10000);
        d.nov_slots = c.outlier_bp > 0 ? std::max(1, d.n_ov) : 1;
        d.pool_cap = c.outlier_bp > 0 ? (std::min(d.n_o, n0) + mn) * D : 1;
        d.kc = take(H * d.cap * d.rowbytes);
        d.vc = take(H * d.cap * d.rowbytes);
        d.kmeta = take(H * D * 8);
        d.vmeta = take(H * d.cap * 4);
        d.krow = take(H * (d.cap + 1) * 4);
        d.kout = take(H * d.pool_cap * 4);
        d.vout = take(H * d.cap * d.nov_slots * 4);
        d.vdel = take(H * d.cap * d.nov_slots * 4);
        break;
      }
      case H2O: {
        d.B = (int)((long long)c.budget_pct * n0 / 100);
        d.R = d.B / 2;
        d.cap = (int)std::min<long long>((long long)d.B + 1, (long long)n0 + mn);
        d.k = take(H * d.cap * D * 2);
        d.v = take(H * d.cap * D * 2);
        d.pos = take(H * d.cap * 4);
        d.score = take(H * d.cap * 4);
        d.logits = take(H * d.cap * G * 4);
        d.vparts = (d.cap + kCombineSlots - 1) / kCombineSlots;
        d.vbest = take(H * d.vparts * 16);
        d.stage_k = take(H * n0 * D * 2);
        d.stage_v = take(H * n0 * D * 2);
        d.aux0 = take(H * n0 * 4);
        d.aux1 = take(H * G * n0 * 8);
        d.q_off = q_h2o;
        q_h2o += n0;
        break;
      }
      case ROCKET: {
        d.T = rocket_keep(c, n0);
        d.window = c.window;
        d.w_eff = std::min(c.window, n0);
        d.pool = c.pool;
        d.nch = c.n_channels;
        d.topk = c.topk > 0 ? c.topk : d.T / 2;
        const int kept = std::min(d.T, n0);
        d.cap = kept + mn;
        const int nchunk = (n0 + 255) / 256;
        d.k = take(H * d.cap * D * 2);
        d.v = take(H * d.cap * D * 2);
        d.cstride = (d.cap + 7) & ~7;
        d.kcm = take(H * d.cstride * D * 2);
        d.pos = take(H * d.cap * 4);
        d.sel = take(H * d.topk * 4);
        d.akeys = take(H * d.cap * 4);
        d.stage_k = take(H * n0 * D * 2);
        d.stage_v = take(H * n0 * D * 2);
        d.aux0 = take(H * n0 * 4);
        d.aux1 = take(std::max({H * d.w_eff * G * nchunk * 4 * 8, H * D * 4, H * n0 * 4}));
        d.q_off = q_rk;
        q_rk += c.window;
        break;
      }
    }
  }
  // attention tiles: per sequence and kv head, ranges of `chunk` tokens over its largest active set;
  // one launch covers them all, RocketKV sequences last (their gathered tiles are the shortest)
  L->tiles.clear();
  L->n_tiles_uq = 0;
  L->n_tiles_rk = 0;
  double total = 0.0;
  for (int s = 0; s < S; ++s) {
    const SeqDesc &d = L->seqs[s];
    total += (double)Hkv * (d.method == ROCKET ? d.topk : d.cap) * token_bytes(d, D);
  }
  // a sequence's tokens per tile and tile count at a given tile size
  // In launches of three or more rounds of workgroups, fp16-row tiles (FP16, H2O) take twice the
  // bytes: they are bandwidth-bound, and each tile a CU starts costs a dispatch gap (a median
  // 2 us from one tile's end to the next one's start on that CU, measured with clock stamps), so
  // fewer, longer row tiles leave the slots busier (mixed batch: 134.0-135.1 against 135.8-136.3
  // us per partial launch; 1.5x and 2.5-3x no better, 0.75x 6 us slower).  Shorter launches keep
  // them (H2O-40 alone: 32.7 against 30.3 us with doubled row tiles, half a round left over).
  bool long_rows = false;
  auto split = [&](const SeqDesc &d, double tb, int *chunk) {
    const int amax = d.method == ROCKET ? d.topk : d.cap;
    if (long_rows && (d.method == FP16 || d.method == H2O)) tb *= 2;
    int c = tile_tokens(d, D, tb), n = std::max(1, (amax + c - 1) / c);
    if (n > kMaxTiles) {  // long sequences: fewer, larger tiles keep the combine short
      c = (((amax + kMaxTiles - 1) / kMaxTiles) + 63) & ~63;
      n = (amax + c - 1) / c;
    }
    *chunk = c;
    return n;
  };
  auto count_at = [&](double tb) {
    long long n = 0;
    int c;
    for (int s = 0; s < S; ++s) n += (long long)Hkv * split(L->seqs[s], tb, &c);
    return n;
  };
  // whole rounds of resident workgroups: when the size rule leaves the last round partly idle,
  // smaller tiles (down to 16 KiB) fill it, the smallest size whose count still fits in the
  // rounds begun.  (Fewer, larger tiles to drop a nearly empty last round were measured worse:
  // H2O-40 alone 32.3 against 29.5 us.)
  double tile_bytes = tile_bytes_for(total);
  long_rows = count_at(tile_bytes) >= 3 * kTileSlots;
  {
    const long long cap = (count_at(tile_bytes) + kTileSlots - 1) / kTileSlots * kTileSlots;
    for (double tb = 16384.0; tb < tile_bytes; tb *= 1.02)
      if (count_at(tb) <= cap) {
        tile_bytes = tb;
        break;
      }
  }
  for (int pass = 0; pass < 2; ++pass)
  for (int s = 0; s < S; ++s) {
    SeqDesc &d = L->seqs[s];
    const int grp = d.method == ROCKET ? 1 : 0;
    if (grp != pass) continue;
    const int amax = d.method == ROCKET ? d.topk : d.cap;
    d.tile_count = split(d, tile_bytes, &d.chunk);
    d.tile_first = (int)L->tiles.size();
    for (int h = 0; h < Hkv; ++h)
      for (int t = 0; t < d.tile_count; ++t)
        L->tiles.push_back(make_int4(s, h, t * d.chunk, std::min(amax, (t + 1) * d.chunk)));
    if (d.method == UQ) L->n_tiles_uq += Hkv * d.tile_count;
    if (pass == 1) L->n_tiles_rk += Hkv * d.tile_count;
  }
  L->n_tiles = (int)L->tiles.size();
  // Launch order (a tile's partial slot stays tile_first + h tile_count + z / chunk, whatever its
  // place): the quantized tiles, the longest-running per byte, spread evenly over the first 3/4 of
  // the fp16-row and quantized tiles, the fp16-row tiles evenly over all of them, RocketKV tiles
  // last.  Long tiles then start early enough to end with the rest, while issue-bound and
  // bandwidth-bound tiles still share the chip throughout (measured on the mixed batch: 136-137
  // against 140-141 us per partial launch for the sequence order; spreading the quantized tiles
  // over 60 %, 90 % or all of the list, or putting them all first, did less or worse).
  {
    constexpr double kQuantSpan = 0.75;
    auto quant = [&](const int4 &t) { const int m = L->seqs[t.x].method; return m == KVQ || m == UQ; };
    double nq = 0, nr = 0;
    for (const int4 &t : L->tiles)
      if (L->seqs[t.x].method != ROCKET) (quant(t) ? nq : nr) += 1;
    std::vector<std::pair<double, int>> key;
    key.reserve(L->tiles.size());
    double iq = 0, ir = 0;
    for (int i = 0; i < (int)L->tiles.size(); ++i) {
      const int4 &t = L->tiles[i];
      const double v = L->seqs[t.x].method == ROCKET ? 2.0 : quant(t) ? (iq++ + 0.5) / nq * kQuantSpan : (ir++ + 0.5) / nr;
      key.push_back({v, i});
    }
    std::stable_sort(key.begin(), key.end(), [](const std::pair<double, int> &a, const std::pair<double, int> &b) {
      return a.first < b.first;
    });
    std::vector<int4> ordered;
    ordered.reserve(L->tiles.size());
    for (const auto &kv : key) ordered.push_back(L->tiles[kv.second]);
    L->tiles.swap(ordered);
  }
  L->off_tiles = take(sizeof(int4) * L->n_tiles);
  // a decode step's append and scoring work: RocketKV scoring parts (one per kScoreTokens tokens
  // of the largest retained set) first, then the plain appends
  L->prep.clear();
  L->rk_pairs.clear();
  for (int s = 0; s < S; ++s) {
    const SeqDesc &d = L->seqs[s];
    if (d.method != ROCKET) continue;
    const int parts = (d.cap + kScoreTokensPerPart - 1) / kScoreTokensPerPart;
    for (int h = 0; h < Hkv; ++h) {
      L->rk_pairs.push_back(make_int2(s, h));
      for (int p = 0; p < parts; ++p) L->prep.push_back(make_int4(s, h, p, parts));
    }
  }
  for (int s = 0; s < S; ++s)
    if (L->seqs[s].method != ROCKET)
      for (int h = 0; h < Hkv; ++h) L->prep.push_back(make_int4(s, h, -1, 0));
  L->off_prep = take(sizeof(int4) * L->prep.size());
  // the combine: H2O kv heads' parts (one per kCombineSlots slots) first, then one item per pair
  L->comb.clear();
  for (int pass = 0; pass < 2; ++pass)
    for (int s = 0; s < S; ++s) {
      const SeqDesc &d = L->seqs[s];
      if ((d.method == H2O) != (pass == 0)) continue;
      const int parts = d.method == H2O ? d.vparts : 1;
      for (int h = 0; h < Hkv; ++h)
        for (int p = 0; p < parts; ++p) L->comb.push_back(make_int4(s, h, p, parts));
    }
  L->off_comb = take(sizeof(int4) * L->comb.size());
  L->off_rk_pairs = take(sizeof(int2) * std::max<size_t>(1, L->rk_pairs.size()));
  L->off_partials = take(sizeof(float) * (size_t)L->n_tiles * G * (D + 2));
  L->total = off;
  return MKV_OK;
}

}  // namespace

struct mkv_cache {
  Shape sh{};
  std::vector<mkv_config> cfg;
  std::vector<SeqDesc> hs;  // absolute device pointers
  Layout L;
  char *arena = nullptr;
  Dev dv{};
  Phase phase = PH_CREATED;
  int steps = 0;
  bool any_h2o = false, any_rocket = false, h2o_done = false, snap_done = false;
  int topk_max = 0;
  int h2o_rows = 0, rocket_rows = 0;
  // profiling
  bool evict_pending = false;  // H2O: the last eviction call's victims await the next decode append
  int prof_mask = 0;  // bit k: launches of kind k are timed
  int prof_cap = 0;
  std::vector<hipEvent_t> ev[kProfKinds][2];
  int prof_n[kProfKinds] = {};
};

namespace {

// The timing events of the next launch of `kind` (none when that kind is not timed or its events
// are used up); the launch itself records its kernel's start and end in them.
LaunchEv prof_ev(mkv_cache *c, int kind) {
  if (!(c->prof_mask >> kind & 1)) return {};
  const int i = c->prof_n[kind];
  if (i >= c->prof_cap) return {};
  c->prof_n[kind] = i + 1;
  return LaunchEv{c->ev[kind][0][i], c->ev[kind][1][i]};
}

mkv_status check_hip(hipError_t e, const char *what) {
  return e == hipSuccess ? MKV_OK : hip_fail(e, what);
}

}  // namespace

namespace mkv {
mkv_status layout_tiles(const mkv_shape *shape, const mkv_config *cfg, const int32_t *prompt_len,
                        std::vector<int4> *tiles, std::vector<SeqDesc> *seqs) {
  Layout L;
  const mkv_status st = make_layout(shape, cfg, prompt_len, &L);
  if (st != MKV_OK) return st;
  *tiles = L.tiles;
  *seqs = L.seqs;
  return MKV_OK;
}
}  // namespace mkv

extern "C" {

const char *mkv_status_str(mkv_status s) {
  switch (s) {
    case MKV_OK: return "ok";
    case MKV_EINVAL: return "invalid argument";
    case MKV_ENOMEM: return "arena too small";
    case MKV_ECAPACITY: return "cache capacity exceeded";
    case MKV_ESTATE: return "call out of order";
    case MKV_EUNSUPPORTED: return "unsupported configuration";
    case MKV_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char *mkv_last_error(void) { return g_err.c_str(); }

mkv_status mkv_cache_bytes(const mkv_shape *shape, const mkv_config *cfg, const int32_t *prompt_len,
                           size_t *arena_bytes) {
  if (!arena_bytes) return fail(MKV_EINVAL, "arena_bytes is NULL");
  Layout L;
  mkv_status st = make_layout(shape, cfg, prompt_len, &L);
  if (st != MKV_OK) return st;
  *arena_bytes = L.total;
  return MKV_OK;
}

mkv_status mkv_cache_create(const mkv_shape *shape, const mkv_config *cfg, const int32_t *prompt_len,
                            const float *codebooks, void *arena, size_t arena_bytes, void *stream,
                            mkv_cache **out) {
  if (!out) return fail(MKV_EINVAL, "out is NULL");
  *out = nullptr;
  Layout L;
  mkv_status st = make_layout(shape, cfg, prompt_len, &L);
  if (st != MKV_OK) return st;
  if (!arena) return fail(MKV_EINVAL, "arena is NULL");
  if (((uintptr_t)arena & 255) != 0) return fail(MKV_EINVAL, "arena must be 256-byte aligned");
  if (arena_bytes < L.total)
    return fail(MKV_ENOMEM, "arena has %zu bytes, the cache needs %zu", arena_bytes, L.total);
  bool any_kvq = false;
  for (int s = 0; s < shape->n_seqs; ++s) any_kvq |= cfg[s].method == MKV_KVQ;
  float table[kCbRegionFloats] = {};
  if (any_kvq) {
    if (!codebooks) return fail(MKV_EINVAL, "codebooks are required for KVQ sequences");
    const float *src = codebooks;
    for (int b = 2; b <= 4; ++b) {
      const int nc = 1 << b;
      float *dst = table + cb_offset(b);
      for (int half = 0; half < 2; ++half) {
        for (int i = 0; i < nc; ++i) {
          const float x = src[half * nc + i];
          if (!std::isfinite(x)) return fail(MKV_EINVAL, "codebook entry is not finite");
          if (round_to_half(x) != x) return fail(MKV_EINVAL, "codebook entry %g is not an fp16 value", (double)x);
          if (i > 0 && !(x >= src[half * nc + i - 1])) return fail(MKV_EINVAL, "codebooks must be ascending");
          dst[half * nc + i] = x;
        }
        for (int i = 0; i + 1 < nc; ++i) {
          volatile float sum = src[half * nc + i] + src[half * nc + i + 1];
          dst[2 * nc + half * (nc - 1) + i] = sum * 0.5f;
        }
      }
      src += 2 * nc;
    }
    // the attention's lookup tables: packed fp16 codebook values per quad (b = 2) or pair of codes
    uint32_t *lut = reinterpret_cast<uint32_t *>(table + kLutBase);
    auto hb = [](float x) { return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)x); };
    for (int b = 2; b <= 4; ++b) {
      const int nc = 1 << b, half = lut_half_words(b);
      for (int which = 0; which < 2; ++which) {
        const float *cb = table + cb_offset(b) + which * nc;
        uint32_t *dst = lut + lut_offset(b) + which * half;
        if (b == 2) {
          for (int q = 0; q < 256; ++q) {
            dst[2 * q] = hb(cb[q & 3]) | hb(cb[(q >> 2) & 3]) << 16;
            dst[2 * q + 1] = hb(cb[(q >> 4) & 3]) | hb(cb[(q >> 6) & 3]) << 16;
          }
        } else {
          for (int f = 0; f < half; ++f) dst[f] = hb(cb[f & (nc - 1)]) | hb(cb[f >> b]) << 16;
        }
      }
    }
  }
  mkv_cache *c = new mkv_cache();
  c->sh = Shape{shape->n_seqs, shape->n_q_heads, shape->n_kv_heads, shape->head_dim,
                shape->n_q_heads / shape->n_kv_heads, shape->max_new_tokens};
  c->cfg.assign(cfg, cfg + shape->n_seqs);
  c->arena = static_cast<char *>(arena);
  c->L = L;
  const uint64_t base = (uint64_t)(uintptr_t)arena;
  c->hs = L.seqs;
  for (auto &d : c->hs) {
    // offset 0 holds the descriptor table, so a zero offset marks a region the method lacks
    for (uint64_t SeqDesc::*f : kRegionFields)
      if (d.*f) d.*f += base;
    if (d.method == H2O) {
      c->any_h2o = true;
      c->h2o_rows += d.n0;
    }
    if (d.method == ROCKET) {
      c->any_rocket = true;
      c->rocket_rows += d.window;
      c->topk_max = std::max(c->topk_max, d.topk);
    }
  }
  c->dv.seqs = reinterpret_cast<const SeqDesc *>(c->arena + L.off_seqs);
  c->dv.state = reinterpret_cast<int32_t *>(c->arena + L.off_state);
  c->dv.tiles = reinterpret_cast<const int4 *>(c->arena + L.off_tiles);
  c->dv.partials = reinterpret_cast<float *>(c->arena + L.off_partials);
  c->dv.cbtab = reinterpret_cast<const float *>(c->arena + L.off_cbtab);
  c->dv.n_tiles = L.n_tiles;
  c->dv.prep = reinterpret_cast<const int4 *>(c->arena + L.off_prep);
  c->dv.rk_pairs = reinterpret_cast<const int2 *>(c->arena + L.off_rk_pairs);
  c->dv.n_prep = (int)L.prep.size();
  c->dv.comb = reinterpret_cast<const int4 *>(c->arena + L.off_comb);
  c->dv.n_comb = (int)L.comb.size();
  c->dv.n_rk_pairs = (int)L.rk_pairs.size();
  c->dv.n_tiles_uq = L.n_tiles_uq;
  c->dv.n_tiles_rk = L.n_tiles_rk;
  hipStream_t hst = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(c->arena + L.off_seqs, c->hs.data(), sizeof(SeqDesc) * c->hs.size(),
                                hipMemcpyHostToDevice, hst);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->arena + L.off_tiles, L.tiles.data(), sizeof(int4) * L.tiles.size(),
                       hipMemcpyHostToDevice, hst);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->arena + L.off_prep, L.prep.data(), sizeof(int4) * L.prep.size(), hipMemcpyHostToDevice, hst);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->arena + L.off_comb, L.comb.data(), sizeof(int4) * L.comb.size(), hipMemcpyHostToDevice, hst);
  if (e == hipSuccess && !L.rk_pairs.empty())
    e = hipMemcpyAsync(c->arena + L.off_rk_pairs, L.rk_pairs.data(), sizeof(int2) * L.rk_pairs.size(),
                       hipMemcpyHostToDevice, hst);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->arena + L.off_cbtab, table, sizeof table, hipMemcpyHostToDevice, hst);
  if (e == hipSuccess) e = launch_init_state(c->dv, c->sh, hst);
  if (e == hipSuccess) e = hipStreamSynchronize(hst);
  if (e != hipSuccess) {
    mkv_cache_destroy(c);
    return hip_fail(e, "mkv_cache_create");
  }
  *out = c;
  return MKV_OK;
}

mkv_status mkv_cache_destroy(mkv_cache *c) {
  if (!c) return MKV_OK;
  for (int k = 0; k < kProfKinds; ++k)
    for (int w = 0; w < 2; ++w)
      for (hipEvent_t e : c->ev[k][w]) (void)hipEventDestroy(e);
  delete c;
  return MKV_OK;
}

namespace {

// The decode append of one row per sequence (the row counts are already known to be 1).
mkv_status decode_append(mkv_cache *c, const uint16_t *k, const uint16_t *v, hipStream_t hst) {
  if (!(c->phase == PH_READY || (c->phase == PH_ATTENDED && !c->any_h2o)))
    return fail(MKV_ESTATE, "decode append must follow prefill or a completed decode step");
  if (c->steps >= c->sh.max_new)
    return fail(MKV_ECAPACITY, "cache holds %d decode steps (max_new_tokens)", c->sh.max_new);
  hipError_t e = launch_append_decode(c->dv, c->sh, k, v, hst, prof_ev(c, 2));
  if (e != hipSuccess) return hip_fail(e, "decode append");
  c->evict_pending = false;
  c->steps++;
  c->phase = PH_APPENDED;
  return MKV_OK;
}

// A decode step's append and top-k selection: the appends with the RocketKV scores, then the
// selection (the caller has made every check of decode_append and mkv_topk_select).
mkv_status decode_append_select(mkv_cache *c, const uint16_t *k, const uint16_t *v, const uint16_t *q,
                                hipStream_t hst) {
  hipError_t e = launch_append_select(c->dv, c->sh, k, v, q, hst, prof_ev(c, 4), prof_ev(c, 3));
  if (e != hipSuccess) return hip_fail(e, "decode append and top-k select");
  c->evict_pending = false;
  c->steps++;
  c->phase = PH_SELECTED;
  return MKV_OK;
}

}  // namespace

mkv_status mkv_append_quantize(mkv_cache *c, const uint16_t *k, const uint16_t *v, const int32_t *cu_new,
                               void *stream) {
  if (!c) return fail(MKV_EINVAL, "cache is NULL");
  if (!k || !v || !cu_new) return fail(MKV_EINVAL, "k, v and cu_new must be non-NULL");
  const int S = c->sh.S;
  hipStream_t hst = static_cast<hipStream_t>(stream);
  if (cu_new[0] != 0) return fail(MKV_EINVAL, "cu_new[0] must be 0");
  if (c->phase == PH_CREATED) {
    for (int s = 0; s < S; ++s)
      if (cu_new[s + 1] - cu_new[s] != c->hs[s].n0)
        return fail(MKV_EINVAL, "prefill: seq %d appends %d rows, prompt_len is %d", s, cu_new[s + 1] - cu_new[s],
                    c->hs[s].n0);
    const size_t row = (size_t)c->sh.Hkv * c->sh.D;
    for (int s = 0; s < S; ++s) {
      hipError_t e = launch_prefill_seq(c->dv, c->sh, c->hs[s], s, k + (size_t)cu_new[s] * row,
                                        v + (size_t)cu_new[s] * row, hst);
      if (e != hipSuccess) return hip_fail(e, "prefill append");
    }
    c->phase = (c->any_h2o || c->any_rocket) ? PH_PROMPT : PH_READY;
    return MKV_OK;
  }
  for (int s = 0; s < S; ++s)
    if (cu_new[s + 1] - cu_new[s] != 1) return fail(MKV_EINVAL, "decode: seq %d must append exactly 1 row", s);
  return decode_append(c, k, v, hst);
}

mkv_status mkv_h2o_update_evict(mkv_cache *c, const uint16_t *q_prompt, void *stream) {
  if (!c) return fail(MKV_EINVAL, "cache is NULL");
  hipStream_t hst = static_cast<hipStream_t>(stream);
  if (q_prompt != nullptr) {
    if (c->phase != PH_PROMPT || c->h2o_done)
      return fail(MKV_ESTATE, "H2O prefill scoring runs once, after the prefill append");
    const size_t row = (size_t)c->sh.Hq * c->sh.D;
    for (int s = 0; s < c->sh.S; ++s) {
      if (c->hs[s].method != H2O) continue;
      hipError_t e = launch_h2o_prefill_seq(c->dv, c->sh, c->hs[s], s, q_prompt + (size_t)c->hs[s].q_off * row, hst);
      if (e != hipSuccess) return hip_fail(e, "H2O prefill");
    }
    c->h2o_done = true;
    if (!c->any_rocket || c->snap_done) c->phase = PH_READY;
    return MKV_OK;
  }
  if (c->phase == PH_PROMPT && c->any_h2o) return fail(MKV_EINVAL, "H2O prefill needs q_prompt");
  if (c->phase != PH_ATTENDED) return fail(MKV_ESTATE, "eviction must follow mkv_decode_attention");
  // the victim chosen by the attention pass leaves the retained set now (exports see it gone);
  // its slot is overwritten by the next decode append, which needs no extra launch for this
  c->evict_pending = c->any_h2o;
  c->phase = PH_READY;
  return MKV_OK;
}

mkv_status mkv_snap_prefill_evict(mkv_cache *c, const uint16_t *q_window, void *stream) {
  if (!c) return fail(MKV_EINVAL, "cache is NULL");
  if (!c->any_rocket) return MKV_OK;
  if (c->phase != PH_PROMPT || c->snap_done)
    return fail(MKV_ESTATE, "SnapKV prefill eviction runs once, after the prefill append");
  if (!q_window) return fail(MKV_EINVAL, "q_window is NULL");
  hipStream_t hst = static_cast<hipStream_t>(stream);
  const size_t row = (size_t)c->sh.Hq * c->sh.D;
  for (int s = 0; s < c->sh.S; ++s) {
    if (c->hs[s].method != ROCKET) continue;
    hipError_t e = launch_snap_prefill_seq(c->dv, c->sh, c->hs[s], s, q_window + (size_t)c->hs[s].q_off * row, hst);
    if (e != hipSuccess) return hip_fail(e, "SnapKV prefill");
  }
  c->snap_done = true;
  if (!c->any_h2o || c->h2o_done) c->phase = PH_READY;
  return MKV_OK;
}

mkv_status mkv_topk_select(mkv_cache *c, const uint16_t *q, int32_t *pos_out, void *stream) {
  if (!c) return fail(MKV_EINVAL, "cache is NULL");
  if (c->phase != PH_APPENDED) return fail(MKV_ESTATE, "top-k selection must follow a decode append");
  if (c->any_rocket) {
    if (!q) return fail(MKV_EINVAL, "q is NULL");
    hipStream_t hst = static_cast<hipStream_t>(stream);
    const hipError_t e = launch_topk(c->dv, c->sh, q, pos_out, c->topk_max, hst, prof_ev(c, 3));
    if (e != hipSuccess) return hip_fail(e, "top-k select");
  }
  c->phase = PH_SELECTED;
  return MKV_OK;
}

mkv_status mkv_decode_attention(mkv_cache *c, const uint16_t *q, float *out, void *stream) {
  if (!c) return fail(MKV_EINVAL, "cache is NULL");
  if (!q || !out) return fail(MKV_EINVAL, "q and out must be non-NULL");
  if (!(c->phase == PH_SELECTED || (c->phase == PH_APPENDED && !c->any_rocket)))
    return fail(MKV_ESTATE, "attention must follow the decode append (and top-k selection)");
  hipStream_t hst = static_cast<hipStream_t>(stream);
  // one partial launch over the tiles of every sequence, then the combine
  hipError_t e = launch_attention_partial(c->dv, c->sh, q, hst, prof_ev(c, 0));
  if (e != hipSuccess) return hip_fail(e, "attention partial");
  e = launch_attention_combine(c->dv, c->sh, out, hst, prof_ev(c, 1));
  if (e != hipSuccess) return hip_fail(e, "attention combine");
  c->phase = PH_ATTENDED;
  return MKV_OK;
}

mkv_status mkv_decode_attention_noalloc(mkv_cache *c, const uint16_t *q, float *out, void *stream) {
  if (!c) return fail(MKV_EINVAL, "cache is NULL");
  if (!q || !out) return fail(MKV_EINVAL, "q and out must be non-NULL");
  if (!(c->phase == PH_SELECTED || (c->phase == PH_APPENDED && !c->any_rocket)))
    return fail(MKV_ESTATE, "attention must follow the decode append (and top-k selection)");
  const size_t need = sizeof(float) * (size_t)c->dv.n_tiles * c->sh.G * (c->sh.D + 2);
  if (need > kStaticScratchBytes)
    return fail(MKV_ENOMEM, "split-K workspace of %zu bytes exceeds the %zu-byte static workspace", need,
                kStaticScratchBytes);
  float *ws = nullptr;
  size_t ws_bytes = 0;
  hipError_t e = static_scratch(&ws, &ws_bytes);
  if (e != hipSuccess) return hip_fail(e, "static workspace address");
  Dev dv = c->dv;
  dv.partials = ws;
  hipStream_t hst = static_cast<hipStream_t>(stream);
  e = launch_attention_partial(dv, c->sh, q, hst, prof_ev(c, 0));
  if (e != hipSuccess) return hip_fail(e, "attention partial");
  e = launch_attention_combine(dv, c->sh, out, hst, prof_ev(c, 1));
  if (e != hipSuccess) return hip_fail(e, "attention combine");
  c->phase = PH_ATTENDED;
  return MKV_OK;
}

mkv_status mkv_decode_step(mkv_cache *c, const uint16_t *k, const uint16_t *v, const uint16_t *q, float *out,
                           void *stream) {
  if (!c) return fail(MKV_EINVAL, "cache is NULL");
  if (!k || !v || !q || !out) return fail(MKV_EINVAL, "k, v, q and out must be non-NULL");
  // every check of the four calls below, made before the first of them enqueues anything, so that
  // a rejected step leaves the handle as it was; past this point only a HIP launch can fail
  if (c->phase == PH_CREATED) return fail(MKV_ESTATE, "decode step before the prefill append");
  if (!(c->phase == PH_READY || (c->phase == PH_ATTENDED && !c->any_h2o)))
    return fail(MKV_ESTATE, "decode step must follow prefill or a completed decode step");
  if (c->steps >= c->sh.max_new)
    return fail(MKV_ECAPACITY, "cache holds %d decode steps (max_new_tokens)", c->sh.max_new);
  // with RocketKV sequences present the append and the top-k share one launch
  mkv_status st = c->any_rocket ? decode_append_select(c, k, v, q, static_cast<hipStream_t>(stream))
                                : decode_append(c, k, v, static_cast<hipStream_t>(stream));
  if (st != MKV_OK) return st;
  if ((st = mkv_decode_attention(c, q, out, stream)) != MKV_OK) return st;
  return mkv_h2o_update_evict(c, nullptr, stream);
}

mkv_status mkv_kv_memory(const mkv_shape *shape, const mkv_config *cfg, int32_t prompt_len, int32_t n_generated,
                         size_t *resident, size_t *peak) {
  mkv_status st = check_shape(shape);
  if (st != MKV_OK) return st;
  if (!cfg || !resident || !peak) return fail(MKV_EINVAL, "cfg, resident and peak must be non-NULL");
  if (n_generated < 0) return fail(MKV_EINVAL, "n_generated must be >= 0");
  const int D = shape->head_dim, G = shape->n_q_heads / shape->n_kv_heads;
  if ((st = check_config(*cfg, prompt_len, D, 0)) != MKV_OK) return st;
  const long long n0 = prompt_len, gen = n_generated, n = n0 + gen, row = 4LL * D;  // K and V fp16 rows
  long long now = 0, top = 0;
  switch (cfg->method) {
    case MKV_FP16:
      now = top = n * row;
      break;
    case MKV_UQ: {
      const long long nb = n / 64;  // complete key blocks are codes, the rest fp16
      const long long k = nb * 64 * (D / 2) + nb * D * 8 + (n - nb * 64) * 2 * D;
      const long long v = n * (D / 2) + n * (D / 64) * 8;
      now = top = k + v;
      break;
    }
    case MKV_KVQ: {
      const long long bp = cfg->outlier_bp, codes = 2 * n * D * cfg->bits / 8;
      const long long n_o = (n0 * bp + 5000) / 10000, n_ov = ((long long)D * bp + 5000) / 10000;
      const long long slots = bp > 0 ? std::max(1LL, n_ov) : 1;
      // key outliers: at most n_o per channel over the prompt; decode tokens at their expected rate
      const long long kout = std::min(n_o, n0) * D + (gen * D * bp + 5000) / 10000;
      now = top = codes + D * 8 + n * 4 + (n + 1) * 4 + kout * 4 + n * slots * 8;
      break;
    }
    case MKV_H2O: {
      const long long B = (long long)cfg->budget_pct * n0 / 100, kept = std::min(B, n0);
      const long long slot = row + 8 + 4LL * G;  // rows, position, score, last logits
      now = std::min(B, kept + gen) * slot;
      // prefill: the whole prompt in fp16 with its scores, beside the kept slots; decode: B + 1
      const long long pre = n0 * row + n0 * 4 + kept * slot;
      top = std::max(pre, (gen > 0 ? std::min(B + 1, kept + gen) : kept) * slot);
      break;
    }
    case MKV_ROCKET: {
      const long long T = rocket_keep(*cfg, prompt_len), kept = std::min(T, n0);
      const long long topk = cfg->topk > 0 ? cfg->topk : T / 2;
      const long long slot = row + 2LL * D + 8;  // rows, channel-major key copy, position, score key
      now = (kept + gen) * slot + topk * 4;
      top = std::max(n0 * row + kept * slot, now);  // prefill: the whole prompt in fp16 before SnapKV
      break;
    }
  }
  *resident = (size_t)(now * shape->n_kv_heads);
  *peak = (size_t)(top * shape->n_kv_heads);
  return MKV_OK;
}

mkv_status mkv_attention_tiles(mkv_cache *c, int32_t *n_tiles, int32_t *n_tiles_uq, int32_t *n_tiles_rocket) {
  if (!c || !n_tiles) return fail(MKV_EINVAL, "NULL argument");
  *n_tiles = c->dv.n_tiles;
  if (n_tiles_uq) *n_tiles_uq = c->dv.n_tiles_uq;
  if (n_tiles_rocket) *n_tiles_rocket = c->dv.n_tiles_rk;
  return MKV_OK;
}

mkv_status mkv_probe_read_bandwidth(const void *buf, size_t bytes, uint32_t *sink, int32_t reps, double *gbs,
                                    void *stream) {
  constexpr size_t kChunk = 256 << 10;
  if (!buf || !sink || !gbs) return fail(MKV_EINVAL, "NULL argument");
  if (bytes == 0 || bytes % kChunk != 0) return fail(MKV_EINVAL, "bytes must be a positive multiple of 256 KiB");
  if (bytes / kChunk > 0x7FFFFFFFu) return fail(MKV_EINVAL, "buffer too large");
  if (reps < 1) return fail(MKV_EINVAL, "reps must be >= 1");
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipEvent_t a = nullptr, b = nullptr;
  hipError_t e = hipEventCreate(&a);
  if (e == hipSuccess) e = hipEventCreate(&b);
  if (e == hipSuccess) e = launch_probe_read(buf, bytes, kChunk, sink, st);
  float best = 0.f;
  for (int r = 0; r < reps && e == hipSuccess; ++r) {
    e = hipEventRecord(a, st);
    if (e == hipSuccess) e = launch_probe_read(buf, bytes, kChunk, sink, st);
    if (e == hipSuccess) e = hipEventRecord(b, st);
    if (e == hipSuccess) e = hipEventSynchronize(b);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
    if (e == hipSuccess && (best == 0.f || ms < best)) best = ms;
  }
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (e != hipSuccess) return hip_fail(e, "read probe");
  *gbs = best > 0.f ? (double)bytes / (best * 1e-3) / 1e9 : 0.0;
  return MKV_OK;
}

mkv_status mkv_profile_enable(mkv_cache *c, int32_t enable, int32_t max_launches) {
  if (!c) return fail(MKV_EINVAL, "cache is NULL");
  if (enable < 0 || enable >= (1 << kProfKinds)) return fail(MKV_EINVAL, "enable must be a mask of kinds 0..%d", kProfKinds - 1);
  if (enable && max_launches < 1) return fail(MKV_EINVAL, "max_launches must be >= 1");
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "profile enable");
  for (int k = 0; k < kProfKinds; ++k) {
    for (int w = 0; w < 2; ++w) {
      for (hipEvent_t ev : c->ev[k][w]) (void)hipEventDestroy(ev);
      c->ev[k][w].clear();
      if (enable >> k & 1)
        for (int i = 0; i < max_launches; ++i) {
          hipEvent_t ev;
          if ((e = hipEventCreate(&ev)) != hipSuccess) return hip_fail(e, "hipEventCreate");
          c->ev[k][w].push_back(ev);
        }
    }
    c->prof_n[k] = 0;
  }
  c->prof_mask = enable;
  c->prof_cap = enable ? max_launches : 0;
  return MKV_OK;
}

mkv_status mkv_profile_read(mkv_cache *c, int32_t kind, int32_t *launches, double *total_ms) {
  if (!c || !launches || !total_ms) return fail(MKV_EINVAL, "NULL argument");
  if (kind < 0 || kind >= kProfKinds) return fail(MKV_EINVAL, "kind out of range");
  double tot = 0.0;
  for (int i = 0; i < c->prof_n[kind]; ++i) {
    hipError_t e = hipEventSynchronize(c->ev[kind][1][i]);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    if ((e = hipEventElapsedTime(&ms, c->ev[kind][0][i], c->ev[kind][1][i])) != hipSuccess)
      return hip_fail(e, "hipEventElapsedTime");
    tot += ms;
  }
  *launches = c->prof_n[kind];
  *total_ms = tot;
  return MKV_OK;
}

}  // extern "C"

// ---- export -------------------------------------------------------------------------------------
namespace {

template <typename T>
mkv_status dget(std::vector<T> &dst, uint64_t src, size_t n) {
  dst.resize(n);
  if (n == 0) return MKV_OK;
  hipError_t e = hipMemcpy(dst.data(), reinterpret_cast<const void *>(src), n * sizeof(T), hipMemcpyDeviceToHost);
  return check_hip(e, "export copy");
}

// Code `i` of a packed bit string: bits [bits*i, bits*i + bits), little-endian.
int unpack_bits(const uint8_t *p, int i, int bits) {
  const int bit = bits * i;
  uint32_t w = p[bit >> 3];
  if ((bit & 7) + bits > 8) w |= (uint32_t)p[(bit >> 3) + 1] << 8;
  return (int)((w >> (bit & 7)) & ((1u << bits) - 1));
}

}  // namespace

extern "C" mkv_status mkv_export(mkv_cache *c, int32_t seq, int32_t h, int32_t what, void *host_dst, size_t cap,
                                 size_t *written) {
  if (!c || !written) return fail(MKV_EINVAL, "NULL argument");
  *written = 0;
  if (seq < 0 || seq >= c->sh.S || h < 0 || h >= c->sh.Hkv) return fail(MKV_EINVAL, "seq or kv_head out of range");
  hipError_t e = hipDeviceSynchronize();
  if (e != hipSuccess) return hip_fail(e, "export sync");
  const SeqDesc &d = c->hs[seq];
  const int D = c->sh.D, G = c->sh.G;
  std::vector<int32_t> stv;
  mkv_status st = dget(stv, (uint64_t)(uintptr_t)(c->dv.state + ((size_t)seq * c->sh.Hkv + h) * ST_WORDS), ST_WORDS);
  if (st != MKV_OK) return st;
  const int count = stv[ST_COUNT];
  // H2O: a victim whose eviction is pending is no longer part of the retained set (the lowest key
  // among the last attention pass's per-part candidates)
  int gone = -1;
  if (d.method == H2O && c->evict_pending) {
    std::vector<uint32_t> vb;
    if ((st = dget(vb, d.vbest + (uint64_t)h * d.vparts * 16, (size_t)d.vparts * 4)) != MKV_OK) return st;
    unsigned long long best = ~0ull;
    for (int p = 0; p < d.vparts; ++p) {
      const unsigned long long key = (unsigned long long)vb[4 * p] | ((unsigned long long)vb[4 * p + 1] << 32);
      if (key < best) {
        best = key;
        gone = (int)vb[4 * p + 2];
      }
    }
  }
  std::vector<uint8_t> out;
  auto put = [&](const void *p, size_t bytes) {
    const uint8_t *b = static_cast<const uint8_t *>(p);
    out.insert(out.end(), b, b + bytes);
  };
  switch (what) {
    case MKV_EXPORT_COUNTS: {
      const int held = gone >= 0 ? count - 1 : count;
      int32_t v[4] = {held, stv[ST_NEXT_POS], d.method == ROCKET ? stv[ST_SEL_COUNT] : held, stv[ST_KEPT]};
      put(v, sizeof v);
      break;
    }
    case MKV_EXPORT_POSITIONS:
    case MKV_EXPORT_SCORES: {
      if (d.method == H2O || d.method == ROCKET) {
        // slots 0..count-1 hold the retained tokens
        const int nread = count;
        std::vector<int32_t> pos;
        if ((st = dget(pos, d.pos + (uint64_t)h * stride_slots(d) * 4, nread)) != MKV_OK) return st;
        std::vector<float> sc;
        if (d.method == H2O && (st = dget(sc, d.score + (uint64_t)h * stride_slots(d) * 4, nread)) != MKV_OK) return st;
        std::vector<int> order;
        for (int i = 0; i < nread; ++i)
          if (pos[i] >= 0 && i != gone) order.push_back(i);
        std::sort(order.begin(), order.end(), [&](int a, int b) { return pos[a] < pos[b]; });
        for (int i : order) {
          if (what == MKV_EXPORT_POSITIONS) put(&pos[i], 4);
          else if (d.method == H2O) put(&sc[i], 4);
        }
        if (what == MKV_EXPORT_SCORES && d.method != H2O) return fail(MKV_EINVAL, "SCORES is for H2O sequences");
      } else {
        if (what == MKV_EXPORT_SCORES) return fail(MKV_EINVAL, "SCORES is for H2O sequences");
        for (int32_t i = 0; i < count; ++i) put(&i, 4);
      }
      break;
    }
    case MKV_EXPORT_CODES_K:
    case MKV_EXPORT_CODES_V: {
      if (d.method != KVQ && d.method != UQ) return fail(MKV_EINVAL, "codes exist for UQ and KVQ sequences");
      const bool isk = what == MKV_EXPORT_CODES_K;
      const int n = (d.method == UQ && isk) ? (count / 64) * 64 : count;
      const int bits = d.method == UQ ? 4 : d.bits;
      // values sit in 4-token blocks: KVQ code of channel c, token j at bit bits*(4c + j); UQ as
      // laid out by uq_vbit; key code rows are one token each
      const bool quad = !isk;
      const size_t nbytes = (size_t)(quad ? (n + 3) & ~3 : n) * d.rowbytes;
      std::vector<uint8_t> raw;
      if ((st = dget(raw, (isk ? d.kc : d.vc) + (uint64_t)h * stride_codes(d), nbytes)) != MKV_OK) return st;
      for (int t = 0; t < n; ++t)
        for (int ch = 0; ch < D; ++ch) {
          const uint8_t *blk = raw.data() + (size_t)(t / 4) * 4 * d.rowbytes;
          uint8_t code;
          if (!quad) code = (uint8_t)unpack_bits(raw.data() + (size_t)t * d.rowbytes, ch, bits);
          else if (d.method == KVQ) code = (uint8_t)unpack_bits(blk, 4 * ch + (t & 3), bits);
          else code = (uint8_t)((blk[uq_vbit(ch, t & 3, D) >> 3] >> (uq_vbit(ch, t & 3, D) & 7)) & 15u);
          put(&code, 1);
        }
      break;
    }
    case MKV_EXPORT_OUTLIERS_K:
    case MKV_EXPORT_OUTLIERS_V: {
      if (d.method != KVQ) return fail(MKV_EINVAL, "outliers exist for KVQ sequences");
      std::vector<int32_t> m((size_t)count * D, -1);
      if (what == MKV_EXPORT_OUTLIERS_K) {
        std::vector<uint32_t> row, pool;
        if ((st = dget(row, d.krow + (uint64_t)h * stride_krow(d) * 4, count + 1)) != MKV_OK) return st;
        if ((st = dget(pool, d.kout + (uint64_t)h * stride_kout(d) * 4, row[count])) != MKV_OK) return st;
        for (int t = 0; t < count; ++t)
          for (uint32_t e2 = row[t]; e2 < row[t + 1]; ++e2) m[(size_t)t * D + outlier_ch(pool[e2])] = (int32_t)(pool[e2] >> 16);
      } else {
        std::vector<uint32_t> vo;
        if ((st = dget(vo, d.vout + (uint64_t)h * stride_vout(d) * 4, (size_t)d.cap * d.nov_slots)) != MKV_OK)
          return st;
        for (int t = 0; t < count; ++t)
          for (int j = 0; j < d.nov_slots; ++j) {
            const uint32_t ent = vo[(size_t)j * d.cap + t];
            if (ent == kNoOutlier) break;
            m[(size_t)t * D + outlier_ch(ent)] = (int32_t)(ent >> 16);
          }
      }
      put(m.data(), m.size() * 4);
      break;
    }
    case MKV_EXPORT_SCALES_K:
    case MKV_EXPORT_SCALES_V: {
      if (d.method == KVQ) {
        if (what == MKV_EXPORT_SCALES_K) {
          std::vector<float> t2;
          if ((st = dget(t2, d.kmeta + (uint64_t)h * D * 8, (size_t)2 * D)) != MKV_OK) return st;
          for (int ch = 0; ch < D; ++ch) put(&t2[2 * ch], 4);
        } else {
          std::vector<float> s;
          if ((st = dget(s, d.vmeta + (uint64_t)h * stride_slots(d) * 4, count)) != MKV_OK) return st;
          put(s.data(), s.size() * 4);
        }
      } else if (d.method == UQ) {
        std::vector<float> m;
        if (what == MKV_EXPORT_SCALES_K) {
          if ((st = dget(m, d.kmeta + (uint64_t)h * stride_uq_kmeta(d, D) * 8, (size_t)(count / 64) * D * 2)) != MKV_OK)
            return st;
        } else {
          if ((st = dget(m, d.vmeta + (uint64_t)h * stride_uq_vmeta(d, D) * 8, (size_t)count * (D / 64) * 2)) != MKV_OK)
            return st;
        }
        put(m.data(), m.size() * 4);
      } else {
        return fail(MKV_EINVAL, "scales exist for UQ and KVQ sequences");
      }
      break;
    }
    case MKV_EXPORT_TOPK: {
      if (d.method != ROCKET) return fail(MKV_EINVAL, "TOPK is for ROCKET sequences");
      const int m = stv[ST_SEL_COUNT];
      std::vector<int32_t> sel, pos;
      if ((st = dget(sel, d.sel + (uint64_t)h * stride_sel(d) * 4, m)) != MKV_OK) return st;
      if ((st = dget(pos, d.pos + (uint64_t)h * stride_slots(d) * 4, count)) != MKV_OK) return st;
      for (int i = 0; i < m; ++i) put(&pos[sel[i]], 4);
      break;
    }
    case MKV_EXPORT_CHANNELS: {
      if (d.method != ROCKET) return fail(MKV_EINVAL, "CHANNELS is for ROCKET sequences");
      std::vector<int32_t> ch;
      if ((st = dget(ch, d.aux1 + (uint64_t)h * D * 4, d.nch)) != MKV_OK) return st;
      put(ch.data(), ch.size() * 4);
      break;
    }
    default:
      return fail(MKV_EINVAL, "unknown export kind %d", what);
  }
  (void)G;
  if (out.size() > cap) return fail(MKV_EINVAL, "export needs %zu bytes, cap is %zu", out.size(), cap);
  if (!out.empty()) std::memcpy(host_dst, out.data(), out.size());
  *written = out.size();
  return MKV_OK;
}
