// Host-side checks of libmkv's C ABI that need no GPU, built with AddressSanitizer and
// UndefinedBehaviorSanitizer on the host code (the kernel launchers are stubbed out: nothing here
// reaches a device).  Exercises arena sizing for every configuration, argument validation, the
// KV-memory accounting, the configuration choice and the host codebook fit.  Exit status 0 when
// every check holds.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <vector>

#include "mkv.h"
#include "mkv_internal.h"

namespace mkv {
// stubs: every path exercised here fails or returns before any launch
hipError_t launch_append_decode(const Dev &, const Shape &, const uint16_t *, const uint16_t *, hipStream_t, LaunchEv) { return hipErrorNotSupported; }
hipError_t launch_prefill_seq(const Dev &, const Shape &, const SeqDesc &, int, const uint16_t *, const uint16_t *, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_attention_partial(const Dev &, const Shape &, const uint16_t *, hipStream_t, LaunchEv) { return hipErrorNotSupported; }
hipError_t launch_attention_combine(const Dev &, const Shape &, float *, hipStream_t, LaunchEv) { return hipErrorNotSupported; }
hipError_t launch_topk(const Dev &, const Shape &, const uint16_t *, int32_t *, int, hipStream_t, LaunchEv) { return hipErrorNotSupported; }
hipError_t launch_append_select(const Dev &, const Shape &, const uint16_t *, const uint16_t *, const uint16_t *, hipStream_t, LaunchEv, LaunchEv) { return hipErrorNotSupported; }
hipError_t launch_h2o_prefill_seq(const Dev &, const Shape &, const SeqDesc &, int, const uint16_t *, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_snap_prefill_seq(const Dev &, const Shape &, const SeqDesc &, int, const uint16_t *, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_init_state(const Dev &, const Shape &, hipStream_t) { return hipErrorNotSupported; }
hipError_t launch_probe_read(const void *, size_t, size_t, uint32_t *, hipStream_t) { return hipErrorNotSupported; }
hipError_t static_scratch(float **, size_t *) { return hipErrorNotSupported; }
}  // namespace mkv

static int failures = 0;
#define CHECK(c)                                                  \
  do {                                                            \
    if (!(c)) {                                                   \
      std::printf("FAILED line %d: %s\n", __LINE__, #c);          \
      ++failures;                                                 \
    }                                                             \
  } while (0)

static mkv_config cfg(int method, int bits = 0, int bp = 0, int pct = 0, int keep = 0, int ratio = 0) {
  mkv_config c;
  std::memset(&c, 0, sizeof c);
  c.method = method;
  c.bits = bits;
  c.group = 64;
  c.outlier_bp = bp;
  c.budget_pct = pct;
  c.keep_tokens = keep;
  c.window = 32;
  c.pool = 7;
  c.n_channels = 32;
  c.keep_ratio = ratio;
  return c;
}

int main() {
  const mkv_config all[] = {cfg(MKV_FP16), cfg(MKV_UQ, 4), cfg(MKV_KVQ, 4, 100), cfg(MKV_KVQ, 3, 100),
                            cfg(MKV_KVQ, 2, 100), cfg(MKV_H2O, 0, 0, 20), cfg(MKV_H2O, 0, 0, 60),
                            cfg(MKV_ROCKET, 0, 0, 0, 1024), cfg(MKV_ROCKET, 0, 0, 0, 0, 16)};
  const int n = sizeof all / sizeof all[0];
  const int lens[] = {1, 5, 63, 64, 65, 300, 4096, 32768};
  for (int d : {64, 128})
    for (int g : {1, 4, 8}) {
      mkv_shape sh{n, 2 * g, 2, d, 17};
      for (int L : lens) {
        std::vector<int32_t> pl(n, L);
        size_t bytes = 0;
        const mkv_status st = mkv_cache_bytes(&sh, all, pl.data(), &bytes);
        CHECK(st == MKV_OK || (L < 5 && st == MKV_EINVAL));  // H2O-20 at tiny prompts: a budget of 0
        for (int i = 0; i < n; ++i) {
          size_t r = 0, p = 0;
          const mkv_status s2 = mkv_kv_memory(&sh, &all[i], L, 9, &r, &p);
          if (s2 == MKV_OK) CHECK(p >= r);
        }
      }
    }
  // validation errors with messages
  {
    mkv_shape bad{1, 6, 4, 128, 8};
    mkv_config c = cfg(MKV_FP16);
    int32_t L = 10;
    size_t b = 0;
    CHECK(mkv_cache_bytes(&bad, &c, &L, &b) == MKV_EINVAL && std::strlen(mkv_last_error()) > 0);
    CHECK(mkv_cache_bytes(nullptr, &c, &L, &b) == MKV_EINVAL);
    mkv_shape sh{1, 8, 2, 128, 8};
    mkv_config k5 = cfg(MKV_KVQ, 5, 100);
    CHECK(mkv_cache_bytes(&sh, &k5, &L, &b) == MKV_EINVAL);
    // create: short arena and malformed codebooks are refused before any device work
    mkv_config kv = cfg(MKV_KVQ, 3, 100);
    CHECK(mkv_cache_bytes(&sh, &kv, &L, &b) == MKV_OK);
    std::vector<float> cb;
    for (int bits = 2; bits <= 4; ++bits)
      for (int half = 0; half < 2; ++half)
        for (int i = 0; i < (1 << bits); ++i) cb.push_back(-1.f + 2.f * i / ((1 << bits) - 1));
    for (float &x : cb) x = mkv::round_to_half(x);
    mkv_cache *h = nullptr;
    void *fake = reinterpret_cast<void *>(uintptr_t(1) << 40);
    CHECK(mkv_cache_create(&sh, &kv, &L, cb.data(), fake, b - 1, nullptr, &h) == MKV_ENOMEM && h == nullptr);
    std::vector<float> nan = cb;
    nan[9] = NAN;
    CHECK(mkv_cache_create(&sh, &kv, &L, nan.data(), fake, b, nullptr, &h) == MKV_EINVAL);
    std::vector<float> off = cb;
    off[2] += 1e-4f;
    CHECK(mkv_cache_create(&sh, &kv, &L, off.data(), fake, b, nullptr, &h) == MKV_EINVAL);
    CHECK(mkv_cache_destroy(nullptr) == MKV_OK);
  }
  // attention tile layout: every (sequence, kv head)'s ranges cover its tokens once, partial
  // slots are distinct, RocketKV tiles launch last, and the quantized tiles are spread over the
  // first 3/4 of the others (so about a quarter of the fp16-row tiles follow the last of them);
  // a long mixed launch (several rounds of workgroups) and a short one
  for (int big = 0; big < 2; ++big) {
    const int S = big ? 64 : 6, Hkv = 8, D = 128;
    mkv_shape sh{S, 4 * Hkv, Hkv, D, 128};
    std::vector<mkv_config> cs(S);
    std::vector<int32_t> pl(S);
    uint32_t r = 777u + big;
    for (int i = 0; i < S; ++i) {
      cs[i] = all[i % n];
      r = r * 1664525u + 1013904223u;
      pl[i] = 1024 + (int)((r >> 8) % (big ? 31744u : 3000u));
    }
    std::vector<int4> tiles;
    std::vector<mkv::SeqDesc> sd;
    CHECK(mkv::layout_tiles(&sh, cs.data(), pl.data(), &tiles, &sd) == MKV_OK);
    int expect = 0;
    for (int i = 0; i < S; ++i) expect += Hkv * sd[i].tile_count;
    CHECK((int)tiles.size() == expect);
    std::vector<int> seen(tiles.size(), 0);
    std::vector<std::vector<int>> cover(S * Hkv);
    int last_nonrocket = -1, first_rocket = (int)tiles.size(), last_quant = -1, n_rows = 0;
    for (int i = 0; i < (int)tiles.size(); ++i) {
      const int4 t = tiles[i];
      CHECK(t.x >= 0 && t.x < S && t.y >= 0 && t.y < Hkv);
      if (!(t.x >= 0 && t.x < S && t.y >= 0 && t.y < Hkv)) continue;
      const mkv::SeqDesc &d = sd[t.x];
      const int amax = d.method == mkv::ROCKET ? d.topk : d.cap;
      CHECK(d.chunk > 0 && d.chunk % 64 == 0 && t.z % d.chunk == 0);
      CHECK(t.z < t.w && t.w == std::min(amax, t.z + d.chunk));
      const int slot = d.tile_first + t.y * d.tile_count + t.z / d.chunk;
      CHECK(slot >= 0 && slot < (int)tiles.size());
      if (slot >= 0 && slot < (int)tiles.size()) ++seen[slot];
      cover[t.x * Hkv + t.y].push_back(t.z);
      if (d.method == mkv::ROCKET) {
        first_rocket = std::min(first_rocket, i);
      } else {
        last_nonrocket = i;
        if (d.method == mkv::KVQ || d.method == mkv::UQ) last_quant = i;
        else ++n_rows;
      }
    }
    for (int v : seen) CHECK(v == 1);
    CHECK(last_nonrocket < first_rocket);
    int rows_after = 0;
    for (int i = last_quant + 1; i < first_rocket; ++i) rows_after += 1;
    CHECK(last_quant < 0 || rows_after >= n_rows / 4 - 1);
    for (int p = 0; p < S * Hkv; ++p) {
      std::vector<int> z = cover[p];
      std::sort(z.begin(), z.end());
      const mkv::SeqDesc &d = sd[p / Hkv];
      CHECK((int)z.size() == d.tile_count);
      for (int j = 0; j < (int)z.size(); ++j) CHECK(z[j] == j * d.chunk);
    }
  }
  // the configuration choice
  {
    mkv_candidate c[3] = {{MKV_KVQ, 0, 3.0, 5.0, 0.6}, {MKV_H2O, 1, 1.0, 9.0, 0.5}, {MKV_FP16, 0, 2.0, 20.0, 0.7}};
    int32_t ch = -1, vi = -1;
    CHECK(mkv_select_config(c, 3, 5.0, 30.0, &ch, &vi) == MKV_OK && ch == 2 && vi == 0);
    CHECK(mkv_select_config(c, 3, 5.0, 10.0, &ch, &vi) == MKV_OK && ch == 0 && vi == 0);
    CHECK(mkv_select_config(c, 3, 0.5, 1.0, &ch, &vi) == MKV_OK && vi == 1);
    CHECK(mkv_select_config(c, 0, 1.0, 1.0, &ch, &vi) == MKV_EINVAL);
  }
  // host codebook fit on a small draw
  {
    const int T = 200, H = 2, D = 64;
    std::vector<uint16_t> k(T * H * D), v(T * H * D);
    uint32_t s = 12345;
    for (size_t i = 0; i < k.size(); ++i) {
      s = s * 1664525u + 1013904223u;
      const float x = ((s >> 8) & 0xFFFF) / 32768.f - 1.f;
      const _Float16 hx = (_Float16)x;
      std::memcpy(&k[i], &hx, 2);
      std::memcpy(&v[i], &hx, 2);
    }
    for (int bits = 2; bits <= 4; ++bits) {
      std::vector<float> a(1 << bits), bb(1 << bits);
      CHECK(mkv_fit_codebooks(k.data(), v.data(), T, H, D, bits, 100, a.data(), bb.data()) == MKV_OK);
      for (int i = 1; i < (1 << bits); ++i) CHECK(a[i] >= a[i - 1] && bb[i] >= bb[i - 1]);
    }
    float a[4], bb[4];
    CHECK(mkv_fit_codebooks(k.data(), v.data(), 0, H, D, 2, 100, a, bb) == MKV_EINVAL);
  }
  std::printf("%s (%d failures)\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
