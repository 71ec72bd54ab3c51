// Host-side KVQ codebook fitting (offline calibration, as in KVQuant): normalise a calibration
// draw with the cache's outlier-threshold rules and fit a 2^b-entry codebook by 1-D Lloyd k-means.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "mkv.h"
#include "mkv_internal.h"

using mkv::report_error;
using mkv::round_to_half;

namespace {

float h2f(uint16_t h) {
  const uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
  const uint32_t exp = (h >> 10) & 0x1Fu, man = h & 0x3FFu;
  uint32_t bits;
  if (exp == 0) {
    if (man == 0) {
      bits = sign;
    } else {  // subnormal: value = man * 2^-24
      float f = std::ldexp((float)man, -24);
      std::memcpy(&bits, &f, 4);
      bits |= sign;
    }
  } else if (exp == 31) {
    bits = sign | 0x7F800000u | (man << 13);
  } else {
    bits = sign | ((exp + 112) << 23) | (man << 13);
  }
  float f;
  std::memcpy(&f, &bits, 4);
  return f;
}

int outlier_count(long long n, int bp) { return (int)((n * bp + 5000) / 10000); }

// idx-th largest (0-based) of |x|; 0 when idx >= n
float order_stat_desc(std::vector<float> a, int idx) {
  if (idx >= (int)a.size()) return 0.f;
  for (float &x : a) x = std::fabs(x);
  std::nth_element(a.begin(), a.begin() + idx, a.end(), std::greater<float>());
  return a[idx];
}

float recip(float t) { return t > 0.f ? 1.0f / t : 0.f; }

std::vector<float> lloyd(std::vector<double> x, int bits) {
  std::sort(x.begin(), x.end());
  const size_t n = x.size();
  const int K = 1 << bits;
  std::vector<double> c(K);
  for (int i = 0; i < K; ++i) c[i] = x[std::min(n - 1, (size_t)(((2 * (size_t)i + 1) * n) / (2 * (size_t)K)))];
  std::vector<int> assign(n, -1), prev;
  for (int it = 0; it < 100; ++it) {
    for (size_t j = 0; j < n; ++j) {
      int best = 0;
      double bd = std::fabs(x[j] - c[0]);
      for (int i = 1; i < K; ++i) {
        const double dd = std::fabs(x[j] - c[i]);
        if (dd < bd) { bd = dd; best = i; }
      }
      assign[j] = best;
    }
    if (!prev.empty() && prev == assign) break;
    prev = assign;
    std::vector<double> sum(K, 0.0);
    std::vector<long long> cnt(K, 0);
    for (size_t j = 0; j < n; ++j) {
      sum[assign[j]] += x[j];
      cnt[assign[j]]++;
    }
    for (int i = 0; i < K; ++i)
      if (cnt[i] > 0) c[i] = sum[i] / (double)cnt[i];
  }
  // the codebook is stored in fp16, like the cache's other values
  std::vector<float> out(K);
  for (int i = 0; i < K; ++i) out[i] = round_to_half(c[i]);
  std::sort(out.begin(), out.end());
  return out;
}

}  // namespace

extern "C" mkv_status mkv_fit_codebooks(const uint16_t *k, const uint16_t *v, int32_t n, int32_t Hkv, int32_t D,
                                        int32_t bits, int32_t bp, float *cb_k, float *cb_v) {
  if (!k || !v || !cb_k || !cb_v) return report_error(MKV_EINVAL, "k, v, cb_k and cb_v must be non-NULL");
  if (n < 1 || Hkv < 1 || D < 1) return report_error(MKV_EINVAL, "n_tokens, n_kv_heads and head_dim must be >= 1");
  if (bits < 1 || bits > 8) return report_error(MKV_EINVAL, "bits must be in 1..8");
  if (bp < 0 || bp > 5000) return report_error(MKV_EINVAL, "outlier_bp must be in 0..5000");
  std::vector<double> ks, vs;
  std::vector<float> col(n), row(D);
  for (int h = 0; h < Hkv; ++h) {
    std::vector<float> tau(D), inv(D);
    for (int c = 0; c < D; ++c) {
      for (int t = 0; t < n; ++t) col[t] = h2f(k[((size_t)t * Hkv + h) * D + c]);
      tau[c] = bp == 0 ? order_stat_desc(col, 0) : order_stat_desc(col, outlier_count(n, bp));
      inv[c] = recip(tau[c]);
    }
    for (int t = 0; t < n; ++t)
      for (int c = 0; c < D; ++c) {
        const float x = h2f(k[((size_t)t * Hkv + h) * D + c]);
        if (std::fabs(x) <= tau[c]) {
          volatile float xh = x * inv[c];
          ks.push_back((double)xh);
        }
      }
    for (int t = 0; t < n; ++t) {
      for (int c = 0; c < D; ++c) row[c] = h2f(v[((size_t)t * Hkv + h) * D + c]);
      const float s = bp == 0 ? order_stat_desc(row, 0) : order_stat_desc(row, outlier_count(D, bp));
      const float is = recip(s);
      for (int c = 0; c < D; ++c)
        if (std::fabs(row[c]) <= s) {
          volatile float xh = row[c] * is;
          vs.push_back((double)xh);
        }
    }
  }
  if (ks.empty() || vs.empty()) return report_error(MKV_EINVAL, "no non-outlier samples to fit");
  const std::vector<float> a = lloyd(ks, bits), b = lloyd(vs, bits);
  std::copy(a.begin(), a.end(), cb_k);
  std::copy(b.begin(), b.end(), cb_v);
  return MKV_OK;
}
