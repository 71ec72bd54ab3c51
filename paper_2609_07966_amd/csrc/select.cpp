// Host side of MetaKV's per-prompt configuration choice (Section 2.3): the budget filter, the
// preference hierarchy, and the violation-score fallback, over candidates whose latency, memory and
// accuracy predictions the caller supplies.
#include <vector>

#include "mkv.h"
#include "mkv_internal.h"

using mkv::report_error;

extern "C" mkv_status mkv_select_config(const mkv_candidate *c, int32_t n, double l_max, double m_max,
                                        int32_t *chosen, int32_t *violated) {
  if (!c || !chosen || !violated || n < 1) return report_error(MKV_EINVAL, "cands, chosen, violated and n >= 1 required");
  if (!(l_max > 0.0) || !(m_max > 0.0)) return report_error(MKV_EINVAL, "l_max and m_max must be positive");
  // Step 3: the budget filter
  std::vector<int> keep;
  for (int i = 0; i < n; ++i)
    if (c[i].latency <= l_max && c[i].memory <= m_max) keep.push_back(i);
  *violated = keep.empty() ? 1 : 0;
  if (keep.empty()) {
    // no candidate fits: the smallest combined relative violation, then the most accurate
    int best = 0;
    double bv = c[0].latency / l_max + c[0].memory / m_max;
    for (int i = 1; i < n; ++i) {
      const double v = c[i].latency / l_max + c[i].memory / m_max;
      if (v < bv || (v == bv && c[i].p_correct > c[best].p_correct)) {
        best = i;
        bv = v;
      }
    }
    *chosen = best;
    return MKV_OK;
  }
  // Step 4: uncompressed FP16 whenever it fits
  for (int i : keep)
    if (c[i].method == MKV_FP16) {
      *chosen = i;
      return MKV_OK;
    }
  // Step 5: the least compressed kept setting of each method
  std::vector<int> least;
  for (int i : keep) {
    bool best_of_method = true;
    for (int j : keep)
      if (c[j].method == c[i].method && (c[j].level < c[i].level || (c[j].level == c[i].level && j < i))) {
        best_of_method = false;
        break;
      }
    if (best_of_method) least.push_back(i);
  }
  // Steps 6-7: a single survivor, else the highest predicted accuracy (least is in index order)
  int best = least[0];
  for (int i : least)
    if (c[i].p_correct > c[best].p_correct) best = i;
  *chosen = best;
  return MKV_OK;
}
