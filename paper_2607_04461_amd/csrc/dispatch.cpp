// Host-side dispatch of one draft step: the action of every block (Eq. 3-6), the Taylor order, the
// cache ring slot, whether a proxy's output is ever read, and the Taylor coefficients.
#include "dispatch.h"

#include <cmath>

namespace fb {

bool meta_valid(const flashbon_cache_meta &m) {
  return m.count >= 0 && m.count <= 3 && m.head >= 0 && m.head <= 2;
}

void plan_step(int L, const uint8_t *skip, const uint8_t *proxy, flashbon_cache_meta *meta,
               float t_cur, flashbon_trace_entry *trace, bool residual) {
  // 1) action per block: skip wins; a proxy needs at least one cached entry
  for (int l = 0; l < L; ++l) {
    int8_t a = FLASHBON_COMPUTE;
    if (skip && skip[l]) a = FLASHBON_SKIP;
    else if (proxy && proxy[l] && meta[l].count >= 1) a = FLASHBON_PROXY;
    trace[l].action = a;
  }
  // 2) order/slot/live from the metadata as it was before this step; liveness looks at the next
  //    non-skipped block; then computed blocks advance their ring.
  for (int l = 0; l < L; ++l) {
    flashbon_trace_entry &e = trace[l];
    flashbon_cache_meta &m = meta[l];
    if (e.action == FLASHBON_SKIP) {
      e.order = -1; e.slot = -1; e.live = 0;
    } else if (e.action == FLASHBON_PROXY) {
      int c = m.count < 3 ? m.count : 3;
      e.order = (int8_t)(c - 1);
      e.slot = (int8_t)((m.head + 2) % 3);
      int next = -1;
      for (int j = l + 1; j < L; ++j)
        if (trace[j].action != FLASHBON_SKIP) { next = trace[j].action; break; }
      e.live = (residual || next == -1 || next == FLASHBON_COMPUTE) ? 1 : 0;
    } else {
      e.order = -1;
      e.slot = (int8_t)m.head;
      e.live = 1;
      m.t[m.head] = t_cur;
      m.head = (m.head + 1) % 3;
      m.count = m.count < 3 ? m.count + 1 : 3;
    }
  }
}

// Eq. 3-5 with Delta = t_cur - tau1, d = tau1 - tau2:
//   Delta * hdot = (Delta/d)(h1 - h2),  Delta^2/2 * hddot = (Delta/d)^2/2 (h1 - 2 h2 + h3).
void taylor_coefficients(const flashbon_cache_meta &m_before, float t_cur, int order, float *ca,
                         float *cb) {
  *ca = 0.f;
  *cb = 0.f;
  if (order < 1) return;
  const int s1 = (m_before.head + 2) % 3, s2 = (m_before.head + 1) % 3;
  const double tau1 = m_before.t[s1], tau2 = m_before.t[s2];
  const double r = ((double)t_cur - tau1) / (tau1 - tau2);
  *ca = (float)r;
  if (order >= 2) *cb = (float)(0.5 * r * r);
}

}  // namespace fb
