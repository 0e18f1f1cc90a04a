// Host-side dispatch of one draft step (no device work).
#pragma once

#include "../../include/flashbon.h"

namespace fb {

bool meta_valid(const flashbon_cache_meta &m);

// Fills trace[L] and advances meta[L] in place (see flashbon_plan_step).  residual: proxies add a
// forecast residual delta to their input, so every proxy is live.
void plan_step(int L, const uint8_t *skip, const uint8_t *proxy, flashbon_cache_meta *meta,
               float t_cur, flashbon_trace_entry *trace, bool residual = false);

// Coefficients (ca, cb) of the difference form h1 + ca (h1 - h2) + cb (h1 - 2 h2 + h3) for a proxy
// of the given order, from the block's metadata before the step.
void taylor_coefficients(const flashbon_cache_meta &m_before, float t_cur, int order, float *ca,
                         float *cb);

}  // namespace fb
