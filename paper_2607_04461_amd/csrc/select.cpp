// Multi-stage candidate selection with Elo ratings (Sec. 4.2 Stage 2, Eq. 9-12), on the host.
//
// Stage 1 seeds every rating from the integer pointwise score, r = 1500 + 100 (s - 5), and keeps the
// top ceil(rho1 M).  Stage 2 plays ceil(kappa M1) matches between neighbours of the rating order,
// re-ordering after each full sweep, and keeps the top ceil(rho2 M1).  Stage 3 plays every pair of
// the survivors once (in the rating order at its start, pairs (i, j), i < j, lexicographically) and
// returns the highest rating.  Elo: E_a = 1 / (1 + 10^((r_b - r_a) / 400)), K = 32 scaled by the
// verifier's confidence (1.2 / 1.0 / 0.7), zero-sum updates.  Orders break rating ties by the smaller
// candidate index; ceil(x) is taken as ceil(x - 1e-9) so exact products are not rounded up.
#include <algorithm>
#include <cmath>
#include <string>
#include <vector>

#include "../../include/flashbon.h"
#include "model.h"

namespace fb {
namespace {

constexpr double kBaseK = 32.0, kScale = 400.0;
constexpr double kConfidenceK[3] = {1.2, 1.0, 0.7};

int ceil_count(double x) { return (int)std::ceil(x - 1e-9); }

struct Elo {
  std::vector<double> r;
  flashbon_judge_fn judge;
  void *ctx;
  int calls = 0;

  std::vector<int32_t> order(std::vector<int32_t> ids) const {
    std::sort(ids.begin(), ids.end(), [&](int32_t x, int32_t y) { return r[x] != r[y] ? r[x] > r[y] : x < y; });
    return ids;
  }
  // one verifier call and rating update; false if the verifier broke its contract
  bool match(int32_t a, int32_t b) {
    int32_t conf = -1;
    const int32_t w = judge(ctx, a, b, &conf);
    ++calls;
    if ((w != a && w != b) || conf < 0 || conf > 2) return false;
    const double expect_a = 1.0 / (1.0 + std::pow(10.0, (r[b] - r[a]) / kScale));
    const double delta = kBaseK * kConfidenceK[conf] * ((w == a ? 1.0 : 0.0) - expect_a);
    r[a] += delta;
    r[b] -= delta;
    return true;
  }
};

}  // namespace
}  // namespace fb

using namespace fb;

extern "C" flashbon_status flashbon_select(int32_t m, const int32_t *scores, double rho1, double rho2,
                                           double kappa, flashbon_judge_fn judge, void *ctx,
                                           int32_t *winner, double *ratings, int32_t *pairwise_calls) {
  if (m < 1) return fail(FLASHBON_ESHAPE, "m must be >= 1");
  if (!scores || !judge || !winner) return fail(FLASHBON_EINVAL, "scores, judge and winner are required");
  if (!(rho1 > 0.0 && rho1 <= 1.0) || !(rho2 > 0.0 && rho2 <= 1.0))
    return fail(FLASHBON_EINVAL, "rho1 and rho2 must lie in (0, 1]");
  if (!(kappa >= 0.0) || !std::isfinite(kappa) || kappa * m > 1e9)
    return fail(FLASHBON_EINVAL, "kappa must be finite and >= 0");
  for (int j = 0; j < m; ++j)
    if (scores[j] < 1 || scores[j] > 10)
      return fail(FLASHBON_EINVAL, "scores[" + std::to_string(j) + "] outside 1..10");

  Elo elo;
  elo.judge = judge;
  elo.ctx = ctx;
  elo.r.resize(m);
  std::vector<int32_t> all(m);
  for (int j = 0; j < m; ++j) {
    elo.r[j] = 1500.0 + 100.0 * (scores[j] - 5);
    all[j] = j;
  }
  // Stage 1: pointwise pruning + Elo seeding (Eq. 10)
  std::vector<int32_t> s1 = elo.order(all);
  s1.resize(std::min<int>(m, std::max(1, ceil_count(rho1 * m))));
  const int m1 = (int)s1.size();
  // Stage 2: neighbour matches in rating order (Eq. 11)
  const int c2 = m1 >= 2 ? ceil_count(kappa * m1) : 0;
  for (int played = 0; played < c2;) {
    const std::vector<int32_t> L = elo.order(s1);
    for (int i = 0; i + 1 < m1 && played < c2; ++i, ++played)
      if (!elo.match(L[i], L[i + 1])) return fail(FLASHBON_EINVAL, "verifier returned an invalid result");
  }
  std::vector<int32_t> s2 = elo.order(s1);
  s2.resize(std::min<int>(m1, std::max(1, ceil_count(rho2 * m1))));
  // Stage 3: dense round robin among the survivors, then the best rating (Eq. 12)
  const std::vector<int32_t> L2 = elo.order(s2);
  for (size_t i = 0; i < L2.size(); ++i)
    for (size_t j = i + 1; j < L2.size(); ++j)
      if (!elo.match(L2[i], L2[j])) return fail(FLASHBON_EINVAL, "verifier returned an invalid result");
  *winner = elo.order(s2)[0];
  if (ratings) std::copy(elo.r.begin(), elo.r.end(), ratings);
  if (pairwise_calls) *pairwise_calls = elo.calls;
  return FLASHBON_OK;
}
