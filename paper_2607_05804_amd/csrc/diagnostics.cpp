// Turn-level loss-allocation diagnostics: host code over the per-turn
// statistics of one batch.  Sec. 4.4 defines s_t, the turn's share of the
// batch's loss mass, and reports (Table 1) the deep/shallow raw-KL ratio, the
// deep third's survivor support and its loss budget over the reliable turn
// prefix; Sec. 7.2 (Table 3) reports the budget spent on the deepest third of
// valid turns; Sec. 4.2 defines G_t = K_t^fail - K_t^succ.

#include <math.h>

#include "turnkl.h"

namespace {

// Leading turns with at least max(n_min, 1) survivors.
int reliable_prefix(const turnkl_turn_stat* s, int n_turns, long long n_min) {
  int p = 0;
  while (p < n_turns && s[p].n_traj > 0 && s[p].n_traj >= n_min) ++p;
  return p;
}

double total_mass(const turnkl_turn_stat* s, int n_turns) {
  double total = 0.0;
  for (int t = 0; t < n_turns; ++t) total += s[t].loss_mass;
  return total;
}

}  // namespace

extern "C" {

int turnkl_loss_share(const turnkl_turn_stat* stats, int32_t n_turns, double* share) {
  if (!stats || !share || n_turns < 1) return TURNKL_ERR_INVALID_ARG;
  const double total = total_mass(stats, n_turns);
  for (int t = 0; t < n_turns; ++t) share[t] = total != 0.0 ? stats[t].loss_mass / total : 0.0;
  return TURNKL_OK;
}

int turnkl_budget_report(const turnkl_turn_stat* stats, int32_t n_turns, int64_t n_traj,
                         int32_t support_floor, double support_frac, turnkl_budget* out) {
  if (!stats || !out || n_turns < 1 || n_traj < 0 || support_floor < 0) return TURNKL_ERR_INVALID_ARG;
  if (!(support_frac >= 0.0 && support_frac <= 1.0)) return TURNKL_ERR_INVALID_ARG;
  const double c = ceil(support_frac * (double)n_traj);
  const long long n_min = support_floor > (long long)c ? support_floor : (long long)c;
  turnkl_budget r{};
  r.n_min = n_min;
  r.prefix = reliable_prefix(stats, n_turns, n_min);
  r.deep_shallow_kl = NAN;
  if (r.prefix > 0) {
    const int P = r.prefix;
    const int k = (P + 2) / 3;
    r.third = k;
    const double total = total_mass(stats, n_turns);
    const double n0 = (double)stats[0].n_traj;
    double kl_shallow = 0.0, kl_deep = 0.0, support = 0.0;
    for (int j = 0; j < k; ++j) {
      const turnkl_turn_stat& sh = stats[j];
      const turnkl_turn_stat& dp = stats[P - k + j];
      if (total != 0.0) {
        r.shallow_budget += sh.loss_mass / total;
        r.deep_budget += dp.loss_mass / total;
      }
      kl_shallow += sh.kl_mean;
      kl_deep += dp.kl_mean;
      support += (double)dp.n_traj / n0;
    }
    r.deep_support = support / k;
    kl_shallow /= k;
    kl_deep /= k;
    if (kl_shallow != 0.0) r.deep_shallow_kl = kl_deep / kl_shallow;
  }
  *out = r;
  return TURNKL_OK;
}

int turnkl_outcome_gap(const turnkl_turn_stat* outcome_stats, int32_t n_turns, double* gap) {
  if (!outcome_stats || !gap || n_turns < 1) return TURNKL_ERR_INVALID_ARG;
  const turnkl_turn_stat* fail = outcome_stats;
  const turnkl_turn_stat* succ = outcome_stats + n_turns;
  for (int t = 0; t < n_turns; ++t)
    gap[t] = (fail[t].n_tokens > 0 && succ[t].n_tokens > 0) ? fail[t].kl_mean - succ[t].kl_mean
                                                            : NAN;
  return TURNKL_OK;
}

}  // extern "C"
