// Adaptive rollout-depth controller (Sec. 5.1; App. D, Algorithm 1 and its
// configuration table): host code that turns a probe batch's per-turn KL
// statistics and its successful completion lengths into the rollout depth
// cap of the following steps.  Turn indices are 0-based; the cap's +1 turns
// an index into a number of turns.

#include <math.h>

#include <algorithm>
#include <vector>

#include "turnkl.h"

namespace {

bool config_ok(const turnkl_depth_config* c) {
  if (!c) return false;
  if (c->h_min < 1 || c->h_max < c->h_min) return false;
  if (c->warmup_steps < 0 || c->probe_interval < 1 || c->min_cov_traj < 0) return false;
  if (!(c->coverage_quantile > 0.0 && c->coverage_quantile <= 1.0)) return false;
  if (!(c->ema_alpha >= 0.0 && c->ema_alpha <= 1.0)) return false;
  if (!(c->eps >= 0.0) || !isfinite(c->eps)) return false;
  return true;
}

// round() of the controller: nearest integer, ties to even (the default
// floating-point rounding mode).
int round_even(double x) { return (int)nearbyint(x); }

// sum_t t q_t with m_t = [K_t]_+ n_t / n_0 and q_t = m_t / (sum_j m_j + eps),
// accumulated in turn order.
double efficiency_centroid(const turnkl_depth_config* c, const turnkl_turn_stat* s, int n_turns) {
  const double n0 = (double)s[0].n_traj;
  std::vector<double> m(n_turns, 0.0);
  double total = 0.0;
  for (int t = 0; t < n_turns; ++t) {
    const double k = s[t].kl_mean > 0.0 ? s[t].kl_mean : 0.0;
    m[t] = n0 > 0.0 ? k * (double)s[t].n_traj / n0 : 0.0;
    total += m[t];
  }
  total += c->eps;
  double centroid = 0.0;
  for (int t = 0; t < n_turns; ++t) centroid += (double)t * (m[t] / total);
  return centroid;
}

// min{H >= 0 : #{i : L_i - 1 <= H} / n >= p}: the completion indices sorted,
// the answer is the first value whose count of entries at or below it
// reaches p n.
int coverage_floor(const turnkl_depth_config* c, const int32_t* len, long long n) {
  std::vector<int32_t> last(len, len + n);
  for (auto& v : last) v -= 1;
  std::sort(last.begin(), last.end());
  long long i = 0;
  while (i < n) {
    long long j = i;
    while (j + 1 < n && last[j + 1] == last[i]) ++j;
    if ((double)(j + 1) / (double)n >= c->coverage_quantile) return last[i];
    i = j + 1;
  }
  return last[n - 1];  // not reached: the full count reaches any p <= 1
}

}  // namespace

extern "C" {

void turnkl_depth_default_config(turnkl_depth_config* cfg) {
  if (!cfg) return;
  cfg->h_min = 2;
  cfg->h_max = 50;
  cfg->warmup_steps = 3;
  cfg->probe_interval = 8;
  cfg->min_cov_traj = 8;
  cfg->coverage_quantile = 0.80;
  cfg->ema_alpha = 0.30;
  cfg->eps = 1e-12;
}

int turnkl_depth_init(const turnkl_depth_config* cfg, turnkl_depth_state* st) {
  if (!config_ok(cfg) || !st) return TURNKL_ERR_INVALID_ARG;
  st->h_bar = (double)cfg->h_max;
  st->h_eff_bar = -1.0;
  st->h_eff = -1;
  st->h_cov = 0;
  st->h_ctrl = -1;
  st->n_probes = 0;
  return TURNKL_OK;
}

int turnkl_depth_plan(const turnkl_depth_config* cfg, const turnkl_depth_state* st, int64_t step,
                      int32_t* cap, int32_t* probe, int32_t* rollout_depth) {
  if (!config_ok(cfg) || !st || !cap || !probe || !rollout_depth || step < 1)
    return TURNKL_ERR_INVALID_ARG;
  if (!isfinite(st->h_bar)) return TURNKL_ERR_INVALID_ARG;
  // clamp before converting, so any finite state maps into [h_min, h_max]
  const double h = std::min(std::max(st->h_bar, -1.0), (double)cfg->h_max + 1.0);
  const int c = std::min(std::max(round_even(h) + 1, (int)cfg->h_min), (int)cfg->h_max);
  const bool is_probe = step <= cfg->warmup_steps || step % cfg->probe_interval == 0;
  *cap = c;
  *probe = is_probe ? 1 : 0;
  *rollout_depth = is_probe ? cfg->h_max : c;
  return TURNKL_OK;
}

int turnkl_depth_update(const turnkl_depth_config* cfg, turnkl_depth_state* st,
                        const turnkl_turn_stat* stats, int32_t n_turns,
                        const int32_t* success_lengths, int64_t n_success) {
  if (!config_ok(cfg) || !st || !stats || n_turns < 1 || n_success < 0) return TURNKL_ERR_INVALID_ARG;
  if (n_success > 0 && !success_lengths) return TURNKL_ERR_INVALID_ARG;
  for (int64_t i = 0; i < n_success; ++i)
    if (success_lengths[i] < 1) return TURNKL_ERR_INVALID_ARG;
  const double centroid = efficiency_centroid(cfg, stats, n_turns);
  st->h_eff_bar = centroid;
  st->h_eff = round_even(centroid);
  if (n_success >= std::max<int64_t>(cfg->min_cov_traj, 1))
    st->h_cov = coverage_floor(cfg, success_lengths, n_success);
  st->h_ctrl = std::max(st->h_eff, st->h_cov);
  st->h_bar = (1.0 - cfg->ema_alpha) * st->h_bar + cfg->ema_alpha * (double)st->h_ctrl;
  st->n_probes += 1;
  return TURNKL_OK;
}

}  // extern "C"
