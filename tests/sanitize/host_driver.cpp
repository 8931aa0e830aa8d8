// Runs the library's host-only code (the rollout-depth controller and the
// loss-allocation diagnostics) under AddressSanitizer and
// UndefinedBehaviorSanitizer.  Test infrastructure: built and run only by
// tests/test_sanitizers.py.
//
// usage: host_driver IN OUT
//   IN : int32 n_turns, int32 n_success, int64 n_traj, int32 support_floor,
//        float64 support_frac, then turnkl_turn_stat stats[n_turns],
//        outcome_stats[2 * n_turns], int32 success_lengths[n_success]
//   OUT: for steps 1..24 of the controller with the default configuration,
//        updated on every probe step with these statistics: int32 cap,
//        probe, rollout_depth, then the state after the step (float64 h_bar,
//        h_eff_bar, int32 h_eff, h_cov, h_ctrl, n_probes); then float64
//        share[n_turns], the turnkl_budget fields (int64 n_min, int32 prefix,
//        third, float64 shallow, deep, support, deep/shallow KL) and float64
//        gap[n_turns]; then int32 return codes of calls with bad arguments.
// Exit status 0 on success, 2 on a usage or file error, 3 when a call on
// valid arguments fails.
#include <stdio.h>
#include <stdlib.h>

#include <vector>

#include "turnkl.h"

namespace {

bool read_all(FILE* f, void* p, size_t n) { return fread(p, 1, n, f) == n; }

template <typename T>
void put(FILE* f, T v) { fwrite(&v, sizeof v, 1, f); }

}  // namespace

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 2;
  int32_t n_turns = 0, n_success = 0, floor_ = 0;
  int64_t n_traj = 0;
  double frac = 0.0;
  if (!read_all(in, &n_turns, 4) || !read_all(in, &n_success, 4) || !read_all(in, &n_traj, 8) ||
      !read_all(in, &floor_, 4) || !read_all(in, &frac, 8))
    return 2;
  if (n_turns < 1 || n_success < 0) return 2;
  std::vector<turnkl_turn_stat> stats(n_turns), ostats(2 * n_turns);
  std::vector<int32_t> lengths(n_success);
  if (!read_all(in, stats.data(), stats.size() * sizeof(turnkl_turn_stat)) ||
      !read_all(in, ostats.data(), ostats.size() * sizeof(turnkl_turn_stat)) ||
      !read_all(in, lengths.data(), lengths.size() * sizeof(int32_t)))
    return 2;
  fclose(in);
  FILE* out = fopen(argv[2], "wb");
  if (!out) return 2;

  turnkl_depth_config cfg;
  turnkl_depth_default_config(&cfg);
  turnkl_depth_state st;
  if (turnkl_depth_init(&cfg, &st) != TURNKL_OK) return 3;
  for (int64_t step = 1; step <= 24; ++step) {
    int32_t cap = 0, probe = 0, depth = 0;
    if (turnkl_depth_plan(&cfg, &st, step, &cap, &probe, &depth) != TURNKL_OK) return 3;
    if (probe && turnkl_depth_update(&cfg, &st, stats.data(), n_turns,
                                     n_success ? lengths.data() : nullptr, n_success) != TURNKL_OK)
      return 3;
    put(out, cap);
    put(out, probe);
    put(out, depth);
    put(out, st.h_bar);
    put(out, st.h_eff_bar);
    put(out, st.h_eff);
    put(out, st.h_cov);
    put(out, st.h_ctrl);
    put(out, st.n_probes);
  }
  std::vector<double> share(n_turns), gap(n_turns);
  if (turnkl_loss_share(stats.data(), n_turns, share.data()) != TURNKL_OK) return 3;
  turnkl_budget b;
  if (turnkl_budget_report(stats.data(), n_turns, n_traj, floor_, frac, &b) != TURNKL_OK) return 3;
  if (turnkl_outcome_gap(ostats.data(), n_turns, gap.data()) != TURNKL_OK) return 3;
  fwrite(share.data(), sizeof(double), share.size(), out);
  put(out, b.n_min);
  put(out, b.prefix);
  put(out, b.third);
  put(out, b.shallow_budget);
  put(out, b.deep_budget);
  put(out, b.deep_support);
  put(out, b.deep_shallow_kl);
  fwrite(gap.data(), sizeof(double), gap.size(), out);

  // argument errors: each must be refused without touching memory
  turnkl_depth_config bad = cfg;
  bad.h_max = 0;
  const int32_t bad_len = 0;
  const int32_t codes[] = {
      turnkl_depth_init(nullptr, &st),
      turnkl_depth_init(&bad, &st),
      turnkl_depth_plan(&cfg, &st, 0, nullptr, nullptr, nullptr),
      turnkl_depth_update(&cfg, &st, nullptr, n_turns, nullptr, 0),
      turnkl_depth_update(&cfg, &st, stats.data(), 0, nullptr, 0),
      turnkl_depth_update(&cfg, &st, stats.data(), n_turns, &bad_len, 1),
      turnkl_depth_update(&cfg, &st, stats.data(), n_turns, nullptr, 3),
      turnkl_loss_share(nullptr, n_turns, share.data()),
      turnkl_loss_share(stats.data(), 0, share.data()),
      turnkl_budget_report(stats.data(), n_turns, -1, floor_, frac, &b),
      turnkl_budget_report(stats.data(), n_turns, n_traj, -1, frac, &b),
      turnkl_budget_report(stats.data(), n_turns, n_traj, floor_, 1.5, &b),
      turnkl_outcome_gap(ostats.data(), 0, gap.data()),
      turnkl_outcome_gap(nullptr, n_turns, gap.data()),
  };
  for (int32_t c : codes) put(out, c);
  fclose(out);
  return 0;
}
