// Loss and per-turn-index statistics from the per-token KL.
//
// seg_moments  one workgroup per segment: n, sum, mean and m2 of the
//              segment's supervised KL (float64, fixed order), and the
//              segment's shares of L_blend = sum_i w_i KL_i (App. D,
//              Algorithm 1), L_traj (alpha = 0) and L_turn (alpha = 1).
// finalize     one workgroup per (group, turn index t): the segments of turn t
//              merged in a fixed order (each thread's segments s, s + 256, ...
//              in turn, then a fixed tree over the threads; pairwise update of
//              Chan, Golub & LeVeque for the mean and m2) -> pooled mean K_t (Sec. 4.3, Eq.
//              observed-turn-kl), population variance, survivors n_t (Sec.
//              5.1, App. D), loss mass (Sec. 4.4); optionally merged into the
//              caller's running statistics.  Group 0 takes every trajectory;
//              groups 1 and 2 the failed and the successful ones (Sec. 4.2:
//              K_t^fail, K_t^succ).  One more workgroup sums the loss shares.
//              No floating-point atomics: results are reproducible.

#include "block_ops.h"
#include "turnkl_internal.h"

namespace turnkl {
namespace {

constexpr int kMomThreads = 128;
constexpr int kFinThreads = 256;

__global__ __launch_bounds__(kMomThreads) void seg_moments(SegParams p, Ws ws, const float* kl,
                                                          double alpha) {
  __shared__ double s_red[kMomThreads / kWave];
  if (ws.hdr->err_key != kNoError) return;
  const int n_seg = ws.hdr->n_seg;
  const double b = (double)ws.hdr->b_eff;
  const int n_min = p.floor_on ? support_n_min(p, ws.hdr->b_eff) : 0;
  for (int s = blockIdx.x; s < n_seg; s += gridDim.x) {
    const int n = ws.seg_nsup[s];
    SegStat out{};
    if (n > 0) {
      const long long start = ws.seg_start[s];
      const long long end = start + ws.seg_len[s];
      double sum = 0.0;
      for (long long i = start + threadIdx.x; i < end; i += kMomThreads)
        if (p.mask[i]) sum += (double)kl[i];
      sum = block_sum<kMomThreads>(sum, s_red);
      const double mean = sum / (double)n;
      double m2 = 0.0;
      for (long long i = start + threadIdx.x; i < end; i += kMomThreads) {
        if (p.mask[i]) {
          const double d = (double)kl[i] - mean;
          m2 += d * d;
        }
      }
      m2 = block_sum<kMomThreads>(m2, s_red);
      const int h = ws.seg_head[s];
      const double n_b = (double)ws.traj_N[h];
      const TurnTerm u = turn_term(p, ws, s, h, n_min);
      const double w = ((1.0 - alpha) / n_b + turn_part(alpha, u, (double)n, n_b)) / b;
      out.sum = sum;
      out.mean = mean;
      out.m2 = m2;
      out.lm = w * sum;
      out.ltraj = sum / (b * n_b);
      if (u.t_v > 0.0) out.lturn = u.valid ? sum / (b * u.t_v * (double)n) : 0.0;
      else out.lturn = sum / (b * n_b);
      out.n = n;
    }
    if (threadIdx.x == 0) {
      ws.seg_stat[s] = out;
      drain_stores();
    }
  }
}

struct Moments {
  double n, mean, m2, lm;
  long long traj;
};

__device__ inline Moments merge(const Moments& x, const Moments& y) {
  Moments r;
  r.n = x.n + y.n;
  r.lm = x.lm + y.lm;
  r.traj = x.traj + y.traj;
  if (y.n == 0.0) {
    r.mean = x.mean;
    r.m2 = x.m2;
  } else if (x.n == 0.0) {
    r.mean = y.mean;
    r.m2 = y.m2;
  } else {
    const double d = y.mean - x.mean;
    r.mean = x.mean + d * (y.n / r.n);
    r.m2 = x.m2 + y.m2 + d * d * (x.n * y.n / r.n);
  }
  return r;
}

// Grid: 3 * max_turns + 1 workgroups (max_turns = 0 without statistics).
// Workgroup j < 3 * max_turns handles group j / max_turns at turn
// j % max_turns; the last one sums the losses.
__global__ __launch_bounds__(kFinThreads) void finalize(Ws ws, int max_turns, float* loss_out,
                                                       turnkl_turn_stat* stats,
                                                       turnkl_turn_stat* ostats,
                                                       const unsigned char* success,
                                                       int accumulate, int* status_out) {
  __shared__ Moments s_m[kFinThreads];
  __shared__ double s_l[3][kFinThreads];
  const unsigned long long key = ws.hdr->err_key;
  const bool bad = key != kNoError;
  const int n_seg = ws.hdr->n_seg;
  if ((int)blockIdx.x == 3 * max_turns) {  // the three losses (and the call's status)
    if (status_out && threadIdx.x == 0) *status_out = status_from_key(key);
    if (bad) {
      if (threadIdx.x < 3) loss_out[threadIdx.x] = __builtin_nanf("");
      return;
    }
    double lb = 0.0, lt = 0.0, lu = 0.0;
    for (int s = threadIdx.x; s < n_seg; s += kFinThreads) {
      lb += ws.seg_stat[s].lm;
      lt += ws.seg_stat[s].ltraj;
      lu += ws.seg_stat[s].lturn;
    }
    s_l[0][threadIdx.x] = lb;
    s_l[1][threadIdx.x] = lt;
    s_l[2][threadIdx.x] = lu;
    __syncthreads();
    for (int st = kFinThreads / 2; st > 0; st >>= 1) {
      if ((int)threadIdx.x < st) {
        s_l[0][threadIdx.x] += s_l[0][threadIdx.x + st];
        s_l[1][threadIdx.x] += s_l[1][threadIdx.x + st];
        s_l[2][threadIdx.x] += s_l[2][threadIdx.x + st];
      }
      __syncthreads();
    }
    if (threadIdx.x < 3) loss_out[threadIdx.x] = (float)s_l[threadIdx.x][0];
    return;
  }
  const int group = (int)blockIdx.x / max_turns;
  const int t = (int)blockIdx.x - group * max_turns;
  turnkl_turn_stat* out = group == 0 ? stats : ostats;
  if (bad || out == nullptr) return;
  if (group > 0) out += (group - 1) * max_turns;
  const bool want_success = group == 2;
  Moments acc{0.0, 0.0, 0.0, 0.0, 0};
  for (int s = threadIdx.x; s < n_seg; s += kFinThreads) {
    if (ws.seg_turn[s] != t) continue;
    if (group > 0 && (success[ws.seg_start[s]] != 0) != want_success) continue;
    const SegStat& g = ws.seg_stat[s];
    if (g.n == 0) continue;
    acc = merge(acc, Moments{(double)g.n, g.mean, g.m2, g.lm, 1});
  }
  s_m[threadIdx.x] = acc;
  __syncthreads();
  for (int st = kFinThreads / 2; st > 0; st >>= 1) {
    if ((int)threadIdx.x < st) s_m[threadIdx.x] = merge(s_m[threadIdx.x], s_m[threadIdx.x + st]);
    __syncthreads();
  }
  if (threadIdx.x != 0) return;
  Moments r = s_m[0];
  turnkl_turn_stat& o = out[t];
  if (accumulate && r.n == 0.0) return;  // nothing to merge at this turn
  if (accumulate) {
    const Moments old{(double)o.n_tokens, o.kl_mean, o.kl_m2, o.loss_mass, (long long)o.n_traj};
    r = merge(old, r);
  }
  // one 64-bit store per field (no multi-dword store data to protect), then
  // wait for them before the wave ends
  volatile long long* oi = reinterpret_cast<volatile long long*>(&o);
  volatile double* od = reinterpret_cast<volatile double*>(&o);
  oi[0] = (long long)r.n;
  oi[1] = r.traj;
  od[2] = r.n > 0 ? r.mean : 0.0;
  od[3] = r.n > 0 ? r.m2 : 0.0;
  od[4] = r.n > 0 ? r.m2 / r.n : 0.0;
  od[5] = r.lm;
  drain_stores();
}

}  // namespace

hipError_t launch_reduce(const SegParams& p, const Ws& ws, const float* kl, double alpha,
                         float* loss_out, turnkl_turn_stat* stats, turnkl_turn_stat* ostats,
                         int accumulate, int* status_out, hipStream_t s) {
  if (p.n > 0) {
    long long g = p.n < 4096 ? p.n : 4096;
    seg_moments<<<dim3((unsigned)g), dim3(kMomThreads), 0, s>>>(p, ws, kl, alpha);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  const int turns = (stats || ostats) ? p.max_turns : 0;
  finalize<<<dim3((unsigned)(3 * turns + 1)), dim3(kFinThreads), 0, s>>>(
      ws, turns, loss_out, stats, ostats, p.success, accumulate, status_out);
  return hipGetLastError();
}

}  // namespace turnkl
