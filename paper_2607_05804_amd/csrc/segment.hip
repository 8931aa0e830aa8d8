// Segment table, validation and token weights.
//
// A segment is a maximal run of consecutive tokens with equal (trajectory id,
// turn id): turn t of a trace is its observation o_t followed by the response
// r_t (Sec. 3), and the segment's supervised count is the paper's n_t for
// that trajectory (Sec. 4.4).  The per-token weights follow the progressive
// turn-normalised blend of Sec. 5.2 / App. D Algorithm 1 expanded per token:
//   w_i = m_i / B * ((1 - alpha) / N_b + alpha / (T_b * n_bt)).
//
// Kernels, in launch order (all integer work is exact, so the table is unique):
//   seg_count   per 1024-token tile: segment starts and the earliest id/mask
//               error of the tile; clears the per-segment counters; the first
//               workgroup resets the workspace header.
//   seg_offsets (batches of more than kFusedScanTiles tiles only) one
//               workgroup: exclusive scan of the tile counts, error key and
//               segment count of the whole batch.
//   seg_write   per tile: its first segment index (the sum of the earlier
//               tiles' counts, summed by every workgroup itself up to
//               kFusedScanTiles tiles), segment index of every token, segment
//               start / turn / trajectory / end, supervised counts (summed
//               per segment in LDS, one global atomic per tile and segment);
//               the first workgroup writes the batch's error key and segment
//               count.
//   seg_link    per segment: ordering check against the previous segment,
//               outcome-flag check against the trajectory's first segment,
//               segment length, trajectory head segment, T_b, N_b and B (the
//               segments of a wave summed per trajectory before the atomics),
//               the batch's supervised-token count, and the survivors n_t of
//               the turn-support floor.
//   seg_valid   (turn-support floor only) per segment: T_vb, the valid
//               supervised turns of each trajectory (n_t >= n_min).
//   token_weights per token: w_i and grad_scale * w_i, clears this call's
//               per-token KL and the row kernel's exchange slots.
//
// With the floor (App. D's internal-blend n_min = max(min_floor,
// ceil(min_frac * B)); the turn term covers only valid turns) the weight is
//   w_i = m_i / B * ((1 - alpha) / N_b + alpha * u_bt),
//   u_bt = [n_t >= n_min] / (T_vb * n_bt) if T_vb > 0, else 1 / N_b.

#include "block_ops.h"
#include "turnkl_internal.h"

namespace turnkl {
namespace {

struct TokenInfo {
  bool pad;
  bool start;
  unsigned long long err;
};

__device__ inline TokenInfo inspect(const SegParams& p, long long i) {
  TokenInfo r{true, false, kNoError};
  const int b = p.traj[i];
  const int t = p.turn[i];
  if (b < 0) {
    if (p.mask[i]) r.err = err_key(i, kPrioPadMask);
    return r;
  }
  r.pad = false;
  if (t < 0 || t >= p.max_turns) r.err = err_key(i, kPrioTurnRange);
  r.start = (i == 0) || p.traj[i - 1] != b || p.turn[i - 1] != t;
  // inside a segment the outcome flag must not change (segment starts are
  // checked against the trajectory's first segment in seg_link)
  if (p.success && !r.start && r.err == kNoError &&
      ((p.success[i] != 0) != (p.success[i - 1] != 0)))
    r.err = err_key(i, kPrioOutcome);
  return r;
}

__global__ __launch_bounds__(kSegThreads) void seg_count(SegParams p, Ws ws, int n_surv) {
  __shared__ int s_cnt[kSegThreads / kWave];
  __shared__ unsigned long long s_err[kSegThreads / kWave];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    volatile Header* h = ws.hdr;
    h->err_key = kNoError;
    h->ticket = 0u;
    h->n_seg = 0;
    h->b_eff = 0;
    h->n_sup = 0;
  }
  for (int t = blockIdx.x * kSegThreads + threadIdx.x; t < n_surv; t += gridDim.x * kSegThreads)
    ws.turn_surv[t] = 0;
  const long long base = (long long)blockIdx.x * kSegTile + (long long)threadIdx.x * kSegTokensPerThread;
  int cnt = 0;
  unsigned long long err = kNoError;
  for (int j = 0; j < kSegTokensPerThread; ++j) {
    const long long i = base + j;
    if (i >= p.n) break;
    const TokenInfo ti = inspect(p, i);
    cnt += ti.start ? 1 : 0;
    err = ti.err < err ? ti.err : err;
    ws.seg_nsup[i] = 0;
    ws.traj_T[i] = 0;
    ws.traj_N[i] = 0;
    ws.traj_Tv[i] = 0;
  }
  cnt = wave_sum(cnt);
  err = wave_min_u64(err);
  const int wid = threadIdx.x / kWave;
  if ((threadIdx.x & (kWave - 1)) == 0) {
    s_cnt[wid] = cnt;
    s_err[wid] = err;
  }
  __syncthreads();
  if (threadIdx.x == 0 && (long long)blockIdx.x * kSegTile < p.n) {
    int c = 0;
    unsigned long long e = kNoError;
    for (int w = 0; w < kSegThreads / kWave; ++w) {
      c += s_cnt[w];
      e = s_err[w] < e ? s_err[w] : e;
    }
    ws.blk_cnt[blockIdx.x] = c;
    ws.blk_err[blockIdx.x] = e;
  }
}

constexpr int kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void seg_offsets(Ws ws, long long nblk) {
  __shared__ int s_scan[kScanThreads / kWave];
  __shared__ unsigned long long s_err[kScanThreads / kWave];
  int carry = 0;
  unsigned long long err = kNoError;
  for (long long b0 = 0; b0 < nblk; b0 += kScanThreads) {
    const long long b = b0 + threadIdx.x;
    const int v = b < nblk ? ws.blk_cnt[b] : 0;
    if (b < nblk) err = ws.blk_err[b] < err ? ws.blk_err[b] : err;
    int total;
    const int ex = block_exclusive_scan<kScanThreads>(v, s_scan, &total);
    if (b < nblk) ws.blk_off[b] = carry + ex;
    carry += total;
  }
  err = wave_min_u64(err);
  if ((threadIdx.x & (kWave - 1)) == 0) s_err[threadIdx.x / kWave] = err;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long e = kNoError;
    for (int w = 0; w < kScanThreads / kWave; ++w) e = s_err[w] < e ? s_err[w] : e;
    volatile Header* h = ws.hdr;
    h->err_key = e;
    h->n_seg = carry;
  }
  drain_stores();
}

// The number of tiles up to which every seg_write workgroup sums the earlier
// tiles' segment counts itself (at most 8 loads per thread), which saves the
// separate scan kernel; larger batches run seg_offsets first.
constexpr long long kFusedScanTiles = 2048;

template <bool kFusedScan>
__global__ __launch_bounds__(kSegThreads) void seg_write(SegParams p, Ws ws, long long nblk) {
  __shared__ int s_scan[kSegThreads / kWave];
  __shared__ unsigned long long s_err[kSegThreads / kWave];
  __shared__ int s_nsup[kSegTile + 1];  // supervised tokens per segment of this tile
  const long long base = (long long)blockIdx.x * kSegTile + (long long)threadIdx.x * kSegTokensPerThread;
  int first;  // segment index of this tile's tokens before its first segment start
  if (kFusedScan) {
    // the earlier tiles' counts, summed in a fixed order (integers: exact);
    // the first workgroup also takes the batch's totals
    const long long upto = blockIdx.x == 0 ? nblk : (long long)blockIdx.x;
    int c = 0, before = 0;
    unsigned long long e = kNoError;
    for (long long b = threadIdx.x; b < upto; b += kSegThreads) {
      const int v = ws.blk_cnt[b];
      c += v;
      before += b < (long long)blockIdx.x ? v : 0;
      if (blockIdx.x == 0) e = ws.blk_err[b] < e ? ws.blk_err[b] : e;
    }
    before = block_sum<kSegThreads>(before, s_scan);
    if (blockIdx.x == 0) {
      c = block_sum<kSegThreads>(c, s_scan);
      e = wave_min_u64(e);
      if ((threadIdx.x & (kWave - 1)) == 0) s_err[threadIdx.x / kWave] = e;
      __syncthreads();
      if (threadIdx.x == 0) {
        for (int w = 0; w < kSegThreads / kWave; ++w) e = s_err[w] < e ? s_err[w] : e;
        volatile Header* h = ws.hdr;
        h->err_key = e;
        h->n_seg = c;
      }
    }
    first = before - 1;
  } else {
    first = ws.blk_off[blockIdx.x] - 1;
  }
  for (int k = threadIdx.x; k <= kSegTile; k += kSegThreads) s_nsup[k] = 0;
  TokenInfo ti[kSegTokensPerThread];
  int cnt = 0;
  for (int j = 0; j < kSegTokensPerThread; ++j) {
    const long long i = base + j;
    ti[j] = TokenInfo{true, false, kNoError};
    if (i < p.n) ti[j] = inspect(p, i);
    cnt += ti[j].start ? 1 : 0;
  }
  int total;
  int seg = first + block_exclusive_scan<kSegThreads>(cnt, s_scan, &total);
  // this thread's supervised tokens, counted per segment before the LDS add
  int run_seg = -1, run_n = 0;
  for (int j = 0; j < kSegTokensPerThread; ++j) {
    const long long i = base + j;
    if (i >= p.n) break;
    if (ti[j].pad) {
      ws.tok_seg[i] = -1;
      continue;
    }
    if (ti[j].start) {
      ++seg;
      ws.seg_start[seg] = (int)i;
      ws.seg_traj[seg] = p.traj[i];
      ws.seg_turn[seg] = p.turn[i];
    }
    ws.tok_seg[i] = seg;
    const bool last = (i + 1 == p.n) || p.traj[i + 1] != p.traj[i] || p.turn[i + 1] != p.turn[i];
    if (last) ws.seg_len[seg] = (int)(i + 1);  // segment end; seg_link turns it into a length
    if (p.mask[i]) {
      if (seg != run_seg) {
        if (run_n) atomicAdd(&s_nsup[run_seg - first], run_n);
        run_seg = seg;
        run_n = 0;
      }
      ++run_n;
    }
  }
  if (run_n) atomicAdd(&s_nsup[run_seg - first], run_n);
  __syncthreads();
  for (int k = threadIdx.x; k <= total; k += kSegThreads)
    if (const int n = s_nsup[k]) atomicAdd(&ws.seg_nsup[first + k], n);
}

__global__ __launch_bounds__(kSegThreads) void seg_link(SegParams p, Ws ws) {
  __shared__ int s_red[kSegThreads / kWave];
  const int n_seg = ws.hdr->n_seg;
  const int lane = threadIdx.x & (kWave - 1);
  int sup_total = 0;
  // every lane of a wave runs the same iterations (the per-trajectory sums
  // below are wave-wide)
  for (int s0 = blockIdx.x * kSegThreads; s0 < n_seg; s0 += gridDim.x * kSegThreads) {
    const int s = s0 + (int)threadIdx.x;
    int head = -1, n = 0;
    if (s < n_seg) {
      const int b = ws.seg_traj[s];
      const int t = ws.seg_turn[s];
      const int start = ws.seg_start[s];
      if (s > 0) {
        const int pb = ws.seg_traj[s - 1];
        const int pt = ws.seg_turn[s - 1];
        if (b < pb || (b == pb && t <= pt)) atomicMin(&ws.hdr->err_key, err_key(start, kPrioUnsorted));
      }
      ws.seg_len[s] = ws.seg_len[s] - start;
      // first segment of this trajectory (ids are sorted when the batch is valid)
      int lo = 0, hi = s;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (ws.seg_traj[mid] < b) lo = mid + 1; else hi = mid;
      }
      head = lo;
      ws.seg_head[s] = head;
      // On a sorted prefix `head` is the trajectory's first segment; otherwise
      // an ordering error at or before this segment's start outranks this one.
      if (p.success && head != s && (p.success[start] != 0) != (p.success[ws.seg_start[head]] != 0))
        atomicMin(&ws.hdr->err_key, err_key(start, kPrioOutcome));
      n = ws.seg_nsup[s];
      if (n > 0 && p.floor_on && t >= 0 && t < p.max_turns) atomicAdd(&ws.turn_surv[t], 1);
    }
    sup_total += n;
    // T_b and N_b: the wave's supervised segments summed per trajectory head,
    // one atomic pair per head; the add that lifts N_b from zero counts the
    // trajectory in B
    unsigned long long todo = __ballot(n > 0);
    while (todo) {
      const int leader = __builtin_ctzll(todo);
      const int h = __shfl(head, leader, kWave);
      const unsigned long long same = __ballot(n > 0 && head == h);
      const int sum_n = wave_sum((same >> lane) & 1ull ? n : 0);
      if (lane == leader) {
        atomicAdd(&ws.traj_T[h], __popcll(same));
        if (atomicAdd(&ws.traj_N[h], sum_n) == 0) atomicAdd(&ws.hdr->b_eff, 1);
      }
      todo &= ~same;
    }
  }
  sup_total = block_sum<kSegThreads>(sup_total, s_red);
  if (threadIdx.x == 0 && sup_total) atomicAdd(&ws.hdr->n_sup, sup_total);
}

__global__ __launch_bounds__(kSegThreads) void seg_valid(SegParams p, Ws ws) {
  if (ws.hdr->err_key != kNoError) return;
  const int n_seg = ws.hdr->n_seg;
  const int n_min = support_n_min(p, ws.hdr->b_eff);
  for (int s = blockIdx.x * kSegThreads + threadIdx.x; s < n_seg; s += gridDim.x * kSegThreads) {
    if (ws.seg_nsup[s] > 0 && ws.turn_surv[ws.seg_turn[s]] >= n_min)
      atomicAdd(&ws.traj_Tv[ws.seg_head[s]], 1);
  }
}

__global__ __launch_bounds__(kSegThreads) void token_weights(SegParams p, Ws ws, double alpha,
                                                             float grad_scale, int slot_words,
                                                             float* kl) {
  if (ws.hdr->err_key != kNoError) return;
  const double inv_b = ws.hdr->b_eff > 0 ? 1.0 / (double)ws.hdr->b_eff : 0.0;
  const int n_min = p.floor_on ? support_n_min(p, ws.hdr->b_eff) : 0;
  for (long long i = (long long)blockIdx.x * kSegThreads + threadIdx.x; i < p.n;
       i += (long long)gridDim.x * kSegThreads) {
    kl[i] = 0.0f;
    if (!p.mask[i]) {
      ws.w[i] = 0.0f;
      ws.wsc[i] = 0.0f;
      continue;
    }
    const int s = ws.tok_seg[i];
    const int h = ws.seg_head[s];
    const double n_bt = (double)ws.seg_nsup[s];
    const double n_b = (double)ws.traj_N[h];
    const TurnTerm u = turn_term(p, ws, s, h, n_min);
    const double w = inv_b * ((1.0 - alpha) / n_b + turn_part(alpha, u, n_bt, n_b));
    ws.w[i] = (float)w;
    ws.wsc[i] = (float)(w * (double)grad_scale);
    if (slot_words) {
      unsigned long long* sl = ws.slots + i * (long long)slot_words;
      for (int q = 0; q < slot_words; ++q) sl[q] = 0ull;
      drain_stores();
    }
  }
}

int grid_for(long long items, int per_block, int cap) {
  long long g = (items + per_block - 1) / per_block;
  if (g < 1) g = 1;
  return (int)(g < cap ? g : cap);
}

}  // namespace

hipError_t launch_segments(const SegParams& p, const Ws& ws, long long nblk, hipStream_t s) {
  const int n_surv = p.floor_on ? p.max_turns : 0;
  seg_count<<<dim3((unsigned)(nblk > 0 ? nblk : 1)), dim3(kSegThreads), 0, s>>>(p, ws, n_surv);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (nblk == 0) return hipSuccess;
  if (nblk <= kFusedScanTiles) {
    seg_write<true><<<dim3((unsigned)nblk), dim3(kSegThreads), 0, s>>>(p, ws, nblk);
  } else {
    seg_offsets<<<1, kScanThreads, 0, s>>>(ws, nblk);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    seg_write<false><<<dim3((unsigned)nblk), dim3(kSegThreads), 0, s>>>(p, ws, nblk);
  }
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  seg_link<<<grid_for(p.n, kSegThreads, 1024), kSegThreads, 0, s>>>(p, ws);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (!p.floor_on) return hipSuccess;
  seg_valid<<<grid_for(p.n, kSegThreads, 1024), kSegThreads, 0, s>>>(p, ws);
  return hipGetLastError();
}

hipError_t launch_weights(const SegParams& p, const Ws& ws, double alpha, float grad_scale,
                          int n_chunks, float* kl, hipStream_t s) {
  if (p.n == 0) return hipSuccess;
  const int slot_words = n_chunks > 1 ? n_chunks * kExchangeWords : 0;
  token_weights<<<grid_for(p.n, kSegThreads, 4096), kSegThreads, 0, s>>>(p, ws, alpha, grad_scale,
                                                                         slot_words, kl);
  return hipGetLastError();
}

}  // namespace turnkl
