// Top-K reverse KL: the teacher's top-K support S_i of each token, both
// distributions renormalised on it (the paper trains with a top-K reverse KL,
// App. D; Sec. 3, Eq. opd-rkl restricted to S_i):
//   p^_s(v) = exp(a_v) / sum_{u in S_i} exp(a_u),  p^_t likewise from the
//   teacher's values b_v on S_i,
//   KL_i = sum_{v in S_i} p^_s(v) d_v,  d_v = log p^_s(v) - log p^_t(v),
//   dKL_i/da_v = p^_s(v) (d_v - KL_i) on S_i, 0 elsewhere.
//
// topk_rows   one wave per token (four tokens per wave for K <= 64, their
//             loads issued together): gathers the K student logits at the
//             support ids (one scattered load per id), reduces max and sum
//             of both distributions with wave shuffles, writes KL_i and
//             grad_scale * w_i * dKL_i/da on the support to the stage (the
//             caller's sparse output, or the workspace);
// topk_fill   zero-fills the vocab columns of every dense gradient row with
//             16-byte streaming stores;
// topk_scatter  writes the staged support values of each supervised row.
//
// Order.  An out-of-place dense gradient is zero-filled first, and topk_rows
// then writes the support values into it directly (no scatter kernel, no
// staging round trip).  In place, topk_rows reads every student logit and
// stages the values, then the fill and the scatter overwrite the rows.

#include <hip/hip_bf16.h>

#include "block_ops.h"
#include "turnkl_internal.h"

// No implicit FMA contraction: identical student and teacher values must give
// bit-identical halves of each difference (exactly zero KL and gradient).
#pragma clang fp contract(off)

namespace turnkl {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

__device__ inline float load_logit(const void* base, long long i, bool bf16) {
  if (bf16) {
    const unsigned short u = static_cast<const unsigned short*>(base)[i];
    return __uint_as_float((unsigned)u << 16);
  }
  return static_cast<const float*>(base)[i];
}

__device__ inline float wave_max_f(float v) { return wave_max(v); }

// kPer support entries per lane (K <= 64 kPer); kRows rows per wave, their
// loads issued together (the kernel is bound by the latency of the id loads
// and the gathers that depend on them).  The scaled gradient on the support
// goes to the stage (when there is one) and, with p.direct, straight into a
// zero-filled, out-of-place dense gradient.
template <int kPer, int kRows>
__global__ __launch_bounds__(kThreads) void topk_rows(TopkParams p) {
  if (p.hdr->err_key != kNoError) return;
  const int lane = threadIdx.x & (kWave - 1);
  const long long wave0 = (long long)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;
  const long long stride = (long long)gridDim.x * kWavesPerBlock;
  for (long long r0 = wave0 * kRows; r0 < p.n_rows; r0 += stride * kRows) {
    bool sup[kRows], bad[kRows], on[kRows][kPer];
    int id[kRows][kPer];
    float a[kRows][kPer], b[kRows][kPer];
    // every load of the kRows rows first: masks, ids and teacher values ...
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const long long row = r0 + r;
      sup[r] = row < p.n_rows && p.mask[row];
      bad[r] = false;
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int j = lane + q * kWave;
        on[r][q] = sup[r] && j < p.k;
        id[r][q] = on[r][q] ? p.ids[row * p.ld_k + j] : 0;
        b[r][q] = on[r][q] ? p.vals[row * p.ld_k + j] : -INFINITY;
      }
    }
    // ... then the student logits at the support ids
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const bool in = id[r][q] >= 0 && id[r][q] < p.vocab;
        bad[r] = bad[r] || (on[r][q] && !in);
        on[r][q] = on[r][q] && in;
        a[r][q] = on[r][q] ? load_logit(p.zs, (r0 + r) * p.ld_s + id[r][q], p.bf16) : -INFINITY;
        b[r][q] = on[r][q] ? b[r][q] : -INFINITY;
      }
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const long long row = r0 + r;
      if (row >= p.n_rows) break;
      float* stage = p.stage ? p.stage + row * p.ld_stage : nullptr;
      if (!sup[r]) {
        if (stage && p.zero_masked_stage)
          for (int j = lane; j < p.k; j += kWave) stage[j] = 0.0f;
        if (p.lse && lane == 0) {  // the row is not read: no log-partition function
          p.lse[2 * row] = __builtin_nanf("");
          p.lse[2 * row + 1] = __builtin_nanf("");
        }
        continue;
      }
      if (__ballot(bad[r]) != 0ull) {
        if (lane == 0) atomicMin(&p.hdr->err_key, err_key(row, kPrioTopkId));
        continue;
      }
      float ma = -INFINITY, mb = -INFINITY;
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        ma = fmaxf(ma, a[r][q]);
        mb = fmaxf(mb, b[r][q]);
      }
      ma = wave_max_f(ma);
      mb = wave_max_f(mb);
      float sa = 0.0f, sb = 0.0f;
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        sa += on[r][q] ? expf(a[r][q] - ma) : 0.0f;
        sb += on[r][q] ? expf(b[r][q] - mb) : 0.0f;
      }
      sa = wave_sum(sa);
      sb = wave_sum(sb);
      const float la = logf(sa);
      const float lb = logf(sb);
      float d[kPer], pr[kPer];
      float kl = 0.0f;
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const float xa = a[r][q] - ma;
        d[q] = on[r][q] ? ((xa - (b[r][q] - mb)) - (la - lb)) : 0.0f;
        pr[q] = on[r][q] ? expf(xa - la) : 0.0f;
        kl = fmaf(pr[q], d[q], kl);
      }
      kl = wave_sum(kl);
      const float sc = p.wsc[row];
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int j = lane + q * kWave;
        if (j >= p.k) continue;
        const float g = sc * (pr[q] * (d[q] - kl));
        if (stage) stage[j] = g;
        if (p.direct && on[r][q]) {
          if (p.bf16) {
            reinterpret_cast<__hip_bfloat16*>(p.grad)[row * p.ld_g + id[r][q]] = __float2bfloat16(g);
          } else {
            reinterpret_cast<float*>(p.grad)[row * p.ld_g + id[r][q]] = g;
          }
        }
      }
      if (lane == 0) {
        p.kl[row] = kl;
        if (p.lse) {  // log sum exp over the support = max + ln(sum)
          p.lse[2 * row] = ma + la;
          p.lse[2 * row + 1] = mb + lb;
        }
      }
    }
  }
}

// Zero-fill of the dense gradient rows (grid-stride over rows): a plain
// streaming store of vocab columns per row.  kVec: the row starts are 16-byte
// aligned and V is a whole number of 16-byte packs, so the fill uses 16-byte
// stores.
template <bool kBf16, bool kVec>
__global__ __launch_bounds__(kThreads) void topk_fill(TopkParams p) {
  if (p.hdr->err_key != kNoError) return;
  constexpr int kEs = kBf16 ? 2 : 4;
  constexpr int kEpv = 16 / kEs;
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  for (long long row = blockIdx.x; row < p.n_rows; row += gridDim.x) {
    char* g = static_cast<char*>(p.grad) + row * p.ld_g * kEs;
    if (kVec) {
      const long long packs = p.vocab / kEpv;
      const auto rsrc = __builtin_amdgcn_make_buffer_rsrc(g, 0, 0x7FFFFFFF, 0x00020000);
      const u32x4 z = {0u, 0u, 0u, 0u};
      for (long long v = threadIdx.x; v < packs; v += kThreads)
        __builtin_amdgcn_raw_buffer_store_b128(z, rsrc, (int)(v * 16), 0, 2 /* nt */);
    } else {
      for (long long v = threadIdx.x; v < p.vocab; v += kThreads) {
        if (kBf16) reinterpret_cast<unsigned short*>(g)[v] = 0;
        else reinterpret_cast<float*>(g)[v] = 0.0f;
      }
    }
  }
  drain_stores();
}

// Zero-fill of a dense gradient whose rows are contiguous (ld == vocab): one
// flat region of n_rows * vocab elements, 16-byte streaming stores over a
// grid-stride loop (the fastest write pattern measured on the device).
__global__ __launch_bounds__(kThreads) void topk_fill_flat(TopkParams p, long long n_packs) {
  if (p.hdr->err_key != kNoError) return;
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  u32x4* g = static_cast<u32x4*>(p.grad);
  const u32x4 z = {0u, 0u, 0u, 0u};
  for (long long i = (long long)blockIdx.x * kThreads + threadIdx.x; i < n_packs;
       i += (long long)gridDim.x * kThreads)
    __builtin_nontemporal_store(z, g + i);
  drain_stores();
}

// Scatter of the staged support values into the zero-filled rows of
// supervised tokens (in place: the rows were read before the fill), kRows
// rows per wave with their loads issued together; runs after topk_fill on
// the stream.
template <bool kBf16, int kRows>
__global__ __launch_bounds__(kThreads) void topk_scatter(TopkParams p) {
  if (p.hdr->err_key != kNoError) return;
  const int lane = threadIdx.x & (kWave - 1);
  const long long wave0 = (long long)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;
  const long long stride = (long long)gridDim.x * kWavesPerBlock;
  for (long long r0 = wave0 * kRows; r0 < p.n_rows; r0 += stride * kRows) {
    for (int j0 = 0; j0 < p.k; j0 += kWave) {
      const int j = j0 + lane;
      bool on[kRows];
      int id[kRows];
      float x[kRows];
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        const long long row = r0 + r;
        on[r] = row < p.n_rows && j < p.k && p.mask[row];
        id[r] = on[r] ? p.ids[row * p.ld_k + j] : 0;
        x[r] = on[r] ? p.stage[row * p.ld_stage + j] : 0.0f;
      }
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        if (!on[r] || id[r] < 0 || id[r] >= p.vocab) continue;  // bad ids: reported by topk_rows
        const long long at = (r0 + r) * p.ld_g + id[r];
        if (kBf16) reinterpret_cast<__hip_bfloat16*>(p.grad)[at] = __float2bfloat16(x[r]);
        else reinterpret_cast<float*>(p.grad)[at] = x[r];
      }
    }
  }
  drain_stores();
}

int grid_for(long long items, int per_block, int cap) {
  long long g = (items + per_block - 1) / per_block;
  if (g < 1) g = 1;
  return (int)(g < cap ? g : cap);
}

void launch_fill_rows(const TopkParams& p, bool vec, hipStream_t s) {
  const int fill_grid = grid_for(p.n_rows, 1, 32768);
  if (p.bf16) {
    if (vec) topk_fill<true, true><<<fill_grid, kThreads, 0, s>>>(p);
    else topk_fill<true, false><<<fill_grid, kThreads, 0, s>>>(p);
  } else {
    if (vec) topk_fill<false, true><<<fill_grid, kThreads, 0, s>>>(p);
    else topk_fill<false, false><<<fill_grid, kThreads, 0, s>>>(p);
  }
}

}  // namespace

// Rows per wave of topk_rows and topk_scatter: four for a support of at
// most 64 ids (one per lane), two up to 128, one beyond.
constexpr int rows_per_wave(int per) { return per <= 1 ? 4 : per <= 2 ? 2 : 1; }

hipError_t launch_topk_rows(const TopkParams& p, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  const int per = (p.k + kWave - 1) / kWave;
#define TURNKL_TOPK(n)                                                                     \
  case n:                                                                                  \
    topk_rows<n, rows_per_wave(n)>                                                         \
        <<<grid_for(p.n_rows, kWavesPerBlock * rows_per_wave(n), 16384), kThreads, 0, s>>>(p); \
    break;
  switch (per <= 1 ? 1 : per <= 2 ? 2 : per <= 4 ? 4 : per <= 8 ? 8 : 16) {
    TURNKL_TOPK(1) TURNKL_TOPK(2) TURNKL_TOPK(4) TURNKL_TOPK(8) TURNKL_TOPK(16)
    default: return hipErrorInvalidValue;
  }
#undef TURNKL_TOPK
  return hipGetLastError();
}

hipError_t launch_topk_fill(const TopkParams& p, hipStream_t s) {
  if (p.n_rows == 0 || !p.grad) return hipSuccess;
  const int es = p.bf16 ? 2 : 4;
  const bool vec = ((uintptr_t)p.grad % 16 == 0) && (p.ld_g * es) % 16 == 0 && (p.vocab * es) % 16 == 0;
  if (vec && p.ld_g == p.vocab) {
    const long long packs = (long long)p.n_rows * p.vocab * es / 16;
    topk_fill_flat<<<grid_for(packs, kThreads, 32768), kThreads, 0, s>>>(p, packs);
  } else {
    launch_fill_rows(p, vec, s);
  }
  return hipGetLastError();
}

hipError_t launch_topk_scatter(const TopkParams& p, hipStream_t s) {
  if (p.n_rows == 0 || !p.grad) return hipSuccess;
  constexpr int kRows = 4;
  const int grid = grid_for(p.n_rows, kWavesPerBlock * kRows, 16384);
  if (p.bf16) topk_scatter<true, kRows><<<grid, kThreads, 0, s>>>(p);
  else topk_scatter<false, kRows><<<grid, kThreads, 0, s>>>(p);
  return hipGetLastError();
}

}  // namespace turnkl
