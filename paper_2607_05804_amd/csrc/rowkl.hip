// Row kernel: per-token reverse KL over the full vocabulary and its gradient
// with respect to the student logits, fused in one read of each logit.
//
// Math (Sec. 3, Eq. opd-rkl; teacher frozen; temperature 1).  For a row with
// student logits a and teacher logits b:
//   p_s = softmax(a),  mu = <p_s, a - b>,  lse = log sum exp
//   KL  = mu - lse(a) + lse(b)
//   dKL/da_v = p_s(v) (log p_s(v) - log p_t(v) - KL) = p_s(v) ((a_v - b_v) - mu)
// so the gradient needs only lse(a) and mu, and the loss needs lse(b) too.
// All exponentials are base 2 (v_exp_f32): a chunk keeps, in log2 units,
//   M_s = max(a) log2(e),  S_s = sum 2^(a log2(e) - M_s),  A = sum 2^(...) (a - b),
//   M_t = max(b) log2(e),  S_t = sum 2^(b log2(e) - M_t).
//
// Work decomposition.  A row of V elements (V / epv packs of 16 bytes) is cut
// into n_chunks chunks whose boundaries chunk_start places on 1 KiB (or
// 128-byte) multiples from the row start when the host's tiling allows, else
// balanced; each of a workgroup's 256 threads holds up to vpt packs.  One
// workgroup owns one (row, chunk) task: it loads its chunk of both rows into
// registers, reduces the chunk's partials, publishes them as seven tagged
// 64-bit words (see the row merge below), reads its row mates' words, merges
// all chunks in chunk order (so every workgroup of the row computes
// bit-identical row scalars), and writes its chunk of the gradient straight
// from registers.  Every logit is read from HBM exactly once and every
// gradient element written once: 3 V s bytes per supervised row, V s per
// unsupervised row (zeros only).
//
// Scheduling.  A wave's priority rises with its task's progress (loads,
// partial sums, stores), and the bf16 kernel comes in two load orders, one
// of which each call runs (both explained where they are set).
//
// Tasks are handed out by an atomic ticket in row-major order, so a
// workgroup only ever waits for tasks that running workgroups already hold
// or that the next free workgroup will take; the wait is bounded and reports
// TURNKL_ERR_SYNC_TIMEOUT instead of hanging.  An in-place gradient is safe
// because each workgroup reads its chunk completely before writing it, and
// chunks do not overlap.

#include <hip/hip_bf16.h>

#include "block_ops.h"
#include "turnkl_internal.h"

// No implicit FMA contraction in this file: every fused multiply-add the
// kernel wants is written as fmaf.  Contraction would evaluate the student
// and teacher halves of a difference asymmetrically (x*c - y*c becoming
// fma(x, c, -(y*c)) leaves the rounding error of y*c when x == y), so
// identical logits would no longer give exactly zero KL and gradient.
#pragma clang fp contract(off)

namespace turnkl {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr int kRowWaves = kRowThreads / kWave;
// Reference magnitude (log2 units, i.e. logits times log2 e) above which a
// chunk, and then its row, subtracts its references per element.  Below it
// the fast path's error term, a few u |m_s - m_t|, stays under 1e-5.
constexpr float kFar2 = 64.0f * kLog2e;

// ---------------------------------------------------------------------------
// packs of kEpv elements moved with one load/store

// Buffer resource over one row chunk (gfx9 dword-3 word for raw dword
// access).  The base is wave-uniform, so each pack's offset splits into a
// per-lane VGPR part and a compile-time SGPR step.
constexpr int kRsrcWord3 = 0x00020000;

// Cache policy of the logit loads and gradient stores: non-temporal (the nt
// bit of gfx940-family buffer instructions).  Every logit is read once and
// every gradient element written once, so nothing is gained by keeping them
// in L2; streaming them measured about 3% faster than the default policy.
constexpr int kStream = 2;

__device__ inline __amdgpu_buffer_rsrc_t chunk_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7FFFFFFF, kRsrcWord3);
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// Store data must stay untouched for a while after a 16-byte store is
// issued: on gfx950 the store can read its data registers later than the
// compiler's wait states assume, so a register reused right after the store
// (observed: the first data dword) lands in memory.  The row kernel pins each
// store in program order and keeps its data live (keep_alive) across the next
// pack's work, or across the end-of-task barrier for the last pack.
__device__ inline void keep_alive(const u32x4& x) { asm volatile("" ::"v"(x)); }
__device__ inline void keep_alive(unsigned x) { asm volatile("" ::"v"(x)); }

template <bool kBf16, int kEpv>
struct Pack;

template <>
struct Pack<true, 8> {  // 8 bf16 = 16 bytes
  using Data = u32x4;
  unsigned w[4];
  __device__ void load(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    const auto u = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kStream);
    w[0] = u[0]; w[1] = u[1]; w[2] = u[2]; w[3] = u[3];
  }
  // Opaque to the optimiser: values unpacked before the fence cannot be
  // reused after it, so only the packed words stay live between passes.
  __device__ void fence() { asm volatile("" : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3])); }
  __device__ float get(int j) const {
    const unsigned x = w[j >> 1];
    return __uint_as_float((j & 1) ? (x & 0xFFFF0000u) : (x << 16));
  }
  // Round to bf16 (nearest even, v_cvt_pk_bf16_f32); flip = 0x80008000
  // negates both halves of every word.
  __device__ static Data encode(const float (&g)[8], unsigned flip) {
    Data o;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const f32x2 x = {g[2 * k], g[2 * k + 1]};
      o[k] = __builtin_bit_cast(unsigned, __builtin_convertvector(x, bf16x2)) ^ flip;
    }
    return o;
  }
  __device__ static Data zero() { return Data{0u, 0u, 0u, 0u}; }
  __device__ static void store(__amdgpu_buffer_rsrc_t r, int voff, int soff, const Data& o) {
    __builtin_amdgcn_raw_buffer_store_b128(o, r, voff, soff, kStream);
  }
};

template <>
struct Pack<false, 4> {  // 4 fp32 = 16 bytes
  using Data = u32x4;
  float f[4];
  __device__ void load(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    const auto u = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, kStream);
    f[0] = __uint_as_float(u[0]); f[1] = __uint_as_float(u[1]);
    f[2] = __uint_as_float(u[2]); f[3] = __uint_as_float(u[3]);
  }
  __device__ void fence() { asm volatile("" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3])); }
  __device__ float get(int j) const { return f[j]; }
  __device__ static Data encode(const float (&g)[4], unsigned flip) {
    const unsigned fl = flip << 16;  // sign bit of an fp32
    Data o;
#pragma unroll
    for (int k = 0; k < 4; ++k) o[k] = __float_as_uint(g[k]) ^ fl;
    return o;
  }
  __device__ static Data zero() { return Data{0u, 0u, 0u, 0u}; }
  __device__ static void store(__amdgpu_buffer_rsrc_t r, int voff, int soff, const Data& o) {
    __builtin_amdgcn_raw_buffer_store_b128(o, r, voff, soff, kStream);
  }
};

template <>
struct Pack<true, 1> {  // one bf16
  using Data = unsigned;
  unsigned w;
  __device__ void load(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    w = __builtin_amdgcn_raw_buffer_load_b16(r, voff, soff, kStream);
  }
  __device__ void fence() { asm volatile("" : "+v"(w)); }
  __device__ float get(int) const { return __uint_as_float(w << 16); }
  __device__ static Data encode(const float (&g)[1], unsigned flip) {
    const f32x2 x = {g[0], 0.0f};
    return (__builtin_bit_cast(unsigned, __builtin_convertvector(x, bf16x2)) ^ flip) & 0xFFFFu;
  }
  __device__ static Data zero() { return 0u; }
  __device__ static void store(__amdgpu_buffer_rsrc_t r, int voff, int soff, const Data& o) {
    __builtin_amdgcn_raw_buffer_store_b16((unsigned short)o, r, voff, soff, kStream);
  }
};

template <>
struct Pack<false, 1> {  // one fp32
  using Data = unsigned;
  float f;
  __device__ void load(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    f = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, kStream));
  }
  __device__ void fence() { asm volatile("" : "+v"(f)); }
  __device__ float get(int) const { return f; }
  __device__ static Data encode(const float (&g)[1], unsigned flip) {
    return __float_as_uint(g[0]) ^ (flip << 16);
  }
  __device__ static Data zero() { return 0u; }
  __device__ static void store(__amdgpu_buffer_rsrc_t r, int voff, int soff, const Data& o) {
    __builtin_amdgcn_raw_buffer_store_b32(o, r, voff, soff, kStream);
  }
};

__device__ inline float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Take a ticket: an atomic increment, which the compiler issues as one plain
// global atomic whose result is waited for only where it is used (an atomic
// add from one lane is rewritten into a wave-aggregated form that waits at
// once).
__device__ inline unsigned take_ticket(unsigned* counter) {
  return __builtin_amdgcn_atomic_inc32(counter, 0xFFFFFFFFu, __ATOMIC_RELAXED, "agent");
}

// Exchange words.  A chunk's seven partials (M_s, S_s, A, M_t, S_t, C_a, C_b)
// and its form tag (kTagFast / kTagOffset, how the partials are expressed)
// travel as four 64-bit words, (M_s, S_s), (A, M_t), (S_t, C_a), (C_b, tag),
// each published with one relaxed 64-bit atomic store and read back with
// relaxed 64-bit atomic loads.  A partial is stored as the bits of v + 0 (so
// -0 becomes +0) with the sign bit flipped, which is never zero; the slots
// are cleared before the kernel, so a nonzero word is a published one.
constexpr unsigned kTagFast = 1;
constexpr unsigned kTagOffset = 2;
__device__ inline unsigned enc(float v) { return __float_as_uint(v + 0.0f) ^ 0x80000000u; }
__device__ inline float dec(unsigned u) { return __uint_as_float(u ^ 0x80000000u); }
__device__ inline unsigned long long word2(unsigned lo, unsigned hi) {
  return ((unsigned long long)hi << 32) | (unsigned long long)lo;
}
// the seven partials of one chunk's four words, in publication order
__device__ inline void unpack_partials(const unsigned long long* w, float (&out)[kPartials]) {
#pragma unroll
  for (int i = 0; i < kPartials; ++i) {
    const unsigned long long x = w[i >> 1];
    out[i] = dec((i & 1) ? (unsigned)(x >> 32) : (unsigned)x);
  }
}

// The low half of the workspace's error key, read with a relaxed atomic
// load: an error key's low nibble is a priority below 15, so the half equals
// 0xFFFFFFFF exactly while no error has been recorded (a waiting workgroup
// polls it to learn that another one has timed out).
__device__ inline unsigned err_low(Header* hdr) {
  return __hip_atomic_load(reinterpret_cast<unsigned*>(&hdr->err_key), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}
constexpr unsigned kNoErrorLow = 0xFFFFFFFFu;

// Row merge.  A chunk reports (M_s, S_s, A, M_t, S_t, C_a, C_b) in one of two
// forms:
//  fast (tag kTagFast): M in log2 units (logits times log2 e), C = (0, 0),
//    S_s = sum 2^(a log2e - M_s),  A = sum 2^(a log2e - M_s) (a - b),  S_t likewise;
//  offset (kTagOffset): M = the chunk's maxima in logit units, C = (a, b)
//    where the student's logit peaks in the chunk,
//    S_s = sum 2^((a - M_s) log2e),  A = sum 2^((a - M_s) log2e) ((a - b) - (C_a - C_b)),
//    with both differences taken exactly (two_diff), so a term is accurate
//    to a few ulps of its own size whatever the magnitude of the logits.
// The maxima are the references of the exponents; C is the reference of the
// difference a - b, taken where the student's probability mass sits, so that
// a spike in the teacher (which sets its maximum) does not inflate every
// other term, and a peaked row's KL does not come from cancelling terms.
// The row works against natural references (R_s, R_t) >= every chunk's
// reference and the difference reference C* of the offset chunk with the
// largest C_a ((0, 0) when all chunks are fast), and accumulates in chunk order
//   S_s = sum_v 2^((a_v - R_s) log2e),  S_t likewise,
//   A   = sum_v 2^((a_v - R_s) log2e) ((a_v - b_v) - (C*_a - C*_b)),
// so that KL = A / S_s + ((C*_a - R_s) - (C*_b - R_t)) + ln(S_t / S_s).
// A fast chunk scales by 2^(M_s - R_s log2e) (one FMA for the exponent), an
// offset chunk by 2^((M_s - R_s) log2e); both add
// S_s ((C_a - C_b) - (C*_a - C*_b)) to A (exact differences), zero for rows of
// fast chunks only.
struct RowSums {
  float ss, aa, st;
};

// Error-free difference (Knuth's TwoSum applied to x + (-y)): hi = fl(x - y)
// and hi + lo = x - y exactly.  Needs plain rounded adds, which this file
// guarantees (no contraction).
struct Float2 {
  float hi, lo;
};
__device__ inline Float2 two_diff(float x, float y) {
  const float hi = x - y;
  const float yv = hi - x;   // the part of hi that came from -y
  const float xv = hi - yv;  // the part of hi that came from x
  return Float2{hi, (x - xv) - (y + yv)};
}

// (x - y) - c for a double-float c, to within a few ulps of the result even
// when x - y and c are large and nearly equal.
__device__ inline float diff_minus(float x, float y, Float2 c) {
  const Float2 d = two_diff(x, y);
  return (d.hi - c.hi) + (d.lo - c.lo);
}

// natural reference of a chunk: a logit-unit value at or above its own
__device__ inline float natural_ref(bool offset, float m) { return offset ? m : m * kLn2; }

__device__ inline void merge_chunk(bool offset, const float* w, float rs, float rt, Float2 c_row,
                                   RowSums& r) {
  float fs, ft;
  if (offset) {
    fs = exp2f((w[0] - rs) * kLog2e);
    ft = exp2f((w[3] - rt) * kLog2e);
  } else {
    fs = exp2f(fmaf(-rs, kLog2e, w[0]));
    ft = exp2f(fmaf(-rt, kLog2e, w[3]));
  }
  const float aa = fmaf(w[1], diff_minus(w[5], w[6], c_row), w[2]);
  r.ss = fmaf(w[1], fs, r.ss);
  r.aa = fmaf(aa, fs, r.aa);
  r.st = fmaf(w[4], ft, r.st);
}

// One (row, chunk) task per iteration.  A chunk is the pack range
// [pack_lo, pack_hi) of the row; thread tid owns packs pack_lo + v * 256 + tid
// for v < kVpt.  The host's tiling makes every chunk at least 256 (kVpt - 1)
// packs long, so every pack v < kVpt - 1 lies inside the chunk and only the
// last one is predicated (kCheckAll: all of them, for the unaligned scalar
// path, whose chunks carry no such guarantee).
template <bool kBf16, int kEpv, int kVpt, bool kCheckAll, bool kSplit>
__global__ __launch_bounds__(kRowThreads) void rowkl_kernel(RowParams p) {
  using P = Pack<kBf16, kEpv>;
  constexpr int kEs = kBf16 ? 2 : 4;
  constexpr int kPackBytes = kEpv * kEs;
  constexpr int kStep = kRowThreads * kPackBytes;  // bytes between a thread's packs

  __shared__ float s_max[2][kRowWaves];
  __shared__ float s_sum[3][kRowWaves];
  __shared__ unsigned long long s_word[kMaxChunks * kExchangeWords];
  __shared__ float s_ref[kRowWaves];
  __shared__ int s_lo[kMaxChunks + 1];  // first pack of each chunk
  __shared__ unsigned s_task;
  __shared__ int s_timeout;

  if (p.hdr->err_key != kNoError) return;
  // Two launches, one per load order (see the loads below): the split order
  // runs when at most 90% of the rows are supervised, the other one exits
  // here before taking any work.
  if (p.pick_order &&
      (10ll * __builtin_amdgcn_readfirstlane(p.hdr->n_sup) < 9ll * (long long)p.n_rows) != kSplit)
    return;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wid = tid / kWave;
  const unsigned n_tasks = (unsigned)p.n_rows * (unsigned)p.n_chunks;
  // chunk c is packs [chunk_start(c), chunk_start(c + 1)) of the row
  for (int k = tid; k <= p.n_chunks; k += kRowThreads)
    s_lo[k] = (int)chunk_start(p.n_packs, p.n_chunks, p.align, k);
  // data of this wave's most recent 16-byte store, kept live until the next
  // task's loads are issued (see keep_alive)
  typename P::Data carry = P::zero();

  // Thread 0 takes the next ticket near the end of the current task: after
  // the last gradient store is issued (a masked row: after its zero stores),
  // so the atomic's latency hides behind the stores draining, and a ticket
  // is started right after it is taken.  The workgroups that take the
  // chunks of one row (consecutive tickets) then start them at nearly the
  // same time and wait little for each other; taking it right after the row
  // merge instead measured 4% slower.  A ticket is never taken before the
  // current task's row mates have all published, so a workgroup never waits
  // for row mates while it holds a ticket it has not started, which keeps
  // the row-major ticket order deadlock-free.
  constexpr unsigned kNoTicket = 0xFFFFFFFFu;
  unsigned next_task = kNoTicket;

  for (;;) {
    if (tid == 0) {
      s_task = next_task != kNoTicket ? next_task : take_ticket(&p.hdr->ticket);
      next_task = kNoTicket;
    }
    __syncthreads();
    // Wave priority follows the task's progress: issuing loads 0, partial
    // sums 1, gradient (or zero) stores 2.  A wave further along its task
    // wins the SIMD's issue arbitration, finishes its stores sooner and
    // starts its next loads sooner; this measured 3.5% faster than equal
    // priorities (6.97 against 7.23 ms for 65,536 rows, same process).
    __builtin_amdgcn_s_setprio(0);
    const unsigned task = __builtin_amdgcn_readfirstlane(s_task);  // uniform: keep it scalar
    if (task >= n_tasks) break;
    // s_task is rewritten only after every wave has passed a later barrier of
    // this task (pass 1's, or the masked path's), so no wave can miss it
    if (tid == 0) s_timeout = 0;
    const long long row = (long long)(task / (unsigned)p.n_chunks);
    const int c = (int)(task - (unsigned)row * (unsigned)p.n_chunks);
    const int pack_lo = __builtin_amdgcn_readfirstlane(s_lo[c]);
    const int n_valid = __builtin_amdgcn_readfirstlane(s_lo[c + 1]) - pack_lo;  // packs in this chunk
    const long long col = (long long)pack_lo * kEpv;  // first element of the chunk
    const int lane_off = tid * kPackBytes;

    bool valid[kVpt];
#pragma unroll
    for (int v = 0; v < kVpt; ++v)
      valid[v] = (kCheckAll || v == kVpt - 1) ? (v * kRowThreads + tid < n_valid) : true;

    if (!p.mask[row]) {
      if (p.lse && c == 0 && tid == 0) {  // the row is not read: no log-partition function
        p.lse[2 * row] = __builtin_nanf("");
        p.lse[2 * row + 1] = __builtin_nanf("");
      }
      if (p.grad) {
        __builtin_amdgcn_s_setprio(2);
        const typename P::Data z = P::zero();
        const auto rg = chunk_rsrc(static_cast<char*>(p.grad) + (row * p.ld_g + col) * kEs);
#pragma unroll
        for (int v = 0; v < kVpt; ++v)
          if (valid[v]) P::store(rg, lane_off, v * kStep, z);
        __builtin_amdgcn_s_setprio(0);
        if (tid == 0) next_task = take_ticket(&p.hdr->ticket);
        // the zeros sit in registers the loop's phi copies may take over
        // right away: let the stores complete first
        drain_stores();
        keep_alive(carry);
      } else if (tid == 0) {
        next_task = take_ticket(&p.hdr->ticket);
      }
      __syncthreads();
      continue;
    }

    // ---- load the chunk of both rows into registers (an out-of-chunk pack
    // reads the chunk's first pack instead and is masked below)
    const auto rs = chunk_rsrc(static_cast<const char*>(p.zs) + (row * p.ld_s + col) * kEs);
    const auto rt = chunk_rsrc(static_cast<const char*>(p.zt) + (row * p.ld_t + col) * kEs);
    // Load order.  kSplit: the student's packs, then the teacher's; else
    // alternating.  On batches that mix masked and supervised rows the split
    // order measured 1.6% faster (6.84 against 6.96 ms for the 65,536-row
    // batch with 40% of its rows masked, 1.47 against 1.49 ms with 60%
    // masked, same process); with every row supervised it is 1.9% slower
    // (9.66 against 9.48 ms), so the host launches both orders and each
    // call runs one (see rowkl_kernel's first lines).  The two orders are
    // separate kernels: in one kernel the bf16 instantiation needs 258 VGPRs
    // (one wave per SIMD), and so does the fp32 one with the split order,
    // which therefore always alternates.
    P xs[kVpt], xt[kVpt];
    if constexpr (kSplit) {
#pragma unroll
      for (int v = 0; v < kVpt; ++v) {
        const bool sure = !kCheckAll && v < kVpt - 1;
        xs[v].load(rs, sure ? lane_off : (valid[v] ? lane_off : 0),
                   sure ? v * kStep : (valid[v] ? v * kStep : 0));
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int v = 0; v < kVpt; ++v) {
        const bool sure = !kCheckAll && v < kVpt - 1;
        xt[v].load(rt, sure ? lane_off : (valid[v] ? lane_off : 0),
                   sure ? v * kStep : (valid[v] ? v * kStep : 0));
      }
    } else {
#pragma unroll
      for (int v = 0; v < kVpt; ++v) {
        const bool sure = !kCheckAll && v < kVpt - 1;
        const int vo = sure ? lane_off : (valid[v] ? lane_off : 0);
        const int so = sure ? v * kStep : (valid[v] ? v * kStep : 0);
        xs[v].load(rs, vo, so);
        xt[v].load(rt, vo, so);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    keep_alive(carry);  // the previous task's last store has long read its data

    // ---- chunk partials.  Any reference works for S = sum 2^(a log2e - M)
    // as long as no term overflows, so the fast path's reference is the
    // maximum over each thread's first pack only, folded into one FMA per
    // exponent (log2 units: the fast form of merge_chunk).  A chunk whose
    // reference is far from zero (|max| > 64), or whose sums overflow, is
    // redone against its exact maximum with the references subtracted per
    // element, directly in natural-reference form (uniform branch; cold for
    // ordinary logits).
#define TURNKL_BLOCK_MAX2(MS, MT)                        \
  {                                                      \
    MS = wave_max(MS);                                   \
    MT = wave_max(MT);                                   \
    if (lane == 0) {                                     \
      s_max[0][wid] = MS;                                \
      s_max[1][wid] = MT;                                \
    }                                                    \
    __syncthreads();                                     \
    MS = s_max[0][0];                                    \
    MT = s_max[1][0];                                    \
    _Pragma("unroll") for (int w = 1; w < kRowWaves; ++w) { \
      MS = fmaxf(MS, s_max[0][w]);                       \
      MT = fmaxf(MT, s_max[1][w]);                       \
    }                                                    \
  }
#define TURNKL_FENCE_ALL()                                \
  _Pragma("unroll") for (int v = 0; v < kVpt; ++v) {     \
    xs[v].fence();                                       \
    xt[v].fence();                                       \
  }
  // OFFSET (a literal): exponents against natural references RS, RT and the
  // exact difference against the double-float C2; otherwise RS, RT are
  // log2-unit references folded into the exponent FMA (C2 unused)
#define TURNKL_CHUNK_SUMS(OFFSET, RS, RT, C2, SS, AA, ST)                     \
  {                                                                           \
    SS = 0.0f;                                                                \
    AA = 0.0f;                                                                \
    ST = 0.0f;                                                                \
    _Pragma("unroll") for (int v = 0; v < kVpt; ++v) {                        \
      _Pragma("unroll") for (int j = 0; j < kEpv; ++j) {                      \
        const float a = xs[v].get(j);                                         \
        const float b = xt[v].get(j);                                         \
        float es, et, d;                                                      \
        if (OFFSET) {                                                         \
          es = exp2_fast((a - (RS)) * kLog2e);                                \
          et = exp2_fast((b - (RT)) * kLog2e);                                \
          d = diff_minus(a, b, (C2));                                         \
        } else {                                                              \
          es = exp2_fast(fmaf(a, kLog2e, -(RS)));                             \
          et = exp2_fast(fmaf(b, kLog2e, -(RT)));                             \
          d = a - b;                                                          \
        }                                                                     \
        if (kCheckAll || v == kVpt - 1) {                                     \
          es = valid[v] ? es : 0.0f;                                          \
          et = valid[v] ? et : 0.0f;                                          \
          d = valid[v] ? d : 0.0f;                                            \
        }                                                                     \
        SS += es;                                                             \
        AA = fmaf(es, d, AA);                                                 \
        ST += et;                                                             \
      }                                                                       \
    }                                                                         \
    SS = wave_sum(SS);                                                        \
    AA = wave_sum(AA);                                                        \
    ST = wave_sum(ST);                                                        \
    if (lane == 0) {                                                          \
      s_sum[0][wid] = SS;                                                     \
      s_sum[1][wid] = AA;                                                     \
      s_sum[2][wid] = ST;                                                     \
    }                                                                         \
    __syncthreads();                                                          \
    SS = s_sum[0][0];                                                         \
    AA = s_sum[1][0];                                                         \
    ST = s_sum[2][0];                                                         \
    _Pragma("unroll") for (int w = 1; w < kRowWaves; ++w) {                   \
      SS += s_sum[0][w];                                                      \
      AA += s_sum[1][w];                                                      \
      ST += s_sum[2][w];                                                      \
    }                                                                         \
  }

    float ms = -INFINITY, mt = -INFINITY;
#pragma unroll
    for (int j = 0; j < kEpv; ++j) {
      ms = fmaxf(ms, valid[0] ? xs[0].get(j) : -INFINITY);
      mt = fmaxf(mt, valid[0] ? xt[0].get(j) : -INFINITY);
    }
    TURNKL_BLOCK_MAX2(ms, mt)
    float m2s = ms * kLog2e;
    float m2t = mt * kLog2e;
    __builtin_amdgcn_s_setprio(1);
    TURNKL_FENCE_ALL()
    float ss, aa, st;
    float c_a = 0.0f, c_b = 0.0f;  // difference reference (offset form only)
    TURNKL_CHUNK_SUMS(false, m2s, m2t, Float2{}, ss, aa, st)
    const bool offset = !(fmaxf(fabsf(m2s), fabsf(m2t)) <= kFar2) ||
                        !(__builtin_isfinite(ss) && __builtin_isfinite(st));
    if (offset) {
      __syncthreads();  // s_max / s_sum are about to be reused
      TURNKL_FENCE_ALL()
      // exact maxima, and the teacher logit at the student's maximum (ties:
      // the larger teacher logit, so every combination order agrees)
      ms = -INFINITY;
      mt = -INFINITY;
      float bm = -INFINITY;
#pragma unroll
      for (int v = 0; v < kVpt; ++v) {
#pragma unroll
        for (int j = 0; j < kEpv; ++j) {
          const float a = valid[v] ? xs[v].get(j) : -INFINITY;
          const float b = valid[v] ? xt[v].get(j) : -INFINITY;
          const bool take = (a > ms) | ((a == ms) & (b > bm));  // branch-free
          ms = take ? a : ms;
          bm = take ? b : bm;
          mt = fmaxf(mt, b);
        }
      }
#pragma unroll
      for (int o = kWave / 2; o > 0; o >>= 1) {
        const float oa = __shfl_xor(ms, o, kWave);
        const float ob = __shfl_xor(bm, o, kWave);
        const bool take = (oa > ms) | ((oa == ms) & (ob > bm));
        ms = take ? oa : ms;
        bm = take ? ob : bm;
        mt = fmaxf(mt, __shfl_xor(mt, o, kWave));
      }
      if (lane == 0) {
        s_max[0][wid] = ms;
        s_max[1][wid] = mt;
        s_ref[wid] = bm;
      }
      __syncthreads();
      ms = s_max[0][0];
      mt = s_max[1][0];
      bm = s_ref[0];
#pragma unroll
      for (int w = 1; w < kRowWaves; ++w) {
        const float oa = s_max[0][w];
        const float ob = s_ref[w];
        const bool take = (oa > ms) | ((oa == ms) & (ob > bm));
        ms = take ? oa : ms;
        bm = take ? ob : bm;
        mt = fmaxf(mt, s_max[1][w]);
      }
      m2s = ms;  // from here on: natural references
      m2t = mt;
      c_a = ms;  // difference reference: (a, b) where the student peaks
      c_b = bm;
      TURNKL_FENCE_ALL()
      __syncthreads();
      TURNKL_CHUNK_SUMS(true, m2s, m2t, two_diff(c_a, c_b), ss, aa, st)
    }
#undef TURNKL_CHUNK_SUMS
#undef TURNKL_FENCE_ALL
#undef TURNKL_BLOCK_MAX2
#pragma unroll
    for (int v = 0; v < kVpt; ++v) {
      xs[v].fence();
      xt[v].fence();
    }

    // ---- row scalars: publish this chunk's partials, read the row mates',
    // merge all of them in chunk order against the row references (the
    // largest chunk references; see merge_chunk), so every workgroup of the
    // row computes the same bits.  If any chunk took the offset path, the
    // whole row writes its gradient with offsets too.
    RowSums r{0.0f, 0.0f, 0.0f};
    float r_s, r_t;              // row references of the exponents, logit units
    float d_s = 0.0f, d_t = 0.0f;  // row reference C* of the difference a - b
    bool row_offset = offset;
    if (p.n_chunks > 1) {
      const int nw = p.n_chunks * kExchangeWords;
      unsigned long long* slot = p.slots + row * (long long)nw;
      if (tid == 0) {
        const unsigned tag = offset ? kTagOffset : kTagFast;
        unsigned long long* mine = slot + c * kExchangeWords;
        const unsigned long long words[kExchangeWords] = {
            word2(enc(m2s), enc(ss)), word2(enc(aa), enc(m2t)), word2(enc(st), enc(c_a)),
            word2(enc(c_b), tag)};
#pragma unroll
        for (int q = 0; q < kExchangeWords; ++q)
          __hip_atomic_store(mine + q, words[q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      // Wait for every word of the row, bounded: after spin_limit empty polls,
      // or as soon as another workgroup of the call has timed out (checked
      // every 256 polls), the task ends with the timeout error.
      for (int q = tid; q < nw; q += kRowThreads) {
        unsigned long long x;
        int spins = 0;
        while ((x = __hip_atomic_load(slot + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) == 0ull) {
          if (++spins > p.spin_limit || ((spins & 255) == 0 && err_low(p.hdr) != kNoErrorLow)) {
            s_timeout = 1;
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
        s_word[q] = x;
      }
      __syncthreads();
      if (s_timeout) {
        if (tid == 0) atomicMin(&p.hdr->err_key, err_key(0, kPrioTimeout));
        drain_stores();
        return;
      }
      // every thread merges all chunks in chunk order (uniform branches):
      // unrolled for the usual handful of chunks, a loop beyond
      constexpr int kUnrolled = 8;
#define TURNKL_TAG(K) \
  (__builtin_amdgcn_readfirstlane((unsigned)(s_word[kExchangeWords * (K) + 3] >> 32)) == kTagOffset)
      r_s = -INFINITY;
      r_t = -INFINITY;
      row_offset = false;
#define TURNKL_REFS(K)                                              \
  {                                                                 \
    const bool o = TURNKL_TAG(K);                                   \
    float w[kPartials];                                             \
    unpack_partials(s_word + kExchangeWords * (K), w);              \
    if (o && (!row_offset || w[5] > d_s)) {                         \
      d_s = w[5];                                                   \
      d_t = w[6];                                                   \
    }                                                               \
    row_offset = row_offset || o;                                   \
    r_s = fmaxf(r_s, natural_ref(o, w[0]));                         \
    r_t = fmaxf(r_t, natural_ref(o, w[3]));                         \
  }
#pragma unroll
      for (int k = 0; k < kUnrolled; ++k)
        if (k < p.n_chunks) TURNKL_REFS(k)
#pragma unroll 1
      for (int k = kUnrolled; k < p.n_chunks; ++k) TURNKL_REFS(k)
#undef TURNKL_REFS
      const Float2 c_row = two_diff(d_s, d_t);
#pragma unroll
      for (int k = 0; k < kUnrolled; ++k)
        if (k < p.n_chunks) {
          float w[kPartials];
          unpack_partials(s_word + kExchangeWords * k, w);
          merge_chunk(TURNKL_TAG(k), w, r_s, r_t, c_row, r);
        }
#pragma unroll 1
      for (int k = kUnrolled; k < p.n_chunks; ++k)
      {
        float w[kPartials];
        unpack_partials(s_word + kExchangeWords * k, w);
        merge_chunk(TURNKL_TAG(k), w, r_s, r_t, c_row, r);
      }
#undef TURNKL_TAG
    } else {
      r_s = natural_ref(offset, m2s);
      r_t = natural_ref(offset, m2t);
      d_s = c_a;
      d_t = c_b;
      const float w[kPartials] = {m2s, ss, aa, m2t, st, c_a, c_b};
      merge_chunk(offset, w, r_s, r_t, two_diff(d_s, d_t), r);
    }
    // without a gradient to write the task ends here
    if (tid == 0 && !p.grad) next_task = take_ticket(&p.hdr->ticket);

    // mu = <p_s, (a - b) - (C*_a - C*_b)>,
    // KL = <p_s, a - b> - lse(a) + lse(b) = mu + ((C*_a - R_s) - (C*_b - R_t)) + ln(S_t / S_s)
    // log sum exp of each row = R + ln S
    const float mu = r.aa / r.ss;
    if (c == 0 && tid == 0) {
      p.kl[row] = (mu + ((d_s - r_s) - (d_t - r_t))) + kLn2 * log2f(r.st / r.ss);
      if (p.lse) {
        p.lse[2 * row] = r_s + kLn2 * log2f(r.ss);
        p.lse[2 * row + 1] = r_t + kLn2 * log2f(r.st);
      }
    }

    // ---- gradient chunk, straight from registers:
    // G = grad_scale * w * 2^((a - R_s) log2e - log2 S_s) * (((a - b) - (C*_a - C*_b)) - mu),
    // with log2 |grad_scale * w| folded into the exponent and the sign applied
    // last.  Rows of fast chunks only (C* = 0) fold R_s into the exponent's
    // FMA; rows with an offset chunk subtract the references per element.
    if (p.grad) {
      __builtin_amdgcn_s_setprio(2);
      const float sc = p.wsc[row];
      const float l2 = log2f(r.ss) - log2f(fabsf(sc));
      const float shift = row_offset ? l2 : fmaf(r_s, kLog2e, l2);
      const unsigned flip = sc < 0.0f ? 0x80008000u : 0u;
      const auto rg = chunk_rsrc(static_cast<char*>(p.grad) + (row * p.ld_g + col) * kEs);
      if (!row_offset) {
        typename P::Data prev = P::zero();
#pragma unroll
        for (int v = 0; v < kVpt; ++v) {
          float out[kEpv];
#pragma unroll
          for (int j = 0; j < kEpv; ++j) {
            const float a = xs[v].get(j);
            const float b = xt[v].get(j);
            out[j] = exp2_fast(fmaf(a, kLog2e, -shift)) * ((a - b) - mu);
          }
          const typename P::Data cur = P::encode(out, flip);
          if (valid[v]) P::store(rg, lane_off, v * kStep, cur);
          // keep the store here, so the next pack's work separates it from
          // any reuse of its data registers; the previous pack's data is free
          __builtin_amdgcn_sched_barrier(0);
          keep_alive(prev);
          prev = cur;
          if (v == kVpt - 1 && tid == 0) next_task = take_ticket(&p.hdr->ticket);
        }
        carry = prev;
        __builtin_amdgcn_s_setprio(0);
      } else {
        // Offset rows (rare): read the chunk again, one pack at a time, so
        // this loop keeps no unpacked values of the unrolled one alive.  Each
        // thread reads a pack before it writes the same pack, which keeps an
        // in-place gradient safe; every store is drained before its data
        // registers can be reused.
        const Float2 c_row = two_diff(d_s, d_t);
        const auto rs2 = chunk_rsrc(static_cast<const char*>(p.zs) + (row * p.ld_s + col) * kEs);
        const auto rt2 = chunk_rsrc(static_cast<const char*>(p.zt) + (row * p.ld_t + col) * kEs);
        keep_alive(carry);
#pragma unroll 1
        for (int v = 0; v < kVpt; ++v) {
          if (v * kRowThreads + tid >= n_valid) break;
          P ya, yb;
          ya.load(rs2, lane_off, v * kStep);
          yb.load(rt2, lane_off, v * kStep);
          float out[kEpv];
#pragma unroll
          for (int j = 0; j < kEpv; ++j) {
            const float a = ya.get(j);
            const float b = yb.get(j);
            out[j] = exp2_fast(fmaf(a - r_s, kLog2e, -shift)) * (diff_minus(a, b, c_row) - mu);
          }
          P::store(rg, lane_off, v * kStep, P::encode(out, flip));
          drain_stores();
        }
        carry = P::zero();
      }
    }
  }
  drain_stores();
}

// ---------------------------------------------------------------------------
// launch

int cu_count() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < 64 && cache[dev] > 0) return cache[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) n = 256;
  if (dev < 64) cache[dev] = n;
  return n;
}

template <bool kBf16, int kEpv, int kVpt, bool kCheckAll, bool kSplit = false>
hipError_t launch_one(const RowParams& p, hipStream_t s) {
  static const int occ = [] {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, rowkl_kernel<kBf16, kEpv, kVpt, kCheckAll, kSplit>,
                                                     kRowThreads, 0) != hipSuccess || n < 1)
      n = 1;
    return n;
  }();
  const long long tasks = (long long)p.n_rows * p.n_chunks;
  long long grid = (long long)occ * cu_count();
  if (grid > tasks) grid = tasks;
  if (grid < 1) return hipSuccess;
  rowkl_kernel<kBf16, kEpv, kVpt, kCheckAll, kSplit><<<dim3((unsigned)grid), dim3(kRowThreads), 0, s>>>(p);
  return hipGetLastError();
}

// bf16: both load orders, each kernel checking which one the call uses;
// fp32: the alternating order alone.
template <bool kBf16, int kEpv, int kVpt>
hipError_t launch_orders(const RowParams& p, hipStream_t s) {
  if constexpr (kBf16) {
    RowParams q = p;
    q.pick_order = 1;
    if (hipError_t e = launch_one<kBf16, kEpv, kVpt, false, true>(q, s); e != hipSuccess) return e;
    return launch_one<kBf16, kEpv, kVpt, false, false>(q, s);
  } else {
    return launch_one<kBf16, kEpv, kVpt, false, false>(p, s);
  }
}

template <bool kBf16, int kEpv>
hipError_t launch_vpt(const RowParams& p, int vpt, hipStream_t s) {
  switch (vpt) {
#define TURNKL_CASE(n) \
    case n: return launch_orders<kBf16, kEpv, n>(p, s);
    TURNKL_CASE(1) TURNKL_CASE(2) TURNKL_CASE(3) TURNKL_CASE(4) TURNKL_CASE(5) TURNKL_CASE(6)
    TURNKL_CASE(7) TURNKL_CASE(8) TURNKL_CASE(9) TURNKL_CASE(10) TURNKL_CASE(11) TURNKL_CASE(12)
    TURNKL_CASE(13) TURNKL_CASE(14) TURNKL_CASE(15) TURNKL_CASE(16) TURNKL_CASE(17) TURNKL_CASE(18)
    TURNKL_CASE(19) TURNKL_CASE(20) TURNKL_CASE(21) TURNKL_CASE(22) TURNKL_CASE(23) TURNKL_CASE(24)
    TURNKL_CASE(25)
#undef TURNKL_CASE
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_rows(const RowParams& p, const RowTiling& t, hipStream_t s) {
  if (p.n_rows == 0) return hipSuccess;
  if (!t.vector) {
    return p.bf16 ? launch_one<true, 1, kScalarVpt, true>(p, s)
                  : launch_one<false, 1, kScalarVpt, true>(p, s);
  }
  return p.bf16 ? launch_vpt<true, 8>(p, t.vpt, s) : launch_vpt<false, 4>(p, t.vpt, s);
}

}  // namespace turnkl
