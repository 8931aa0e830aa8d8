// C-ABI of the fused turn-KL library: argument checks on the host, workspace
// carve-up and the launch sequence (segments -> weights -> rows -> reduce),
// all on the caller's stream with no host synchronisation.

#include <math.h>
#include <string.h>

#include <initializer_list>
#include <mutex>

#include "turnkl_internal.h"
#include "turnkl_testing.h"

namespace turnkl {

namespace {
// Measurement and test hooks (turnkl_testing.h), per host thread.  None of
// them changes what turnkl_workspace_bytes returns.
thread_local hipEvent_t t_row_before = nullptr;
thread_local hipEvent_t t_row_after = nullptr;
thread_local int t_vpt_override = 0;
thread_local int t_spin_limit = 0;

bool vpt_allowed(int v) { return v >= 1 && v <= kMaxVpt; }

// Default cap on packs per thread.  25 packs of both rows fit in 256 VGPRs
// (two workgroups per CU) and cut a V = 151936 bf16 row into 3 chunks; larger
// chunks measured faster than more workgroups per CU with smaller chunks
// (3 chunks: 6.97 ms, 4: 7.46 ms, 5: 7.39 ms, 6 chunks at three workgroups
// per CU: 7.40 ms for 65,536 rows, same process).
constexpr int kDefaultVmax = 25;

long long ceil_div(long long a, long long b) { return (a + b - 1) / b; }
}  // namespace

// k = ceil(P / (256 * vmax)) chunks of a row of P packs, with boundaries
// from chunk_start: 1 KiB-aligned when that keeps vpt = ceil(widest / 256)
// within vmax and every chunk at least 256 * (vpt - 1) packs long (the row
// kernel relies on that: only a thread's last pack can fall outside its
// chunk), else 128-byte-aligned, else balanced (chunks of P / k packs, for
// which both conditions hold by construction).
RowTiling vector_tiling(long long vocab, int dtype, int vmax) {
  RowTiling t{};
  t.vector = true;
  t.epv = dtype == TURNKL_BF16 ? 8 : 4;
  if (vmax == 0) vmax = kDefaultVmax;
  const long long packs = ceil_div(vocab, t.epv);
  t.n_chunks = (int)ceil_div(packs, (long long)kRowThreads * vmax);
  // balanced chunks: ceil(P / k) and floor(P / k) packs
  t.align = 1;
  t.min_chunk = packs / t.n_chunks;
  t.vpt = (int)ceil_div(ceil_div(packs, t.n_chunks), kRowThreads);
  t.chunk = ceil_div(packs, t.n_chunks) * t.epv;
  if (t.n_chunks < 2 || t.n_chunks > kMaxChunks) return t;
  for (int align : {64, 8}) {
    long long widest = 0, narrowest = packs;
    for (int c = 0; c < t.n_chunks; ++c) {
      const long long w = chunk_start(packs, t.n_chunks, align, c + 1) -
                          chunk_start(packs, t.n_chunks, align, c);
      widest = w > widest ? w : widest;
      narrowest = w < narrowest ? w : narrowest;
    }
    const int vpt = (int)ceil_div(widest, kRowThreads);
    if (vpt <= vmax && narrowest >= 1 && narrowest >= (long long)kRowThreads * (vpt - 1)) {
      t.align = align;
      t.vpt = vpt;
      t.chunk = widest * t.epv;
      t.min_chunk = narrowest;
      break;
    }
  }
  return t;
}

RowTiling scalar_tiling(long long vocab) {
  RowTiling t{};
  t.vector = false;
  t.epv = 1;
  t.vpt = kScalarVpt;
  t.n_chunks = (int)ceil_div(vocab, (long long)kRowThreads * kScalarVpt);
  t.chunk = ceil_div(vocab, t.n_chunks);
  t.min_chunk = vocab / t.n_chunks;
  t.align = 1;
  return t;
}

namespace {

// Whether a vocabulary admits the vector path at all (whole 16-byte packs, and
// chunks long enough for the kernel's one-predicated-pack layout); a call then
// takes it when its rows also start on 16-byte boundaries.
bool vector_possible(const RowTiling& t, long long vocab) {
  return vocab % t.epv == 0 && t.min_chunk >= (long long)kRowThreads * (t.vpt - 1);
}

// Chunks per row whose exchange slots a workspace holds (0: one chunk, no
// slots): the vector path's when the caller promises aligned rows and the
// vocabulary admits it, else the larger of the two paths'.
int workspace_chunks(long long vocab, int dtype, bool aligned_rows, int vpt) {
  const RowTiling v = vector_tiling(vocab, dtype, vpt);
  const int sc = scalar_tiling(vocab).n_chunks;
  int m = sc;
  if (vector_possible(v, vocab)) m = aligned_rows ? v.n_chunks : (v.n_chunks > sc ? v.n_chunks : sc);
  return m > 1 ? m : 0;
}

size_t workspace_bytes_for(int64_t n_tokens, int64_t vocab, int dtype, int32_t max_turns,
                           int aligned_rows, int vpt);

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  const char* pa = static_cast<const char*>(a);
  const char* pb = static_cast<const char*>(b);
  return pa < pb + nb && pb < pa + na;
}

size_t matrix_bytes(long long rows, long long ld, long long vocab, size_t es) {
  return rows > 0 ? (size_t)((rows - 1) * ld + vocab) * es : 0;
}

// A byte range of a caller buffer (p may be null: no range).
struct Region {
  const void* p;
  size_t n;
};

bool overlaps_any(const void* p, size_t n, std::initializer_list<Region> rs) {
  for (const Region& r : rs)
    if (r.p && r.n && overlaps(p, n, r.p, r.n)) return true;
  return false;
}

// What the options add to a call besides the segment parameters.
struct Extras {
  turnkl_turn_stat* outcome_stats = nullptr;
  float* weights = nullptr;  // per-token w_i
  float* lse = nullptr;      // per-token (student, teacher) log-partition functions
};

// Validates the options shared by both fused entry points and fills the
// segment parameters and outputs they imply.  `taken`: the call's inputs and
// other outputs, which the per-token outputs must not overlap.  Returns
// TURNKL_OK or the error code.
int apply_options(const turnkl_options* o, long long n_tokens, int max_turns,
                  const turnkl_turn_stat* turn_stats_out, std::initializer_list<Region> taken,
                  SegParams* sp, Extras* x) {
  *x = Extras{};
  if (!o) return TURNKL_OK;
  if (o->support_floor < 0) return TURNKL_ERR_INVALID_ARG;
  if (!(o->support_frac >= 0.0 && o->support_frac <= 1.0)) return TURNKL_ERR_INVALID_ARG;
  if (o->success && !o->outcome_stats_out) return TURNKL_ERR_INVALID_ARG;
  if (o->outcome_stats_out && !o->success && n_tokens > 0) return TURNKL_ERR_INVALID_ARG;
  if (o->outcome_stats_out && turn_stats_out &&
      overlaps(o->outcome_stats_out, 2 * (size_t)max_turns * sizeof(turnkl_turn_stat),
               turn_stats_out, (size_t)max_turns * sizeof(turnkl_turn_stat)))
    return TURNKL_ERR_ALIAS;
  if (((uintptr_t)o->token_weight_out & 3u) != 0 || ((uintptr_t)o->token_lse_out & 3u) != 0)
    return TURNKL_ERR_INVALID_ARG;
  if (n_tokens > 0) {
    const size_t nw = (size_t)n_tokens * 4, nl = (size_t)n_tokens * 8;
    const size_t nst = (size_t)max_turns * sizeof(turnkl_turn_stat);
    const Region own[] = {{turn_stats_out, nst}, {o->outcome_stats_out, 2 * nst}};
    for (const Region& r : own) {
      if (!r.p) continue;
      if (o->token_weight_out && overlaps(o->token_weight_out, nw, r.p, r.n)) return TURNKL_ERR_ALIAS;
      if (o->token_lse_out && overlaps(o->token_lse_out, nl, r.p, r.n)) return TURNKL_ERR_ALIAS;
    }
    if (o->token_weight_out && overlaps_any(o->token_weight_out, nw, taken)) return TURNKL_ERR_ALIAS;
    if (o->token_lse_out && overlaps_any(o->token_lse_out, nl, taken)) return TURNKL_ERR_ALIAS;
    if (o->token_weight_out && o->token_lse_out &&
        overlaps(o->token_weight_out, nw, o->token_lse_out, nl))
      return TURNKL_ERR_ALIAS;
    x->weights = o->token_weight_out;
    x->lse = o->token_lse_out;
  }
  sp->floor_on = o->support_floor > 0 || o->support_frac > 0.0;
  sp->floor = o->support_floor;
  sp->frac = o->support_frac;
  sp->success = o->outcome_stats_out ? o->success : nullptr;
  x->outcome_stats = o->outcome_stats_out;
  return TURNKL_OK;
}

// max_turns bounds: the statistics kernel runs 3 * max_turns + 1 workgroups.
constexpr int kMaxTurns = (0x7FFFFFFF - 1) / 3;

size_t workspace_bytes_for(int64_t n_tokens, int64_t vocab, int dtype, int32_t max_turns,
                           int aligned_rows, int vpt) {
  if (n_tokens < 0 || vocab < 1 || max_turns < 1 || max_turns > kMaxTurns) return 0;
  if (dtype != TURNKL_BF16 && dtype != TURNKL_F32) return 0;
  if (vpt != 0 && !vpt_allowed(vpt)) return 0;
  return make_layout(n_tokens, workspace_chunks(vocab, dtype, aligned_rows != 0, vpt), 0, max_turns)
      .total;
}

// ---------------------------------------------------------------------------
// Scratch of the no-allocation entry point (turnkl_fwd_bwd_noalloc): one
// array in every GPU's memory that runs the library, held until the process
// ends.  Host code never passes the array's name to a kernel or a copy (on
// the host it names a stand-in, not device memory): the device address comes
// from hipGetSymbolAddress, taken once per device with that device current
// and kept below.
constexpr size_t kScratchBytes = TURNKL_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, or null when it cannot be had.
void* scratch_address() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

// The fused call on a given workspace.  noalloc: the workspace is the scratch
// array (its own size check and error code); status_out: optional device
// int32 that receives the device-side status at the end of the call.
int fwd_bwd_impl(const void* student_logits, int64_t ld_student, const void* teacher_logits,
                 int64_t ld_teacher, int dtype, int64_t n_tokens, int64_t vocab,
                 const int32_t* turn_id, const int32_t* traj_id, const uint8_t* loss_mask,
                 double alpha, float grad_scale, float* loss_out, void* grad_out, int64_t ld_grad,
                 turnkl_turn_stat* turn_stats_out, int32_t max_turns, int accumulate_stats,
                 float* token_kl_out, const turnkl_options* options, void* workspace,
                 size_t workspace_bytes, bool noalloc, int32_t* status_out, hipStream_t stream) {
  // ---- arguments
  if (dtype != TURNKL_BF16 && dtype != TURNKL_F32) return TURNKL_ERR_INVALID_ARG;
  if (n_tokens < 0 || n_tokens > 0x7FFFFFFFll || vocab < 1 || max_turns < 1 ||
      max_turns > kMaxTurns)
    return TURNKL_ERR_INVALID_ARG;
  if (!(alpha >= 0.0 && alpha <= 1.0)) return TURNKL_ERR_INVALID_ARG;  // rejects NaN
  if (!isfinite(grad_scale)) return TURNKL_ERR_INVALID_ARG;
  if (!loss_out || (!noalloc && !workspace)) return TURNKL_ERR_INVALID_ARG;
  if (((uintptr_t)status_out & 3u) != 0) return TURNKL_ERR_INVALID_ARG;
  if (n_tokens > 0) {
    if (!student_logits || !teacher_logits || !turn_id || !traj_id || !loss_mask)
      return TURNKL_ERR_INVALID_ARG;
    if (ld_student < vocab || ld_teacher < vocab) return TURNKL_ERR_INVALID_ARG;
    if (grad_out && ld_grad < vocab) return TURNKL_ERR_INVALID_ARG;
  }
  if (!noalloc && ((uintptr_t)workspace & 255u) != 0) return TURNKL_ERR_WORKSPACE;

  const size_t es = dtype == TURNKL_BF16 ? 2 : 4;
  const size_t ns = matrix_bytes(n_tokens, ld_student, vocab, es);
  const size_t nt = matrix_bytes(n_tokens, ld_teacher, vocab, es);
  const size_t ng = grad_out ? matrix_bytes(n_tokens, ld_grad, vocab, es) : 0;
  if (grad_out && n_tokens > 0) {
    if (overlaps(grad_out, ng, teacher_logits, nt)) return TURNKL_ERR_ALIAS;
    const bool in_place = grad_out == student_logits && ld_grad == ld_student;
    if (!in_place && overlaps(grad_out, ng, student_logits, ns)) return TURNKL_ERR_ALIAS;
  }
  if (status_out &&
      overlaps_any(status_out, 4, {{student_logits, ns}, {teacher_logits, nt}, {grad_out, ng},
                                   {token_kl_out, (size_t)n_tokens * 4},
                                   {loss_out, 3 * sizeof(float)},
                                   {turn_stats_out, (size_t)max_turns * sizeof(turnkl_turn_stat)}}))
    return TURNKL_ERR_ALIAS;

  // ---- row tiling: 16-byte vectors when every row start is 16-byte aligned
  RowTiling tiling = vector_tiling(vocab, dtype, t_vpt_override);
  {
    const long long epv = tiling.epv;
    bool ok = vector_possible(tiling, vocab) && ld_student % epv == 0 && ld_teacher % epv == 0;
    ok = ok && ((uintptr_t)student_logits & 15u) == 0 && ((uintptr_t)teacher_logits & 15u) == 0;
    if (grad_out) ok = ok && ld_grad % epv == 0 && ((uintptr_t)grad_out & 15u) == 0;
    if (!ok) tiling = scalar_tiling(vocab);
  }
  if (tiling.n_chunks > kMaxChunks) return TURNKL_ERR_INVALID_ARG;
  if (n_tokens > 0 && (ld_student > 0x7FFFFFFFll || ld_teacher > 0x7FFFFFFFll ||
                       (grad_out && ld_grad > 0x7FFFFFFFll)))
    return TURNKL_ERR_INVALID_ARG;
  if ((unsigned long long)n_tokens * (unsigned long long)tiling.n_chunks > 0x7FFFFFFFull)
    return TURNKL_ERR_INVALID_ARG;

  SegParams sp{traj_id, turn_id, loss_mask, nullptr, (long long)n_tokens, max_turns, 0, 0, 0.0};
  Extras ex;
  if (int rc = apply_options(options, n_tokens, max_turns, turn_stats_out,
                             {{student_logits, ns}, {teacher_logits, nt}, {grad_out, ng},
                              {token_kl_out, (size_t)n_tokens * 4}, {loss_out, 3 * sizeof(float)},
                              {status_out, status_out ? 4u : 0u}},
                             &sp, &ex))
    return rc;

  // the layout of this call: exchange slots for the path it takes
  const Layout L = make_layout(n_tokens, tiling.n_chunks > 1 ? tiling.n_chunks : 0, 0, max_turns);
  if (noalloc) {
    if (L.total > kScratchBytes) return TURNKL_ERR_SCRATCH;
    workspace = scratch_address();
    if (!workspace) return TURNKL_ERR_HIP;
  } else if (workspace_bytes < L.total) {
    return TURNKL_ERR_WORKSPACE;
  }
  Ws ws = bind(workspace, L);
  if (ex.weights) ws.w = ex.weights;
  float* kl = token_kl_out ? token_kl_out : ws.kl;

  // ---- launches
  if (launch_segments(sp, ws, L.nblk, stream) != hipSuccess) return TURNKL_ERR_HIP;
  if (launch_weights(sp, ws, alpha, grad_scale, tiling.n_chunks, kl, stream) != hipSuccess)
    return TURNKL_ERR_HIP;

  RowParams rp{};
  rp.zs = student_logits;
  rp.ld_s = (int)ld_student;
  rp.zt = teacher_logits;
  rp.ld_t = (int)ld_teacher;
  rp.grad = grad_out;
  rp.ld_g = grad_out ? (int)ld_grad : 0;
  rp.mask = loss_mask;
  rp.wsc = ws.wsc;
  rp.kl = kl;
  rp.hdr = ws.hdr;
  rp.slots = ws.slots;
  rp.n_rows = (int)n_tokens;
  rp.n_packs = (int)(vocab / tiling.epv);
  rp.n_chunks = tiling.n_chunks;
  rp.align = tiling.align;
  rp.bf16 = dtype == TURNKL_BF16;
  rp.lse = ex.lse;
  rp.spin_limit = t_spin_limit > 0 ? t_spin_limit : kDefaultSpinLimit;
  const bool prof = t_row_before && t_row_after;
  if (prof && hipEventRecord(t_row_before, stream) != hipSuccess) return TURNKL_ERR_HIP;
  if (launch_rows(rp, tiling, stream) != hipSuccess) return TURNKL_ERR_HIP;
  if (prof && hipEventRecord(t_row_after, stream) != hipSuccess) return TURNKL_ERR_HIP;

  if (launch_reduce(sp, ws, kl, alpha, loss_out, turn_stats_out, ex.outcome_stats,
                    accumulate_stats, status_out, stream) != hipSuccess)
    return TURNKL_ERR_HIP;
  return TURNKL_OK;
}

}  // namespace
}  // namespace turnkl

using namespace turnkl;

extern "C" {

size_t turnkl_workspace_bytes(int64_t n_tokens, int64_t vocab, int dtype, int32_t max_turns,
                              int aligned_rows) {
  return workspace_bytes_for(n_tokens, vocab, dtype, max_turns, aligned_rows, 0);
}

size_t turnkl_testing_workspace_bytes(int64_t n_tokens, int64_t vocab, int dtype,
                                      int32_t max_turns, int aligned_rows,
                                      int vectors_per_thread) {
  return workspace_bytes_for(n_tokens, vocab, dtype, max_turns, aligned_rows, vectors_per_thread);
}

int turnkl_fwd_bwd(const void* student_logits, int64_t ld_student, const void* teacher_logits,
                   int64_t ld_teacher, int dtype, int64_t n_tokens, int64_t vocab,
                   const int32_t* turn_id, const int32_t* traj_id, const uint8_t* loss_mask,
                   double alpha, float grad_scale, float* loss_out, void* grad_out,
                   int64_t ld_grad, turnkl_turn_stat* turn_stats_out, int32_t max_turns,
                   int accumulate_stats, float* token_kl_out, const turnkl_options* options,
                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return fwd_bwd_impl(student_logits, ld_student, teacher_logits, ld_teacher, dtype, n_tokens,
                      vocab, turn_id, traj_id, loss_mask, alpha, grad_scale, loss_out, grad_out,
                      ld_grad, turn_stats_out, max_turns, accumulate_stats, token_kl_out, options,
                      workspace, workspace_bytes, false, nullptr, stream);
}

int turnkl_fwd_bwd_noalloc(const void* student_logits, int64_t ld_student,
                           const void* teacher_logits, int64_t ld_teacher, int dtype,
                           int64_t n_tokens, int64_t vocab, const int32_t* turn_id,
                           const int32_t* traj_id, const uint8_t* loss_mask, double alpha,
                           float grad_scale, float* loss_out, void* grad_out, int64_t ld_grad,
                           turnkl_turn_stat* turn_stats_out, int32_t max_turns,
                           int accumulate_stats, float* token_kl_out,
                           const turnkl_options* options, int32_t* status_out,
                           hipStream_t stream) {
  return fwd_bwd_impl(student_logits, ld_student, teacher_logits, ld_teacher, dtype, n_tokens,
                      vocab, turn_id, traj_id, loss_mask, alpha, grad_scale, loss_out, grad_out,
                      ld_grad, turn_stats_out, max_turns, accumulate_stats, token_kl_out, options,
                      nullptr, 0, true, status_out, stream);
}

size_t turnkl_topk_workspace_bytes(int64_t n_tokens, int32_t k, int32_t max_turns) {
  if (n_tokens < 0 || k < 1 || k > kMaxTopK || max_turns < 1 || max_turns > kMaxTurns) return 0;
  return make_layout(n_tokens, 0, k, max_turns).total;
}

int turnkl_fwd_bwd_topk(const void* student_logits, int64_t ld_student, int dtype,
                        int64_t n_tokens, int64_t vocab, const int32_t* teacher_ids,
                        const float* teacher_vals, int64_t ld_topk, int32_t k,
                        const int32_t* turn_id, const int32_t* traj_id, const uint8_t* loss_mask,
                        double alpha, float grad_scale, float* loss_out, void* grad_out,
                        int64_t ld_grad, float* grad_topk_out, int64_t ld_grad_topk,
                        turnkl_turn_stat* turn_stats_out, int32_t max_turns, int accumulate_stats,
                        float* token_kl_out, const turnkl_options* options, void* workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  // ---- arguments
  if (dtype != TURNKL_BF16 && dtype != TURNKL_F32) return TURNKL_ERR_INVALID_ARG;
  const size_t es = dtype == TURNKL_BF16 ? 2 : 4;
  if (n_tokens < 0 || n_tokens > 0x7FFFFFFFll || vocab < 1 || max_turns < 1 ||
      max_turns > kMaxTurns)
    return TURNKL_ERR_INVALID_ARG;
  if ((unsigned long long)vocab * es > 0x7FFFFFFFull) return TURNKL_ERR_INVALID_ARG;
  if (k < 1 || k > kMaxTopK || k > vocab) return TURNKL_ERR_INVALID_ARG;
  if (!(alpha >= 0.0 && alpha <= 1.0)) return TURNKL_ERR_INVALID_ARG;
  if (!isfinite(grad_scale)) return TURNKL_ERR_INVALID_ARG;
  if (!loss_out || !workspace) return TURNKL_ERR_INVALID_ARG;
  if (n_tokens > 0) {
    if (!student_logits || !teacher_ids || !teacher_vals || !turn_id || !traj_id || !loss_mask)
      return TURNKL_ERR_INVALID_ARG;
    if (ld_student < vocab || ld_topk < k) return TURNKL_ERR_INVALID_ARG;
    if (grad_out && ld_grad < vocab) return TURNKL_ERR_INVALID_ARG;
    if (grad_topk_out && ld_grad_topk < k) return TURNKL_ERR_INVALID_ARG;
  }
  if (((uintptr_t)workspace & 255u) != 0) return TURNKL_ERR_WORKSPACE;
  const size_t nid = matrix_bytes(n_tokens, ld_topk, k, 4);
  const size_t ns = matrix_bytes(n_tokens, ld_student, vocab, es);
  const size_t ng = grad_out ? matrix_bytes(n_tokens, ld_grad, vocab, es) : 0;
  const size_t ngk = grad_topk_out ? matrix_bytes(n_tokens, ld_grad_topk, k, 4) : 0;
  if (n_tokens > 0) {
    if (grad_out) {
      if (overlaps(grad_out, ng, teacher_ids, nid) || overlaps(grad_out, ng, teacher_vals, nid))
        return TURNKL_ERR_ALIAS;
      const bool in_place = grad_out == student_logits && ld_grad == ld_student;
      if (!in_place && overlaps(grad_out, ng, student_logits, ns)) return TURNKL_ERR_ALIAS;
      if (grad_topk_out && overlaps(grad_out, ng, grad_topk_out, ngk)) return TURNKL_ERR_ALIAS;
    }
    if (grad_topk_out) {
      if (overlaps(grad_topk_out, ngk, teacher_ids, nid) ||
          overlaps(grad_topk_out, ngk, teacher_vals, nid) ||
          overlaps(grad_topk_out, ngk, student_logits, ns))
        return TURNKL_ERR_ALIAS;
    }
  }
  SegParams sp{traj_id, turn_id, loss_mask, nullptr, (long long)n_tokens, max_turns, 0, 0, 0.0};
  Extras ex;
  if (int rc = apply_options(options, n_tokens, max_turns, turn_stats_out,
                             {{student_logits, ns}, {teacher_ids, nid}, {teacher_vals, nid},
                              {grad_out, ng}, {grad_topk_out, ngk},
                              {token_kl_out, (size_t)n_tokens * 4}, {loss_out, 3 * sizeof(float)}},
                             &sp, &ex))
    return rc;
  const Layout L = make_layout(n_tokens, 0, k, max_turns);
  if (workspace_bytes < L.total) return TURNKL_ERR_WORKSPACE;
  Ws ws = bind(workspace, L);
  if (ex.weights) ws.w = ex.weights;
  float* kl = token_kl_out ? token_kl_out : ws.kl;

  // ---- launches
  if (launch_segments(sp, ws, L.nblk, stream) != hipSuccess) return TURNKL_ERR_HIP;
  if (launch_weights(sp, ws, alpha, grad_scale, 0, kl, stream) != hipSuccess) return TURNKL_ERR_HIP;
  TopkParams tp{};
  tp.zs = student_logits;
  tp.ids = teacher_ids;
  tp.vals = teacher_vals;
  tp.stage = grad_topk_out ? grad_topk_out : ws.topk;
  tp.grad = grad_out;
  tp.mask = loss_mask;
  tp.wsc = ws.wsc;
  tp.kl = kl;
  tp.hdr = ws.hdr;
  tp.ld_s = ld_student;
  tp.ld_k = ld_topk;
  tp.ld_stage = grad_topk_out ? ld_grad_topk : k;
  tp.ld_g = grad_out ? ld_grad : 0;
  tp.n_rows = (int)n_tokens;
  tp.vocab = (int)vocab;
  tp.k = k;
  tp.bf16 = dtype == TURNKL_BF16;
  tp.zero_masked_stage = grad_topk_out != nullptr;
  tp.lse = ex.lse;
  // out of place: fill the dense gradient first, then the rows write their
  // support values into it; in place the rows must read the logits first
  tp.direct = grad_out != nullptr && grad_out != student_logits;
  if (tp.direct) tp.stage = grad_topk_out;
  const bool prof = t_row_before && t_row_after;
  if (prof && hipEventRecord(t_row_before, stream) != hipSuccess) return TURNKL_ERR_HIP;
  if (tp.direct) {
    if (launch_topk_fill(tp, stream) != hipSuccess) return TURNKL_ERR_HIP;
    if (launch_topk_rows(tp, stream) != hipSuccess) return TURNKL_ERR_HIP;
  } else {
    if (launch_topk_rows(tp, stream) != hipSuccess) return TURNKL_ERR_HIP;
    if (launch_topk_fill(tp, stream) != hipSuccess) return TURNKL_ERR_HIP;
    if (launch_topk_scatter(tp, stream) != hipSuccess) return TURNKL_ERR_HIP;
  }
  if (prof && hipEventRecord(t_row_after, stream) != hipSuccess) return TURNKL_ERR_HIP;
  if (launch_reduce(sp, ws, kl, alpha, loss_out, turn_stats_out, ex.outcome_stats,
                    accumulate_stats, nullptr, stream) != hipSuccess)
    return TURNKL_ERR_HIP;
  return TURNKL_OK;
}

int turnkl_get_status(const void* workspace, hipStream_t stream) {
  if (!workspace) return TURNKL_ERR_INVALID_ARG;
  const Header* hdr = static_cast<const Header*>(workspace);
  unsigned long long key = 0;
  if (hipMemcpyAsync(&key, &hdr->err_key, sizeof key, hipMemcpyDeviceToHost, stream) != hipSuccess)
    return TURNKL_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return TURNKL_ERR_HIP;
  return status_from_key(key);
}

int turnkl_get_segments(const void* workspace, int64_t n_tokens, hipStream_t stream,
                        int32_t* n_seg, int32_t* seg_start, int32_t* seg_len, int32_t* seg_traj,
                        int32_t* seg_turn, int32_t* seg_nsup) {
  if (!workspace || !n_seg || n_tokens < 0) return TURNKL_ERR_INVALID_ARG;
  const Layout L = make_layout(n_tokens, 0);
  const Ws ws = bind(const_cast<void*>(workspace), L);
  int n = 0;
  if (hipMemcpyAsync(&n, &ws.hdr->n_seg, sizeof n, hipMemcpyDeviceToHost, stream) != hipSuccess)
    return TURNKL_ERR_HIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return TURNKL_ERR_HIP;
  if (n < 0 || n > n_tokens) return TURNKL_ERR_INVALID_ARG;
  *n_seg = n;
  const size_t bytes = (size_t)n * 4;
  struct { int32_t* dst; const int* src; } cp[] = {{seg_start, ws.seg_start}, {seg_len, ws.seg_len},
                                                   {seg_traj, ws.seg_traj}, {seg_turn, ws.seg_turn},
                                                   {seg_nsup, ws.seg_nsup}};
  for (auto& c : cp) {
    if (!c.dst || bytes == 0) continue;
    if (hipMemcpyAsync(c.dst, c.src, bytes, hipMemcpyDeviceToDevice, stream) != hipSuccess)
      return TURNKL_ERR_HIP;
  }
  return hipStreamSynchronize(stream) == hipSuccess ? TURNKL_OK : TURNKL_ERR_HIP;
}

double turnkl_alpha_schedule(int64_t k, int64_t K, double s, double e) {
  if (K < 1) return NAN;
  const double prog = (double)k / (double)K;
  if (e <= s) return prog >= s ? 1.0 : 0.0;
  const double a = (prog - s) / (e - s);
  return a < 0.0 ? 0.0 : (a > 1.0 ? 1.0 : a);
}

const char* turnkl_status_string(int status) {
  switch (status) {
    case TURNKL_OK: return "ok";
    case TURNKL_ERR_INVALID_ARG: return "invalid argument";
    case TURNKL_ERR_ALIAS: return "grad_out overlaps an input";
    case TURNKL_ERR_WORKSPACE: return "workspace too small or misaligned";
    case TURNKL_ERR_UNSORTED: return "trajectory or turn ids out of order";
    case TURNKL_ERR_TURN_RANGE: return "turn id outside [0, max_turns)";
    case TURNKL_ERR_PAD_MASK: return "padding token with loss mask set";
    case TURNKL_ERR_HIP: return "HIP runtime error";
    case TURNKL_ERR_SYNC_TIMEOUT: return "row exchange timed out";
    case TURNKL_ERR_TOPK_ID: return "top-K support id outside [0, vocab)";
    case TURNKL_ERR_OUTCOME: return "outcome flag not constant over a trajectory";
    case TURNKL_ERR_SCRATCH:
      return "problem larger than the built-in scratch of turnkl_fwd_bwd_noalloc";
    default: return "unknown status";
  }
}

int turnkl_profile_row_kernel(hipEvent_t before, hipEvent_t after) {
  t_row_before = before;
  t_row_after = after;
  return TURNKL_OK;
}

int turnkl_set_spin_limit(int polls) {
  if (polls < 0) return TURNKL_ERR_INVALID_ARG;
  t_spin_limit = polls;
  return TURNKL_OK;
}

int turnkl_set_row_tiling(int vectors_per_thread) {
  if (vectors_per_thread != 0 && !vpt_allowed(vectors_per_thread)) return TURNKL_ERR_INVALID_ARG;
  t_vpt_override = vectors_per_thread;
  return TURNKL_OK;
}

}  // extern "C"
