// Internal declarations shared by the turnkl kernels and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "turnkl.h"

namespace turnkl {

// ---------------------------------------------------------------------------
// error keys: the earliest offending token wins; at one token a padding-mask
// error, then a turn-range error, then an ordering error, then an outcome-flag
// error.

constexpr unsigned long long kNoError = ~0ull;
enum : unsigned {
  kPrioPadMask = 0,
  kPrioTurnRange = 1,
  kPrioUnsorted = 2,
  kPrioTimeout = 3,
  kPrioTopkId = 4,  // top-K path: a support id outside [0, vocab)
  kPrioOutcome = 5,  // outcome flag not constant over a trajectory
};

__host__ __device__ inline unsigned long long err_key(long long pos, unsigned prio) {
  return ((unsigned long long)pos << 4) | prio;
}

__host__ __device__ inline int status_from_key(unsigned long long key) {
  if (key == kNoError) return TURNKL_OK;
  switch ((unsigned)(key & 0xF)) {
    case kPrioPadMask: return TURNKL_ERR_PAD_MASK;
    case kPrioTurnRange: return TURNKL_ERR_TURN_RANGE;
    case kPrioUnsorted: return TURNKL_ERR_UNSORTED;
    case kPrioTopkId: return TURNKL_ERR_TOPK_ID;
    case kPrioOutcome: return TURNKL_ERR_OUTCOME;
    default: return TURNKL_ERR_SYNC_TIMEOUT;
  }
}

// ---------------------------------------------------------------------------
// workspace

struct Header {
  unsigned long long err_key;  // min over detected error keys; kNoError = none
  unsigned int ticket;         // row-kernel work counter
  int n_seg;                   // number of segments
  int b_eff;                   // trajectories with >= 1 supervised token
  int n_sup;                   // supervised tokens
  int pad[58];
};
static_assert(sizeof(Header) == 256, "header is one 256-byte line");

struct SegStat {
  double sum;    // sum of KL over the segment's supervised tokens
  double mean;   // sum / n
  double m2;     // sum of (KL - mean)^2
  double lm;     // w_seg * sum, the segment's share of L_blend
  double ltraj;  // sum / (B * N_b), its share of L_traj
  double lturn;  // sum / (B * T_b * n), its share of L_turn
  long long n;   // supervised tokens
  long long pad;
};

constexpr int kSegThreads = 256;
constexpr int kSegTokensPerThread = 4;
constexpr int kSegTile = kSegThreads * kSegTokensPerThread;

// Byte offsets into the caller's workspace.  Everything up to and including
// the segment table depends on n_tokens only (turnkl_get_segments relies on
// that).
struct Layout {
  size_t header, blk_cnt, blk_off, blk_err, tok_seg, seg_start, seg_len, seg_traj, seg_turn,
      seg_nsup, seg_head, traj_T, traj_N, w, wsc, kl, seg_stat, slots, topk, traj_Tv, turn_surv,
      total;
  long long nblk;
  int n_chunks;
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// A row-kernel chunk reports seven fp32 partials to its row mates, packed two
// to a 64-bit word with a tag in the last half: four words per chunk, each
// published with one 64-bit atomic store (see rowkl.hip, "Exchange words").
constexpr int kPartials = 7;
constexpr int kExchangeWords = 4;

// n_chunks > 1: exchange slots of the full-vocabulary row kernel; topk_k > 0:
// the top-K path's staging of the scaled gradient on each row's support;
// max_turns: per-turn survivor counts of the turn-support floor.
inline Layout make_layout(long long n_tokens, int n_chunks, int topk_k = 0, int max_turns = 0) {
  Layout L{};
  const size_t n = (size_t)n_tokens;
  L.nblk = (n_tokens + kSegTile - 1) / kSegTile;
  L.n_chunks = n_chunks;
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = align256(o + bytes); return at; };
  L.header = take(sizeof(Header));
  L.blk_cnt = take((size_t)L.nblk * 4);
  L.blk_off = take((size_t)L.nblk * 4);
  L.blk_err = take((size_t)L.nblk * 8);
  L.tok_seg = take(n * 4);
  L.seg_start = take(n * 4);
  L.seg_len = take(n * 4);
  L.seg_traj = take(n * 4);
  L.seg_turn = take(n * 4);
  L.seg_nsup = take(n * 4);
  L.seg_head = take(n * 4);
  L.traj_T = take(n * 4);
  L.traj_N = take(n * 4);
  L.w = take(n * 4);
  L.wsc = take(n * 4);
  L.kl = take(n * 4);
  L.seg_stat = take(n * sizeof(SegStat));
  L.slots = take(n * (size_t)n_chunks * kExchangeWords * 8);
  L.topk = take(n * (size_t)topk_k * 4);
  L.traj_Tv = take(n * 4);
  L.turn_surv = take((size_t)max_turns * 4);
  L.total = o;
  return L;
}

// Device pointers into one workspace.
struct Ws {
  Header* hdr;
  int* blk_cnt;
  int* blk_off;
  unsigned long long* blk_err;
  int* tok_seg;
  int* seg_start;
  int* seg_len;
  int* seg_traj;
  int* seg_turn;
  int* seg_nsup;
  int* seg_head;
  int* traj_T;
  int* traj_N;
  float* w;
  float* wsc;
  float* kl;
  SegStat* seg_stat;
  unsigned long long* slots;
  float* topk;
  int* traj_Tv;    // valid supervised turns of the trajectory (at its head segment)
  int* turn_surv;  // survivors n_t per turn index
};

inline Ws bind(void* base, const Layout& L) {
  char* b = static_cast<char*>(base);
  Ws w;
  w.hdr = reinterpret_cast<Header*>(b + L.header);
  w.blk_cnt = reinterpret_cast<int*>(b + L.blk_cnt);
  w.blk_off = reinterpret_cast<int*>(b + L.blk_off);
  w.blk_err = reinterpret_cast<unsigned long long*>(b + L.blk_err);
  w.tok_seg = reinterpret_cast<int*>(b + L.tok_seg);
  w.seg_start = reinterpret_cast<int*>(b + L.seg_start);
  w.seg_len = reinterpret_cast<int*>(b + L.seg_len);
  w.seg_traj = reinterpret_cast<int*>(b + L.seg_traj);
  w.seg_turn = reinterpret_cast<int*>(b + L.seg_turn);
  w.seg_nsup = reinterpret_cast<int*>(b + L.seg_nsup);
  w.seg_head = reinterpret_cast<int*>(b + L.seg_head);
  w.traj_T = reinterpret_cast<int*>(b + L.traj_T);
  w.traj_N = reinterpret_cast<int*>(b + L.traj_N);
  w.w = reinterpret_cast<float*>(b + L.w);
  w.wsc = reinterpret_cast<float*>(b + L.wsc);
  w.kl = reinterpret_cast<float*>(b + L.kl);
  w.seg_stat = reinterpret_cast<SegStat*>(b + L.seg_stat);
  w.slots = reinterpret_cast<unsigned long long*>(b + L.slots);
  w.topk = reinterpret_cast<float*>(b + L.topk);
  w.traj_Tv = reinterpret_cast<int*>(b + L.traj_Tv);
  w.turn_surv = reinterpret_cast<int*>(b + L.turn_surv);
  return w;
}

// ---------------------------------------------------------------------------
// row-kernel tiling

constexpr int kRowThreads = 256;
constexpr int kScalarVpt = 32;         // elements per thread on the unaligned path
constexpr int kMaxVpt = 25;            // packs per thread of the widest vector instantiation
constexpr int kMaxChunks = 128;        // chunks per row

struct RowTiling {
  bool vector;  // 16-byte vector loads (aligned rows, vocab a multiple of the vector)
  int vpt;      // vectors (or scalar elements) per thread per chunk
  int epv;      // elements per vector (8 bf16, 4 fp32, 1 on the scalar path)
  long long chunk;      // elements of the widest chunk
  long long min_chunk;  // packs of the narrowest chunk
  int n_chunks;
  int align;    // chunk boundaries are multiples of this many packs (see chunk_start)
};

// First pack of chunk c (0 <= c <= n_chunks) of a row of n_packs packs: the
// balanced boundary n_packs c / n_chunks rounded up to a multiple of `align`
// packs.  With align = 64 every interior boundary sits on a 1 KiB multiple
// from the row start, so each wave's 1 KiB load or store covers whole cache
// lines when rows start on a line; boundaries between lines made two waves
// share a line and measured about 4% slower.  align = 1 gives balanced chunks.
__host__ __device__ inline long long chunk_start(long long n_packs, int n_chunks, int align, int c) {
  if (c <= 0) return 0;
  if (c >= n_chunks) return n_packs;
  const long long b = n_packs * c / n_chunks;
  const long long r = (b + align - 1) / align * align;
  return r < n_packs ? r : n_packs;
}

// Tiling of the vector path for a given vectors-per-thread (0 = automatic).
RowTiling vector_tiling(long long vocab, int dtype, int vpt);
RowTiling scalar_tiling(long long vocab);

// ---------------------------------------------------------------------------
// launches (each returns hipSuccess or the launch error)

struct SegParams {
  const int* traj;
  const int* turn;
  const unsigned char* mask;
  const unsigned char* success;  // per-token outcome flags, or null
  long long n;
  int max_turns;
  int floor_on;   // turn-support floor active (support_floor > 0 or support_frac > 0)
  int floor;      // support_floor
  double frac;    // support_frac
};

// n_min = max(floor, ceil(frac * B)), with frac * B rounded once in double.
__host__ __device__ inline int support_n_min(const SegParams& p, int b_eff) {
  const double c = ceil(p.frac * (double)b_eff);
  return p.floor > (int)c ? p.floor : (int)c;
}

// The turn term of one supervised segment under the support floor: t_v is
// T_vb (T_b without a floor) and `valid` says whether the segment's turn is
// valid (always, without a floor).  u = [valid] / (t_v * n_bt) if t_v > 0,
// else 1 / N_b; callers fold the constant factors in the order the plain
// weights use, so that the floor-off results are unchanged bit for bit.
struct TurnTerm {
  double t_v;
  bool valid;
};

// Segment s of the trajectory whose head segment is h; only called on a batch
// without data errors (every turn id is in range).
__device__ inline TurnTerm turn_term(const SegParams& p, const Ws& ws, int s, int h, int n_min) {
  if (!p.floor_on) return TurnTerm{(double)ws.traj_T[h], true};
  return TurnTerm{(double)ws.traj_Tv[h], ws.turn_surv[ws.seg_turn[s]] >= n_min};
}

// alpha * u for the segment (see TurnTerm) with n_bt supervised tokens and
// N_b in its trajectory.
__device__ inline double turn_part(double alpha, const TurnTerm& u, double n_bt, double n_b) {
  if (u.t_v > 0.0) return u.valid ? alpha / (u.t_v * n_bt) : 0.0;
  return alpha / n_b;
}

hipError_t launch_segments(const SegParams& p, const Ws& ws, long long nblk, hipStream_t s);
hipError_t launch_weights(const SegParams& p, const Ws& ws, double alpha, float grad_scale,
                          int n_chunks, float* kl, hipStream_t s);

// Sizes are 32-bit here (the host rejects larger ones): the row kernel's
// scalar registers are its scarcest resource.
struct RowParams {
  const void* zs;
  const void* zt;
  void* grad;
  const unsigned char* mask;
  const float* wsc;
  float* kl;
  Header* hdr;
  unsigned long long* slots;
  int ld_s;
  int ld_t;
  int ld_g;
  int n_rows;
  int n_packs;   // vocab / elements per pack
  int n_chunks;  // <= kMaxChunks
  int align;     // chunk boundary alignment in packs (chunk_start)
  int bf16;
  int spin_limit;  // polls of a missing row-mate partial before the call times out
  int pick_order;  // 1: one of two launches (one per load order) that picks by
                   // the supervised share of the rows; 0: the only launch
  float* lse;    // [n_rows][2] log-partition functions of both rows, or null
};

// Default bound on those polls (s_sleep between polls; every 256th poll also
// checks whether another workgroup of the call has already timed out).
constexpr int kDefaultSpinLimit = 1 << 22;

hipError_t launch_rows(const RowParams& p, const RowTiling& t, hipStream_t s);

// Top-K path (the teacher's top-K support; both distributions renormalised on
// it).  The row kernel writes each supervised row's scaled gradient on the
// support to `stage` (row stride ld_stage) and its KL; the dense kernel then
// zero-fills every gradient row and scatters the staged values into it.
struct TopkParams {
  const void* zs;
  const int* ids;
  const float* vals;
  float* stage;
  void* grad;
  const unsigned char* mask;
  const float* wsc;
  float* kl;
  Header* hdr;
  long long ld_s;
  long long ld_k;      // row stride of ids and vals
  long long ld_stage;  // row stride of stage
  long long ld_g;
  int n_rows;
  int vocab;
  int k;
  int bf16;
  int zero_masked_stage;  // write zeros to stage rows of unsupervised tokens
  float* lse;             // [n_rows][2] log-partition functions on the support, or null
  int direct;             // topk_rows also writes the support values into grad
                          // (out of place, after the fill); stage may then be null
};

constexpr int kMaxTopK = 1024;

hipError_t launch_topk_rows(const TopkParams& p, hipStream_t s);
hipError_t launch_topk_fill(const TopkParams& p, hipStream_t s);
hipError_t launch_topk_scatter(const TopkParams& p, hipStream_t s);

// status_out: optional device int32 that receives the call's status
// (TURNKL_OK or the device-detected error) once the loss is written.
hipError_t launch_reduce(const SegParams& p, const Ws& ws, const float* kl, double alpha,
                         float* loss_out, turnkl_turn_stat* stats, turnkl_turn_stat* ostats,
                         int accumulate, int* status_out, hipStream_t s);

}  // namespace turnkl
