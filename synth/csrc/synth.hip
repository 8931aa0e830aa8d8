// Seeded synthetic logits for the turn-KL workloads.
//
// Every value is a pure function of (seed, stream, row, column): the device
// fills full-size batches directly in HBM, and the host regenerates any row
// bit-for-bit to feed the CPU checker.  Both paths come from the single
// per-element routine below, which uses only 64-bit integer hashing, exact
// int->float conversion and IEEE fp32 multiply/add with contraction disabled,
// so host and device results are identical.
//
// Generator: SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom
// number generators", OOPSLA 2014) used in counter mode: output n of a stream
// with key k is mix64(k + (n + 1) * GOLDEN), mix64 being SplitMix64's
// finaliser.  A value with approximately normal distribution is the centred
// sum of the four 16-bit fields of one output (Irwin-Hall, n = 4: variance
// 4 * (2^32 - 1) / 12 in field units), scaled by sigma * sqrt(3) / 65536.
//
// This module holds none of the loss arithmetic; it only produces inputs.

#pragma clang fp contract(off)

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <thread>
#include <vector>

extern "C" {

// Recipe of one batch of logits (shared layout with synth/_lib.py).
typedef struct {
  uint64_t seed;             // batch seed
  int64_t vocab;             // V
  int64_t ld;                // row stride of the output buffers, elements
  int32_t dtype;             // 0 = bf16 (RNE from fp32), 1 = fp32
  int32_t n_peaks;           // peaked columns per row (0 = none)
  float student_scale;       // sigma_student * sqrt(3) / 65536
  float peak_boost;          // added to both models at the peak columns
  uint32_t shift_threshold;  // teacher peaks re-drawn iff hi32(hash) < this
  uint32_t reserved;
} synth_params;

}  // extern "C"

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

enum : uint64_t {
  kStreamStudent = 0,
  kStreamTeacherNoise = 1,
  kStreamStudentPeaks = 2,
  kStreamShiftFlag = 3,
  kStreamTeacherPeaks = 4,
};

__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Output n of the SplitMix64 sequence whose state starts at `key`.
__host__ __device__ inline uint64_t splitmix_at(uint64_t key, uint64_t n) {
  return mix64(key + (n + 1) * kGolden);
}

__host__ __device__ inline uint64_t stream_key(uint64_t seed, uint64_t stream) {
  return splitmix_at(seed, stream);
}

// Centred Irwin-Hall(4) integer in [-131070, 131070]; exact in fp32.
__host__ __device__ inline int32_t gauss4(uint64_t x) {
  int32_t s = (int32_t)(x & 0xFFFF) + (int32_t)((x >> 16) & 0xFFFF) +
              (int32_t)((x >> 32) & 0xFFFF) + (int32_t)(x >> 48);
  return s - 131070;
}

__host__ __device__ inline uint16_t bf16_rne(float f) {
  uint32_t u;
  __builtin_memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

struct RowPeaks {
  int64_t student[8];
  int64_t teacher[8];
  int n;
};

__host__ __device__ inline void row_peaks(const synth_params& p, int64_t row, RowPeaks& pk) {
  const int n = p.n_peaks < 8 ? p.n_peaks : 8;
  pk.n = n;
  const uint64_t ks = stream_key(p.seed, kStreamStudentPeaks);
  const uint64_t kf = stream_key(p.seed, kStreamShiftFlag);
  const uint64_t kt = stream_key(p.seed, kStreamTeacherPeaks);
  const bool shifted = (uint32_t)(splitmix_at(kf, (uint64_t)row) >> 32) < p.shift_threshold;
  for (int j = 0; j < n; ++j) {
    const uint64_t c = (uint64_t)row * 8u + (uint64_t)j;
    pk.student[j] = (int64_t)(splitmix_at(ks, c) % (uint64_t)p.vocab);
    pk.teacher[j] = shifted ? (int64_t)(splitmix_at(kt, c) % (uint64_t)p.vocab) : pk.student[j];
  }
}

__host__ __device__ inline bool is_peak(const int64_t* cols, int n, int64_t col) {
  bool hit = false;
  for (int j = 0; j < n; ++j) hit |= (cols[j] == col);
  return hit;
}

// The per-element recipe.  Student = base (+ boost at its peaks);
// teacher = (base + noise) (+ boost at its peaks); both rounded once.
__host__ __device__ inline void element(const synth_params& p, uint64_t key_s, uint64_t key_n,
                                        float teacher_scale, const RowPeaks& pk, int64_t row,
                                        int64_t col, float& s_out, float& t_out) {
  const uint64_t n = (uint64_t)row * (uint64_t)p.vocab + (uint64_t)col;
  const float base = (float)gauss4(splitmix_at(key_s, n)) * p.student_scale;
  const float noise = (float)gauss4(splitmix_at(key_n, n)) * teacher_scale;
  float s = base;
  float t = base + noise;
  if (is_peak(pk.student, pk.n, col)) s = s + p.peak_boost;
  if (is_peak(pk.teacher, pk.n, col)) t = t + p.peak_boost;
  s_out = s;
  t_out = t;
}

template <bool kBf16>
__host__ __device__ inline void store(void* base, int64_t off, float v) {
  if (kBf16) {
    static_cast<uint16_t*>(base)[off] = bf16_rne(v);
  } else {
    static_cast<float*>(base)[off] = v;
  }
}

constexpr int kThreads = 256;
constexpr int kColsPerThread = 8;
constexpr int kColsPerBlock = kThreads * kColsPerThread;

template <bool kBf16>
__global__ __launch_bounds__(kThreads) void fill_kernel(synth_params p, const float* __restrict__ kt,
                                                        int64_t r0, int64_t blocks_per_row,
                                                        void* zs, void* zt) {
  const int64_t b = blockIdx.x;
  const int64_t rel = b / blocks_per_row;
  const int64_t cb = b - rel * blocks_per_row;
  const int64_t row = r0 + rel;
  __shared__ RowPeaks s_pk;
  if (threadIdx.x == 0) row_peaks(p, row, s_pk);
  __syncthreads();
  const RowPeaks pk = s_pk;
  const uint64_t key_s = stream_key(p.seed, kStreamStudent);
  const uint64_t key_n = stream_key(p.seed, kStreamTeacherNoise);
  const float tsc = kt[row];
  const int64_t c0 = cb * kColsPerBlock + (int64_t)threadIdx.x * kColsPerThread;
  for (int j = 0; j < kColsPerThread; ++j) {
    const int64_t col = c0 + j;
    if (col >= p.vocab) break;
    float s, t;
    element(p, key_s, key_n, tsc, pk, row, col, s, t);
    const int64_t off = rel * p.ld + col;
    if (zs) store<kBf16>(zs, off, s);
    if (zt) store<kBf16>(zt, off, t);
  }
}

template <bool kBf16>
void fill_rows_host(const synth_params& p, const float* kt, int64_t r0, int64_t ra, int64_t rb,
                    void* zs, void* zt) {
  const uint64_t key_s = stream_key(p.seed, kStreamStudent);
  const uint64_t key_n = stream_key(p.seed, kStreamTeacherNoise);
  for (int64_t row = ra; row < rb; ++row) {
    RowPeaks pk;
    row_peaks(p, row, pk);
    const float tsc = kt[row];
    for (int64_t col = 0; col < p.vocab; ++col) {
      float s, t;
      element(p, key_s, key_n, tsc, pk, row, col, s, t);
      const int64_t off = (row - r0) * p.ld + col;
      if (zs) store<kBf16>(zs, off, s);
      if (zt) store<kBf16>(zt, off, t);
    }
  }
}

int check_params(const synth_params* p, const float* kt, int64_t r0, int64_t r1) {
  if (!p || !kt || p->vocab < 1 || p->ld < p->vocab || r0 < 0 || r1 < r0) return -1;
  if (p->dtype != 0 && p->dtype != 1) return -1;
  if (p->n_peaks < 0 || p->n_peaks > 8) return -1;
  return 0;
}

}  // namespace

extern "C" {

// Fill rows [r0, r1) of the student and/or teacher logits on the device.
// zs_row0 / zt_row0 point at row r0 of device buffers with row stride p->ld
// (either may be NULL to skip it); kt_dev holds the per-row teacher-noise
// scale indexed by absolute row.  Asynchronous on `stream`.  Returns 0, or -1
// on a bad argument, or -2 when the launch fails.
int synth_fill_device(const synth_params* p, const float* kt_dev, int64_t r0, int64_t r1,
                      void* zs_row0, void* zt_row0, hipStream_t stream) {
  if (check_params(p, kt_dev, r0, r1)) return -1;
  if (r1 == r0) return 0;
  const int64_t bpr = (p->vocab + kColsPerBlock - 1) / kColsPerBlock;
  const int64_t blocks = bpr * (r1 - r0);
  if (blocks > 0x7FFFFFFFll) return -1;
  if (p->dtype == 0) {
    hipLaunchKernelGGL(fill_kernel<true>, dim3((unsigned)blocks), dim3(kThreads), 0, stream, *p,
                       kt_dev, r0, bpr, zs_row0, zt_row0);
  } else {
    hipLaunchKernelGGL(fill_kernel<false>, dim3((unsigned)blocks), dim3(kThreads), 0, stream, *p,
                       kt_dev, r0, bpr, zs_row0, zt_row0);
  }
  return hipGetLastError() == hipSuccess ? 0 : -2;
}

// Host twin of synth_fill_device: same bits, written to host buffers, rows
// split over n_threads std::threads (<= 0 means one).
int synth_fill_host(const synth_params* p, const float* kt_host, int64_t r0, int64_t r1,
                    void* zs_row0, void* zt_row0, int n_threads) {
  if (check_params(p, kt_host, r0, r1)) return -1;
  const int64_t rows = r1 - r0;
  if (rows == 0) return 0;
  int nt = n_threads < 1 ? 1 : n_threads;
  if ((int64_t)nt > rows) nt = (int)rows;
  std::vector<std::thread> pool;
  for (int i = 0; i < nt; ++i) {
    const int64_t ra = r0 + rows * i / nt;
    const int64_t rb = r0 + rows * (i + 1) / nt;
    pool.emplace_back([=] {
      if (p->dtype == 0)
        fill_rows_host<true>(*p, kt_host, r0, ra, rb, zs_row0, zt_row0);
      else
        fill_rows_host<false>(*p, kt_host, r0, ra, rb, zs_row0, zt_row0);
    });
  }
  for (auto& t : pool) t.join();
  return 0;
}

// Host rows listed in `rows` (n_rows absolute row indices, any order):
// row rows[k] is written at zs_out / zt_out + k * p->ld elements.  Same bits
// as the other fills.  Returns 0 or -1 on a bad argument.
int synth_fill_host_rows(const synth_params* p, const float* kt_host, const int64_t* rows,
                         int64_t n_rows, void* zs_out, void* zt_out, int n_threads) {
  if (check_params(p, kt_host, 0, 0) || n_rows < 0 || (n_rows > 0 && !rows)) return -1;
  if (n_rows == 0) return 0;
  int nt = n_threads < 1 ? 1 : n_threads;
  if ((int64_t)nt > n_rows) nt = (int)n_rows;
  const size_t es = p->dtype == 0 ? 2 : 4;
  std::vector<std::thread> pool;
  for (int i = 0; i < nt; ++i) {
    const int64_t ka = n_rows * i / nt;
    const int64_t kb = n_rows * (i + 1) / nt;
    pool.emplace_back([=] {
      for (int64_t k = ka; k < kb; ++k) {
        char* zs = zs_out ? static_cast<char*>(zs_out) + (size_t)k * (size_t)p->ld * es : nullptr;
        char* zt = zt_out ? static_cast<char*>(zt_out) + (size_t)k * (size_t)p->ld * es : nullptr;
        if (p->dtype == 0)
          fill_rows_host<true>(*p, kt_host, rows[k], rows[k], rows[k] + 1, zs, zt);
        else
          fill_rows_host<false>(*p, kt_host, rows[k], rows[k], rows[k] + 1, zs, zt);
      }
    });
  }
  for (auto& t : pool) t.join();
  return 0;
}

}  // extern "C"
