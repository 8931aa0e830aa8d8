// Seeded synthetic logits for the turn-KL workloads.
//
// Every value is a pure function of (seed, stream, row, column): the device
// fills full-size batches directly in HBM, and the host regenerates any row
// bit-for-bit to feed the CPU checker.  Both paths come from the single
// per-element routine below, which uses only 64-bit integer hashing, exact
// integer -> double conversion, and IEEE double add, multiply and divide
// (correctly rounded on both sides) with contraction disabled, so host and
// device results are identical.  No library math function is called: the
// logarithm, square root, sine and cosine are written out below from their
// series, so that no platform's math library can make the two sides differ.
//
// Generator: SplitMix64 (Steele, Lea & Flood, "Fast splittable pseudorandom
// number generators", OOPSLA 2014) used in counter mode: output n of a stream
// with key k is mix64(k + (n + 1) * GOLDEN), mix64 being SplitMix64's
// finaliser.  Element n takes outputs 2n and 2n + 1 as two 52-bit uniforms
// and turns them into two independent standard normals with the Box-Muller
// transform (Box & Muller, Ann. Math. Statist. 29, 1958):
//   z1 = sqrt(-2 ln u1) cos(2 pi u2),  z2 = sqrt(-2 ln u1) sin(2 pi u2),
// u1 in [2^-52, 1], so |z| reaches sqrt(104 ln 2) = 8.49 standard deviations.
// z1 drives the student logit, z2 the teacher's noise.
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
  float student_sigma;       // standard deviation of the student logits
  float peak_boost;          // added to both models at the peak columns
  uint32_t shift_threshold;  // teacher peaks re-drawn iff hi32(hash) < this
  uint32_t reserved;
} synth_params;

}  // extern "C"

namespace {

constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

enum : uint64_t {
  kStreamNormals = 0,
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

// ---- double-precision helpers from +, -, *, / only (see the header)

constexpr double kLn2 = 0.69314718055994530942;
constexpr double kPiOver4 = 0.78539816339744830962;

__host__ __device__ inline uint64_t dbits(double x) {
  uint64_t u;
  __builtin_memcpy(&u, &x, 8);
  return u;
}

__host__ __device__ inline double from_bits(uint64_t u) {
  double x;
  __builtin_memcpy(&x, &u, 8);
  return x;
}

// ln x for a normal x > 0: x = m 2^e with m in [sqrt(1/2), sqrt(2)), then
// ln m = 2 atanh(s) = 2 (s + s^3/3 + s^5/5 + ...), s = (m - 1) / (m + 1),
// |s| <= 0.1716; thirteen terms leave a truncation error below 1e-19.
// Branch-free (selects only), so that the host loop vectorises.
__host__ __device__ inline double ln_normal(double x) {
  const uint64_t u = dbits(x);
  const double m0 = from_bits((u & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull);  // [1, 2)
  const bool hi = m0 >= 1.4142135623730951;  // the double nearest sqrt(2)
  const double m = hi ? m0 * 0.5 : m0;
  const int e = (int)((u >> 52) & 0x7FF) - 1023 + (hi ? 1 : 0);
  const double s = (m - 1.0) / (m + 1.0);
  const double s2 = s * s;
  constexpr double kInvOdd[13] = {1.0,        1.0 / 3.0,  1.0 / 5.0,  1.0 / 7.0,  1.0 / 9.0,
                                  1.0 / 11.0, 1.0 / 13.0, 1.0 / 15.0, 1.0 / 17.0, 1.0 / 19.0,
                                  1.0 / 21.0, 1.0 / 23.0, 1.0 / 25.0};
  double p = kInvOdd[12];
#pragma unroll
  for (int k = 11; k >= 0; --k) p = p * s2 + kInvOdd[k];
  return (double)e * kLn2 + 2.0 * (s * p);
}

// sqrt q for q >= 0 (0 for q <= 0): q = m 4^k with m in [1, 4); y ~ 1/sqrt(m)
// from the chord 1 - (m - 1)/6 (exact at m = 1 and 4, within 18% between),
// six Newton steps y <- y (3 - m y^2) / 2 (relative error e -> about 1.5 e^2,
// so the last steps only round), then sqrt q = m y 2^k.
__host__ __device__ inline double sqrt_nonneg(double q) {
  const uint64_t u = dbits(q);
  const int e0 = (int)((u >> 52) & 0x7FF) - 1023;
  const double m0 = from_bits((u & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull);  // [1, 2)
  const bool odd = (e0 & 1) != 0;
  const double m = odd ? m0 * 2.0 : m0;  // [1, 4)
  const int e = odd ? e0 - 1 : e0;
  double y = 1.0 - (m - 1.0) * (1.0 / 6.0);
#pragma unroll
  for (int it = 0; it < 6; ++it) y = y * (1.5 - (0.5 * m) * (y * y));
  const double r = (m * y) * from_bits((uint64_t)(e / 2 + 1023) << 52);
  return q > 0.0 ? r : 0.0;
}

// cos a and sin a for a in [0, pi/4], Taylor series by Horner in a^2 (the
// first omitted terms, a^18/18! and a^19/19!, are below 2e-18).
__host__ __device__ inline void sincos_octant(double a, double& c, double& s) {
  constexpr double kCos[9] = {1.0,
                              -1.0 / 2.0,
                              1.0 / 24.0,
                              -1.0 / 720.0,
                              1.0 / 40320.0,
                              -1.0 / 3628800.0,
                              1.0 / 479001600.0,
                              -1.0 / 87178291200.0,
                              1.0 / 20922789888000.0};
  constexpr double kSin[9] = {1.0,
                              -1.0 / 6.0,
                              1.0 / 120.0,
                              -1.0 / 5040.0,
                              1.0 / 362880.0,
                              -1.0 / 39916800.0,
                              1.0 / 6227020800.0,
                              -1.0 / 1307674368000.0,
                              1.0 / 355687428096000.0};
  const double a2 = a * a;
  double pc = kCos[8], ps = kSin[8];
#pragma unroll
  for (int k = 7; k >= 0; --k) {
    pc = pc * a2 + kCos[k];
    ps = ps * a2 + kSin[k];
  }
  c = pc;
  s = a * ps;
}

// (cos 2 pi v, sin 2 pi v) for v in [0, 1): octant k = floor(8 v), reduced
// to an angle a in [0, pi/4] measured from the nearer octant edge.  Octants
// 1, 2, 5, 6 swap cosine and sine; the cosine is negative in octants 2..5,
// the sine in 4..7.
__host__ __device__ inline void cos_sin_turn(double v, double& cv, double& sv) {
  const double t = v * 8.0;  // exact
  const int k = (int)t;
  const double f = t - (double)k;  // exact, [0, 1)
  const double a = ((k & 1) ? (1.0 - f) : f) * kPiOver4;
  double c, s;
  sincos_octant(a, c, s);
  const bool swap = ((k + 1) & 2) != 0;
  const double x = swap ? s : c;
  const double y = swap ? c : s;
  cv = ((k + 2) & 4) ? -x : x;
  sv = (k & 4) ? -y : y;
}

// Two independent standard normals from two SplitMix64 outputs (Box-Muller):
// u1 = 2 - (1 + 52 bits) in [2^-52, 1] and u2 = (1 + 52 bits) - 1 in [0, 1),
// both exact.
__host__ __device__ inline void normal_pair(uint64_t x1, uint64_t x2, double& z1, double& z2) {
  const double u1 = 2.0 - from_bits(0x3FF0000000000000ull | (x1 >> 12));
  const double u2 = from_bits(0x3FF0000000000000ull | (x2 >> 12)) - 1.0;
  const double r = sqrt_nonneg(-2.0 * ln_normal(u1));
  double c, s;
  cos_sin_turn(u2, c, s);
  z1 = r * c;
  z2 = r * s;
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

// The per-element recipe.  Student = sigma_s z1 (+ boost at its peaks);
// teacher = (sigma_s z1 + sigma_t z2) (+ boost at its peaks), the two terms
// rounded to fp32 and added in fp32; each logit is rounded once to bf16.
__host__ __device__ inline void element(const synth_params& p, uint64_t key, float teacher_sigma,
                                        const RowPeaks& pk, int64_t row, int64_t col,
                                        float& s_out, float& t_out) {
  const uint64_t n = (uint64_t)row * (uint64_t)p.vocab + (uint64_t)col;
  double z1, z2;
  normal_pair(splitmix_at(key, 2 * n), splitmix_at(key, 2 * n + 1), z1, z2);
  const float base = (float)(z1 * (double)p.student_sigma);
  const float noise = (float)(z2 * (double)teacher_sigma);
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
  const uint64_t key = stream_key(p.seed, kStreamNormals);
  const float tsc = kt[row];
  const int64_t c0 = cb * kColsPerBlock + (int64_t)threadIdx.x * kColsPerThread;
  for (int j = 0; j < kColsPerThread; ++j) {
    const int64_t col = c0 + j;
    if (col >= p.vocab) break;
    float s, t;
    element(p, key, tsc, pk, row, col, s, t);
    const int64_t off = rel * p.ld + col;
    if (zs) store<kBf16>(zs, off, s);
    if (zt) store<kBf16>(zt, off, t);
  }
}

// Host rows, in blocks of kHostBlock columns: the SplitMix64 outputs first,
// then the normals (a branch-free loop the compiler vectorises), then the
// scaling, peaks and rounding of element().  Per element the operations are
// those of element(), in the same order, so the bits match the device's.
constexpr int kHostBlock = 256;

template <bool kBf16>
void fill_rows_host(const synth_params& p, const float* kt, int64_t r0, int64_t ra, int64_t rb,
                    void* zs, void* zt) {
  const uint64_t key = stream_key(p.seed, kStreamNormals);
  uint64_t x1[kHostBlock], x2[kHostBlock];
  double z1[kHostBlock], z2[kHostBlock];
  for (int64_t row = ra; row < rb; ++row) {
    RowPeaks pk;
    row_peaks(p, row, pk);
    const float tsc = kt[row];
    for (int64_t c0 = 0; c0 < p.vocab; c0 += kHostBlock) {
      const int nb = (int)(p.vocab - c0 < kHostBlock ? p.vocab - c0 : kHostBlock);
      const uint64_t n0 = (uint64_t)row * (uint64_t)p.vocab + (uint64_t)c0;
      for (int j = 0; j < nb; ++j) {
        x1[j] = splitmix_at(key, 2 * (n0 + j));
        x2[j] = splitmix_at(key, 2 * (n0 + j) + 1);
      }
      for (int j = 0; j < nb; ++j) normal_pair(x1[j], x2[j], z1[j], z2[j]);
      for (int j = 0; j < nb; ++j) {
        const int64_t col = c0 + j;
        const float base = (float)(z1[j] * (double)p.student_sigma);
        const float noise = (float)(z2[j] * (double)tsc);
        float s = base;
        float t = base + noise;
        if (is_peak(pk.student, pk.n, col)) s = s + p.peak_boost;
        if (is_peak(pk.teacher, pk.n, col)) t = t + p.peak_boost;
        const int64_t off = (row - r0) * p.ld + col;
        if (zs) store<kBf16>(zs, off, s);
        if (zt) store<kBf16>(zt, off, t);
      }
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


// The Box-Muller pair that one element draws, for tests of the transform:
// z1, z2 from the SplitMix64 outputs x1, x2 (host code, same routine as the
// fills).
void synth_normal_pair(uint64_t x1, uint64_t x2, double* z1, double* z2) {
  double a, b;
  normal_pair(x1, x2, a, b);
  *z1 = a;
  *z2 = b;
}

// ln, sqrt and (cos, sin) of a full turn as the generator computes them, for
// tests against the platform's library: out[0] = ln(x) (x normal, > 0),
// out[1] = sqrt(x) (x >= 0), out[2], out[3] = cos, sin of 2 pi v (v in [0, 1)).
void synth_math(double x, double v, double* out) {
  out[0] = x > 0.0 ? ln_normal(x) : 0.0;
  out[1] = sqrt_nonneg(x);
  cos_sin_turn(v, out[2], out[3]);
}

}  // extern "C"
