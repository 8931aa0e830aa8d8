/*
 * Runs the oracle's per-row routine (oracle/rows.c) under AddressSanitizer
 * and UndefinedBehaviorSanitizer.  Test infrastructure: built and run only
 * by tests/test_sanitizers.py.
 *
 * usage: rows_driver IN OUT
 *   IN : int64 dtype, rows, vocab, threads; then the student rows and the
 *        teacher rows, rows * vocab elements each (uint16 bf16 patterns,
 *        float32 or float64 by dtype 0 / 1 / 2)
 *   OUT: float64 kl[rows], lse[rows][2], grad[rows][vocab]
 * Exit status 0 on success, 2 on a usage or file error, 3 when oracle_rows
 * fails.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_rows(const void* zs, int64_t ld_s, const void* zt, int64_t ld_t, int dtype,
                int64_t rows, int64_t vocab, double* kl, double* grad, int64_t ld_g,
                double* lse, int n_threads);

static int read_all(FILE* f, void* p, size_t n) { return fread(p, 1, n, f) == n; }

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 2;
  int64_t hdr[4];
  if (!read_all(in, hdr, sizeof hdr)) return 2;
  const int dtype = (int)hdr[0];
  const int64_t rows = hdr[1], vocab = hdr[2];
  const size_t es = dtype == 0 ? 2 : dtype == 1 ? 4 : 8;
  const size_t n = (size_t)(rows * vocab);
  void* zs = malloc(n * es);
  void* zt = malloc(n * es);
  double* kl = malloc((size_t)rows * sizeof(double));
  double* lse = malloc((size_t)rows * 2 * sizeof(double));
  double* g = malloc(n * sizeof(double));
  if (!zs || !zt || !kl || !lse || !g) return 2;
  if (!read_all(in, zs, n * es) || !read_all(in, zt, n * es)) return 2;
  fclose(in);
  if (oracle_rows(zs, vocab, zt, vocab, dtype, rows, vocab, kl, g, vocab, lse, (int)hdr[3]) != 0)
    return 3;
  FILE* out = fopen(argv[2], "wb");
  if (!out) return 2;
  fwrite(kl, sizeof(double), (size_t)rows, out);
  fwrite(lse, sizeof(double), (size_t)rows * 2, out);
  fwrite(g, sizeof(double), n, out);
  fclose(out);
  free(zs);
  free(zt);
  free(kl);
  free(lse);
  free(g);
  return 0;
}
