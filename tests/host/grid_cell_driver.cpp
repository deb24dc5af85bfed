// Host driver for the spatial-cell arithmetic the statistics kernel runs.
// Reads "p rows cols M" lines and prints "r c cell ok" for position p of a
// rows x cols span on the M x M grid: (r, c, cell) from the exact integer
// division, and ok = 1 when the kernel's reciprocal-estimate path gives the
// same row, column and cell with every reciprocal one ulp off either way
// (that path runs for positions below kSmallQuot).
// With the argument "quot" it instead checks small_quot exhaustively near
// every multiple of n for n = 1..4096 and at sampled larger n, for
// p < kSmallQuot, and prints the number of mismatches.
#include <cmath>
#include <cstdio>
#include <cstring>

#include "grid_cell.h"

using namespace starkv;

static float rcp_off(int n, int ulps) {
  float r = 1.0f / (float)n;
  for (int k = 0; k < ulps; ++k) r = std::nextafterf(r, 2.0f);
  for (int k = 0; k > ulps; --k) r = std::nextafterf(r, 0.0f);
  return r;
}

static long check_quot(int p, int n) {
  long bad = 0;
  for (int u = -1; u <= 1; ++u) bad += small_quot(p, n, rcp_off(n, u)) != p / n;
  return bad;
}

int main(int argc, char** argv) {
  if (argc > 1 && std::strcmp(argv[1], "quot") == 0) {
    long bad = 0, checked = 0;
    auto near = [&](int n) {
      for (long k = 0; k * n < kSmallQuot; k += (n < 64 ? 1 : 1 + (kSmallQuot / n) / 4096)) {
        for (long dp = -1; dp <= 1; ++dp) {
          const long p = k * n + dp;
          if (p < 0 || p >= kSmallQuot) continue;
          bad += check_quot((int)p, n);
          ++checked;
        }
      }
      for (long p = kSmallQuot - 3; p < kSmallQuot; ++p) { bad += check_quot((int)p, n); ++checked; }
    };
    for (int n = 1; n <= 4096; ++n) near(n);
    for (long n = 4097; n < (1L << 26); n = n * 17 / 16 + 1) near((int)n);
    std::printf("%ld %ld\n", bad, checked);
    return 0;
  }
  int p, rows, cols, M;
  while (std::scanf("%d %d %d %d", &p, &rows, &cols, &M) == 4) {
    int r, c;
    span_row_col(p, cols, &r, &c);
    const int cell = grid_cell(r, c, rows, cols, M, (float)M / (float)rows, (float)M / (float)cols);
    int ok = 1;
    if (p < kSmallQuot) {
      for (int u = -1; u <= 1; ++u) {
        const float rc = rcp_off(cols, u), rr = rcp_off(rows, u);
        const int r2 = small_quot(p, cols, rc);
        const int c2 = p - r2 * cols;
        const int dq = small_quot(1024, cols, rc);
        const int cell2 = grid_cell(r2, c2, rows, cols, M, (float)M * rr, (float)M * rc);
        ok &= r2 == r && c2 == c && dq == 1024 / cols && cell2 == cell;
      }
    }
    std::printf("%d %d %d %d\n", r, c, cell, ok);
  }
  return 0;
}
