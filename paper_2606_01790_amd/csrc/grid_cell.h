// Spatial cell of a visual token (sec. 3.4, SpatialBin in Eq. MI): a frame
// of rows x cols patch tokens, raster row-major from its span's first token,
// is mapped onto an M x M grid by floor(r*M/rows) and floor(c*M/cols).
// Host and device share this code so that the CPU tests exercise the exact
// arithmetic the statistics kernel runs.
#pragma once

#if defined(__HIPCC__)
#define STARKV_HD __host__ __device__
#else
#define STARKV_HD
#endif

namespace starkv {

// floor(x * M / n) without an integer division, for 0 <= x < n,
// 1 <= M <= 16 and n < 2^27 (so x * M < 2^31).  The quotient is below M,
// so a float estimate m_over_n of M / n good to a few ulps puts x *
// m_over_n within one of it, and one correction step makes it exact.
STARKV_HD inline int scaled_index(int x, int M, int n, float m_over_n) {
  int q = (int)((float)x * m_over_n);
  const int xm = x * M;
  if (q * n > xm) --q;
  else if ((q + 1) * n <= xm) ++q;
  return q;
}

// floor(p / n) for 0 <= p < kSmallQuot and n >= 1, from rn, the reciprocal
// of n to within one ulp: there the estimate p * rn is within one of the
// quotient (n = 1 and 2 have exact reciprocals; for n >= 3 the error is at
// most p / n * 2^-22 < 1/3), and one correction step makes it exact.
constexpr int kSmallQuot = 1 << 22;
STARKV_HD inline int small_quot(int p, int n, float rn) {
  int q = (int)((float)p * rn);
  if (q * n > p) --q;
  else if ((q + 1) * n <= p) ++q;
  return q;
}

// Row and column of position p in a span with `cols` columns: an exact
// integer division (positions reach 2^26, where a float estimate of p/cols
// can be off by more than one).
STARKV_HD inline void span_row_col(int p, int cols, int* r, int* c) {
  *r = p / cols;
  *c = p - *r * cols;
}

// Cell id row*M + col of (r, c) in a rows x cols frame on the M x M grid.
STARKV_HD inline int grid_cell(int r, int c, int rows, int cols, int M, float m_over_rows,
                               float m_over_cols) {
  return scaled_index(r, M, rows, m_over_rows) * M + scaled_index(c, M, cols, m_over_cols);
}

}  // namespace starkv
