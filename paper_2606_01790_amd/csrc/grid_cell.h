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
// so the float estimate is within one of it and one correction step makes
// it exact.
STARKV_HD inline int scaled_index(int x, int M, int n, float m_over_n) {
  int q = (int)((float)x * m_over_n);
  const int xm = x * M;
  if (q * n > xm) --q;
  else if ((q + 1) * n <= xm) ++q;
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
