// Host driver for the spatial-cell arithmetic the statistics kernel runs:
// reads "p rows cols M" lines, prints "r c cell" for position p of a
// rows x cols span on the M x M grid.
#include <cstdio>

#include "grid_cell.h"

int main() {
  int p, rows, cols, M;
  while (std::scanf("%d %d %d %d", &p, &rows, &cols, &M) == 4) {
    int r, c;
    starkv::span_row_col(p, cols, &r, &c);
    const int cell = starkv::grid_cell(r, c, rows, cols, M, (float)M / (float)rows,
                                       (float)M / (float)cols);
    std::printf("%d %d %d\n", r, c, cell);
  }
  return 0;
}
