// Spectral-diagnostics and phase-progress tile kernels of one tile height: this
// file is compiled once per height CAST_DIAG_HP in 1..8, for widths 1..8.
#include "diag_device.h"

#ifndef CAST_DIAG_HP
#error "CAST_DIAG_HP must be defined (1..8)"
#endif

#define CAST_CAT2(a, b) a##b
#define CAST_CAT(a, b) CAST_CAT2(a, b)

namespace cast {
namespace diagdev {

void CAST_CAT(diag_row_, CAST_DIAG_HP)(DiagRow& r) {
  constexpr int HP = CAST_DIAG_HP;
  r.k[0] = diag_tile<HP, 1>;
  r.k[1] = diag_tile<HP, 2>;
  r.k[2] = diag_tile<HP, 3>;
  r.k[3] = diag_tile<HP, 4>;
  r.k[4] = diag_tile<HP, 5>;
  r.k[5] = diag_tile<HP, 6>;
  r.k[6] = diag_tile<HP, 7>;
  r.k[7] = diag_tile<HP, 8>;
  r.p[0] = diag_progress<HP, 1>;
  r.p[1] = diag_progress<HP, 2>;
  r.p[2] = diag_progress<HP, 3>;
  r.p[3] = diag_progress<HP, 4>;
  r.p[4] = diag_progress<HP, 5>;
  r.p[5] = diag_progress<HP, 6>;
  r.p[6] = diag_progress<HP, 7>;
  r.p[7] = diag_progress<HP, 8>;
}

}  // namespace diagdev
}  // namespace cast
