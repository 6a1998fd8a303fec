// Fused Phase-Aware Reconstruction kernels for the default 8x8 tiling, one row
// of the (HR, WR) remainder table per translation unit: this file is compiled
// once per bottom-remainder height CAST_PAR_HR in 1..8 (8 = no remainder row).
#include "par_device.h"

#ifndef CAST_PAR_HR
#error "CAST_PAR_HR must be defined (1..8)"
#endif

#define CAST_CAT2(a, b) a##b
#define CAST_CAT(a, b) CAST_CAT2(a, b)

namespace cast {
namespace pardev {

template <int HR, int WR>
static void set_entry(FusedRow& r) {
  r.xspec[WR - 1] = par_xspec_fused<HR, WR>;
  r.recon_w[WR - 1] = par_recon_fused<HR, WR, false, false, false>;
  r.recon_a[WR - 1] = par_recon_fused<HR, WR, true, false, false>;
  r.recon_as[WR - 1] = par_recon_fused<HR, WR, true, true, false>;
  r.inl_w[WR - 1] = par_recon_fused<HR, WR, false, false, true>;
  r.inl_a[WR - 1] = par_recon_fused<HR, WR, true, false, true>;
  r.inl_as[WR - 1] = par_recon_fused<HR, WR, true, true, true>;
}

void CAST_CAT(fused_row_, CAST_PAR_HR)(FusedRow& r) {
  constexpr int HR = CAST_PAR_HR;
  set_entry<HR, 1>(r);
  set_entry<HR, 2>(r);
  set_entry<HR, 3>(r);
  set_entry<HR, 4>(r);
  set_entry<HR, 5>(r);
  set_entry<HR, 6>(r);
  set_entry<HR, 7>(r);
  set_entry<HR, 8>(r);
}

}  // namespace pardev
}  // namespace cast
