// Spectral diagnostics of reconstructed residuals (App. C eq:oracles,
// eq:bandenergy, eq:phaseerror; the relative error e_t of Sec. 3.1
// eq:sensitivity): the launches, and the per-frame reduction.
//
// diag_tile<HP, WP>  (diag_device.h) one launch per tile shape of the tiling,
//             writing one partial per (frame, tile, channel block of 256).
// diag_final  one wave per frame: the partials in fixed order (fp64), then e_t,
//             the band fractions and the phase error.
// diag_progress<HP, WP>  (diag_device.h) the phase progress of every coefficient,
//             one launch per tile shape.
#include "diag_device.h"

namespace cast {

namespace {

using diagdev::kDiagThreads;
using diagdev::kVals;

struct FinalArgs {
  const float* partial;
  float* nrmse_out;
  float* band_out;
  float* phase_err_out;
  int n_items;             // n_tiles * n_chblk
  int n_bands;
  float eps;
  short anchors[kParMaxAnchors];
  int n_anchor;
};

__global__ __launch_bounds__(64) void diag_final_kernel(FinalArgs a) {
  const int t = blockIdx.x, lane = threadIdx.x;
  bool is_anchor = false;
  for (int j = 0; j < a.n_anchor; ++j) is_anchor |= a.anchors[j] == t;
  double s[kVals];
  for (int v = 0; v < kVals; ++v) s[v] = 0.0;
  if (!is_anchor)
    for (int it = lane; it < a.n_items; it += 64)
      for (int v = 0; v < kVals; ++v) s[v] += (double)a.partial[((long long)t * a.n_items + it) * kVals + v];
  for (int v = 0; v < kVals; ++v)
    for (int o = 32; o > 0; o >>= 1) s[v] += __shfl_xor(s[v], o);
  if (lane != 0) return;
  double err = 0.0;
  for (int k = 0; k < a.n_bands; ++k) err += s[k];
  const double eps = (double)a.eps;
  if (a.nrmse_out) a.nrmse_out[t] = is_anchor ? 0.0f : (float)(sqrt(err) / (sqrt(s[kDiagMaxBands]) + eps));
  if (a.band_out)
    for (int k = 0; k < a.n_bands; ++k)
      a.band_out[(long long)t * a.n_bands + k] = is_anchor ? 0.0f : (float)(s[k] / (err + eps));
  if (a.phase_err_out)
    a.phase_err_out[t] = is_anchor ? 0.0f : (float)(s[kDiagMaxBands + 1] / (s[kDiagMaxBands + 2] + eps));
}

const diagdev::DiagRow& diag_row(int hp) {
  static const diagdev::DiagRow* rows = [] {
    static diagdev::DiagRow r[8];
    diagdev::diag_row_1(r[0]);
    diagdev::diag_row_2(r[1]);
    diagdev::diag_row_3(r[2]);
    diagdev::diag_row_4(r[3]);
    diagdev::diag_row_5(r[4]);
    diagdev::diag_row_6(r[5]);
    diagdev::diag_row_7(r[6]);
    diagdev::diag_row_8(r[7]);
    return r;
  }();
  return rows[hp - 1];
}

}  // namespace

size_t diag_workspace_bytes(int n_frames, int Hg, int Wg, int D, int tile_h, int tile_w) {
  const long long tiles = (long long)((Hg + tile_h - 1) / tile_h) * ((Wg + tile_w - 1) / tile_w);
  const long long chblk = (D + kDiagThreads - 1) / kDiagThreads;
  return align_up((size_t)(n_frames * tiles * chblk * kVals) * sizeof(float));
}

cast_status_t launch_diag(const float* ref, const float* approx, const float* theta,
                          const int* anchors, int n_anchor, int n_frames, int Hg, int Wg, int D,
                          const cast_diag_params_t& p, float* nrmse_out, float* band_out,
                          float* phase_err_out, float* r_phase_out, float* r_mag_out, void* ws,
                          hipStream_t stream) {
  diagdev::DiagArgs a{};
  a.ref = ref;
  a.approx = approx;
  a.theta = theta;
  a.r_phase = r_phase_out;
  a.r_mag = r_mag_out;
  a.partial = static_cast<float*>(ws);
  a.frame_elems = (long long)Hg * Wg * D;
  a.Hg = Hg;
  a.Wg = Wg;
  a.D = D;
  a.tile_h = p.tile_h;
  a.tile_w = p.tile_w;
  a.n_tx = (Wg + p.tile_w - 1) / p.tile_w;
  a.n_tiles = a.n_tx * ((Hg + p.tile_h - 1) / p.tile_h);
  a.n_chblk = (D + kDiagThreads - 1) / kDiagThreads;
  a.n_anchor = n_anchor;
  a.n_frames = n_frames;
  a.n_bands = p.n_bands;
  a.eps = p.eps;
  for (int k = 0; k <= p.n_bands; ++k) a.edges[k] = (double)p.band_edges[k];
  for (int j = 0; j < n_anchor; ++j) a.anchors[j] = (short)anchors[j];
  // the tile classes: full tiles, right edge column, bottom edge row, corner
  const int th = p.tile_h, tw = p.tile_w;
  const int nfy = Hg / th, hr = Hg % th, nfx = Wg / tw, wr = Wg % tw;
  struct Cls { int ty0, tx0, nty, ntx, hp, wp; } cls[4];
  int ncls = 0;
  if (nfy > 0 && nfx > 0) cls[ncls++] = {0, 0, nfy, nfx, th, tw};
  if (nfy > 0 && wr > 0) cls[ncls++] = {0, nfx, nfy, 1, th, wr};
  if (hr > 0 && nfx > 0) cls[ncls++] = {nfy, 0, 1, nfx, hr, tw};
  if (hr > 0 && wr > 0) cls[ncls++] = {nfy, nfx, 1, 1, hr, wr};
  for (int k = 0; k < ncls; ++k) {
    a.ty0 = cls[k].ty0;
    a.tx0 = cls[k].tx0;
    a.ntx_c = cls[k].ntx;
    hipLaunchKernelGGL(diag_row(cls[k].hp).k[cls[k].wp - 1], dim3(cls[k].nty * cls[k].ntx, a.n_chblk, n_frames),
                       dim3(kDiagThreads), 0, stream, a);
    cast_status_t st = check_launch("diag_tile");
    if (st != CAST_OK) return st;
  }
  FinalArgs f{};
  f.partial = a.partial;
  f.nrmse_out = nrmse_out;
  f.band_out = band_out;
  f.phase_err_out = theta != nullptr ? phase_err_out : nullptr;
  f.n_items = a.n_tiles * a.n_chblk;
  f.n_bands = p.n_bands;
  f.eps = p.eps;
  for (int j = 0; j < n_anchor; ++j) f.anchors[j] = (short)anchors[j];
  f.n_anchor = n_anchor;
  hipLaunchKernelGGL(diag_final_kernel, dim3(n_frames), dim3(64), 0, stream, f);
  return check_launch("diag_final");
}

cast_status_t launch_phase_progress(const float* ref, const int* anchors, int n_anchor, int Hg,
                                    int Wg, int D, int tile_h, int tile_w, float* p_out,
                                    hipStream_t stream) {
  diagdev::ProgArgs a{};
  a.ref = ref;
  a.p_out = p_out;
  a.frame_elems = (long long)Hg * Wg * D;
  a.Hg = Hg;
  a.Wg = Wg;
  a.D = D;
  a.tile_h = tile_h;
  a.tile_w = tile_w;
  a.n_tx = (Wg + tile_w - 1) / tile_w;
  a.n_tiles = a.n_tx * ((Hg + tile_h - 1) / tile_h);
  for (int j = 0; j < n_anchor; ++j) a.anchors[j] = (short)anchors[j];
  const int n_chblk = (D + kDiagThreads - 1) / kDiagThreads;
  const int nfy = Hg / tile_h, hr = Hg % tile_h, nfx = Wg / tile_w, wr = Wg % tile_w;
  struct Cls { int ty0, tx0, nty, ntx, hp, wp; } cls[4];
  int ncls = 0;
  if (nfy > 0 && nfx > 0) cls[ncls++] = {0, 0, nfy, nfx, tile_h, tile_w};
  if (nfy > 0 && wr > 0) cls[ncls++] = {0, nfx, nfy, 1, tile_h, wr};
  if (hr > 0 && nfx > 0) cls[ncls++] = {nfy, 0, 1, nfx, hr, tile_w};
  if (hr > 0 && wr > 0) cls[ncls++] = {nfy, nfx, 1, 1, hr, wr};
  for (int k = 0; k < ncls; ++k) {
    a.ty0 = cls[k].ty0;
    a.tx0 = cls[k].tx0;
    a.ntx_c = cls[k].ntx;
    hipLaunchKernelGGL(diag_row(cls[k].hp).p[cls[k].wp - 1],
                       dim3(cls[k].nty * cls[k].ntx, n_chblk, n_anchor - 1), dim3(kDiagThreads), 0,
                       stream, a);
    cast_status_t st = check_launch("diag_progress");
    if (st != CAST_OK) return st;
  }
  return CAST_OK;
}

}  // namespace cast
