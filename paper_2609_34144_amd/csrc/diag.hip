// Spectral diagnostics of reconstructed residuals on gfx950 (App. C eq:oracles,
// eq:bandenergy, eq:phaseerror; the relative error e_t of Sec. 3.1
// eq:sensitivity), with PAR's tile and FFT conventions (App. A.2).
//
// diag_tile   grid (tile, channel block of 64, frame); frames that are anchors
//             exit.  Each lane owns one channel of one tile of the skipped frame t
//             and transforms (orthonormal real 2-D DFT, any tile size up to 8x8,
//             runtime loops over per-lane LDS columns) the reference R_t, the
//             reconstruction R_hat_t and the two anchors of t's pair.  It adds up
//             kappa |F_t - F_hat_t|^2 per radial band, kappa |F_t|^2, and the
//             energy-weighted circular distance of the transport phase; it writes
//             the oracle corrections of the linear interpolation
//             (|F_lin| e^{i Arg F_t} and |F_t| e^{i Arg F_lin}, inverted) when
//             asked.  The 64 lanes are summed by a butterfly into one partial per
//             (frame, tile, channel block).
// diag_final  one block per frame: the partials in fixed order (fp64), then e_t,
//             the band fractions and the phase error.
// Not a hot path: clarity over speed (runtime tile sizes, spectra in LDS).
#include "cast_common.h"

namespace cast {

namespace {

constexpr int kLanes = 64;
constexpr int kT = kParMaxTile;            // largest tile edge
constexpr int kNkx = kT / 2 + 1;
constexpr int kSpec = kT * kNkx;           // stored bins of the largest tile
constexpr int kVals = kDiagMaxBands + 3;   // band energies, |F_t|^2, phase sum, weight sum
constexpr float kPi = 3.14159265358979323846f;

struct DiagArgs {
  const float* ref;
  const float* approx;
  const float* theta;      // [n_pairs, n_tiles, tile_h * (tile_w / 2 + 1)] or null
  float* r_phase;
  float* r_mag;
  float* partial;          // [n_frames, n_tiles, n_chblk, kVals]
  long long frame_elems;
  int Hg, Wg, D, tile_h, tile_w, n_tx, n_tiles, n_chblk, n_anchor, n_frames, n_bands;
  float eps;
  double edges[kDiagMaxBands + 1];
  short anchors[kParMaxAnchors];
};

// Per-lane LDS storage: element k of lane l at [k * 64 + l] (conflict-free).
struct Spec {
  float* re;
  float* im;
  __device__ float& r(int k) { return re[k * kLanes + threadIdx.x]; }
  __device__ float& i(int k) { return im[k * kLanes + threadIdx.x]; }
};

// twiddles e^{-2 pi i j / n} for n = 1 .. 8: c[n][j], s[n][j] = cos, sin of 2 pi j / n
struct Tw {
  float c[kT + 1][kT];
  float s[kT + 1][kT];
};

__device__ void load_tile(const float* frame, const DiagArgs& a, int y0, int x0, int hp, int wp,
                          int c, float* x) {
  for (int y = 0; y < hp; ++y)
    for (int xx = 0; xx < wp; ++xx)
      x[(y * wp + xx) * kLanes + threadIdx.x] = frame[((long long)(y0 + y) * a.Wg + x0 + xx) * a.D + c];
}

// Orthonormal forward real 2-D DFT of the lane's tile values x[hp][wp] into F
// (bins ky in [0, hp), kx in [0, wp/2], slot ky * kNkx + kx); t holds the rows.
__device__ void fwd(const float* x, int hp, int wp, const Tw& tw, Spec t, Spec F) {
  const int nkx = wp / 2 + 1;
  for (int y = 0; y < hp; ++y)
    for (int kx = 0; kx < nkx; ++kx) {
      float re = 0.0f, im = 0.0f;
      for (int xx = 0; xx < wp; ++xx) {
        const float v = x[(y * wp + xx) * kLanes + threadIdx.x];
        const int j = (kx * xx) % wp;
        re = fmaf(v, tw.c[wp][j], re);
        im = fmaf(-v, tw.s[wp][j], im);
      }
      t.r(y * kNkx + kx) = re;
      t.i(y * kNkx + kx) = im;
    }
  const float sc = 1.0f / sqrtf((float)(hp * wp));
  for (int kx = 0; kx < nkx; ++kx)
    for (int ky = 0; ky < hp; ++ky) {
      float re = 0.0f, im = 0.0f;
      for (int y = 0; y < hp; ++y) {
        const int j = (ky * y) % hp;
        const float cr = t.r(y * kNkx + kx), ci = t.i(y * kNkx + kx);
        const float c = tw.c[hp][j], s = tw.s[hp][j];   // e^{-i phi} = c - i s
        re += cr * c + ci * s;
        im += ci * c - cr * s;
      }
      F.r(ky * kNkx + kx) = re * sc;
      F.i(ky * kNkx + kx) = im * sc;
    }
}

// Inverse: x[y][x] = (hp wp)^-1/2 sum_{stored bins} kappa Re(F e^{+i phi}), the real
// inverse of the Hermitian spectrum; t holds the column pass.
__device__ void inv(Spec F, int hp, int wp, const Tw& tw, Spec t, float* x) {
  const int nkx = wp / 2 + 1;
  for (int kx = 0; kx < nkx; ++kx)
    for (int y = 0; y < hp; ++y) {
      float re = 0.0f, im = 0.0f;
      for (int ky = 0; ky < hp; ++ky) {
        const int j = (ky * y) % hp;
        const float fr = F.r(ky * kNkx + kx), fi = F.i(ky * kNkx + kx);
        const float c = tw.c[hp][j], s = tw.s[hp][j];   // e^{+i phi} = c + i s
        re += fr * c - fi * s;
        im += fi * c + fr * s;
      }
      t.r(y * kNkx + kx) = re;
      t.i(y * kNkx + kx) = im;
    }
  const float sc = 1.0f / sqrtf((float)(hp * wp));
  for (int y = 0; y < hp; ++y)
    for (int xx = 0; xx < wp; ++xx) {
      float v = 0.0f;
      for (int kx = 0; kx < nkx; ++kx) {
        const int j = (kx * xx) % wp;
        const float kap = (kx == 0 || 2 * kx == wp) ? 1.0f : 2.0f;
        v += kap * (t.r(y * kNkx + kx) * tw.c[wp][j] - t.i(y * kNkx + kx) * tw.s[wp][j]);
      }
      x[(y * wp + xx) * kLanes + threadIdx.x] = v * sc;
    }
}

__device__ void store_tile(float* frame, const DiagArgs& a, int y0, int x0, int hp, int wp, int c,
                           const float* x) {
  for (int y = 0; y < hp; ++y)
    for (int xx = 0; xx < wp; ++xx)
      frame[((long long)(y0 + y) * a.Wg + x0 + xx) * a.D + c] = x[(y * wp + xx) * kLanes + threadIdx.x];
}

__global__ __launch_bounds__(kLanes) void diag_tile_kernel(DiagArgs a) {
  const int tile = blockIdx.x, chb = blockIdx.y, t = blockIdx.z;
  // the pair of frame t (eq:block), or nothing for an anchor
  int j = 0;
  while (j < a.n_anchor && a.anchors[j] < t) ++j;
  if (j < a.n_anchor && a.anchors[j] == t) return;
  const int pr = j == 0 ? 0 : (j == a.n_anchor ? a.n_anchor - 2 : j - 1);
  const int fa = a.anchors[pr], fb = a.anchors[pr + 1];
  const float alpha = (float)(t - fa) / (float)(fb - fa);

  __shared__ Tw tw;
  __shared__ float xs[kT * kT * kLanes];
  __shared__ float s_re[4][kSpec * kLanes], s_im[4][kSpec * kLanes];
  const int lane = threadIdx.x;
  for (int k = lane; k < (kT + 1) * kT; k += kLanes) {
    const int n = k / kT, jj = k % kT;
    float sn = 0.0f, cs = 1.0f;
    if (n > 0) sincospif(2.0f * (float)jj / (float)n, &sn, &cs);
    tw.c[n][jj] = cs;
    tw.s[n][jj] = sn;
  }
  __syncthreads();
  Spec Ft{s_re[0], s_im[0]}, Fo{s_re[1], s_im[1]}, Fl{s_re[2], s_im[2]}, T{s_re[3], s_im[3]};

  const int ty = tile / a.n_tx, tx = tile - (tile / a.n_tx) * a.n_tx;
  const int y0 = ty * a.tile_h, x0 = tx * a.tile_w;
  const int hp = min(a.tile_h, a.Hg - y0), wp = min(a.tile_w, a.Wg - x0), nkx = wp / 2 + 1;
  const int c_raw = chb * kLanes + lane;
  const bool live = c_raw < a.D;
  const int c = live ? c_raw : a.D - 1;
  const float* ref = a.ref;
  // maximum physical radius of the tile's stored bins (for nu)
  double rmax = 0.0;
  for (int ky = 0; ky < hp; ++ky)
    for (int kx = 0; kx < nkx; ++kx) {
      const int kys = 2 * ky <= hp ? ky : ky - hp;
      rmax = fmax(rmax, sqrt((double)kys * kys / ((double)hp * hp) + (double)kx * kx / ((double)wp * wp)));
    }

  float acc[kVals];
  for (int v = 0; v < kVals; ++v) acc[v] = 0.0f;
  // reference and reconstruction: band energies of the error, reference energy
  load_tile(ref + (long long)t * a.frame_elems, a, y0, x0, hp, wp, c, xs);
  fwd(xs, hp, wp, tw, T, Ft);
  load_tile(a.approx + (long long)t * a.frame_elems, a, y0, x0, hp, wp, c, xs);
  fwd(xs, hp, wp, tw, T, Fo);
  for (int ky = 0; ky < hp; ++ky)
    for (int kx = 0; kx < nkx; ++kx) {
      const int b = ky * kNkx + kx;
      const float kap = (kx == 0 || 2 * kx == wp) ? 1.0f : 2.0f;
      const float dr = Ft.r(b) - Fo.r(b), di = Ft.i(b) - Fo.i(b);
      const int kys = 2 * ky <= hp ? ky : ky - hp;
      const double nu = rmax > 0.0 ? sqrt((double)kys * kys / ((double)hp * hp) +
                                          (double)kx * kx / ((double)wp * wp)) / rmax : 0.0;
      int band = 0;
      while (band + 1 < a.n_bands && nu >= a.edges[band + 1]) ++band;
      acc[band] += kap * (dr * dr + di * di);
      acc[kDiagMaxBands] += kap * (Ft.r(b) * Ft.r(b) + Ft.i(b) * Ft.i(b));
    }
  // anchor a: transport phase error; F_lin = (1 - alpha) F_a + alpha F_b
  const bool want_corr = a.r_phase != nullptr || a.r_mag != nullptr;
  if (a.theta != nullptr || want_corr) {
    load_tile(ref + (long long)fa * a.frame_elems, a, y0, x0, hp, wp, c, xs);
    fwd(xs, hp, wp, tw, T, Fo);
    const int nkx_out = a.tile_w / 2 + 1;
    for (int ky = 0; ky < hp; ++ky)
      for (int kx = 0; kx < nkx; ++kx) {
        const int b = ky * kNkx + kx;
        Fl.r(b) = (1.0f - alpha) * Fo.r(b);
        Fl.i(b) = (1.0f - alpha) * Fo.i(b);
        if (a.theta == nullptr) continue;
        const float th = a.theta[((long long)pr * a.n_tiles + tile) * (a.tile_h * nkx_out) + ky * nkx_out + kx];
        const float at2 = Ft.r(b) * Ft.r(b) + Ft.i(b) * Ft.i(b);
        const float aa2 = Fo.r(b) * Fo.r(b) + Fo.i(b) * Fo.i(b);
        if (at2 > 0.0f && aa2 > 0.0f) {
          const float kap = (kx == 0 || 2 * kx == wp) ? 1.0f : 2.0f;
          const float w = kap * at2;
          float x = atan2f(Ft.i(b), Ft.r(b)) - atan2f(Fo.i(b), Fo.r(b)) - alpha * th;
          x = x - 2.0f * kPi * floorf((x + kPi) / (2.0f * kPi));
          acc[kDiagMaxBands + 1] += w * fabsf(x);
          acc[kDiagMaxBands + 2] += w;
        }
      }
  }
  if (want_corr) {
    load_tile(ref + (long long)fb * a.frame_elems, a, y0, x0, hp, wp, c, xs);
    fwd(xs, hp, wp, tw, T, Fo);
    for (int ky = 0; ky < hp; ++ky)
      for (int kx = 0; kx < nkx; ++kx) {
        const int b = ky * kNkx + kx;
        Fl.r(b) += alpha * Fo.r(b);
        Fl.i(b) += alpha * Fo.i(b);
      }
    for (int which = 0; which < 2; ++which) {
      float* dst = which == 0 ? a.r_phase : a.r_mag;
      if (dst == nullptr) continue;
      for (int ky = 0; ky < hp; ++ky)
        for (int kx = 0; kx < nkx; ++kx) {
          const int b = ky * kNkx + kx;
          const float mt = sqrtf(Ft.r(b) * Ft.r(b) + Ft.i(b) * Ft.i(b));
          const float ml = sqrtf(Fl.r(b) * Fl.r(b) + Fl.i(b) * Fl.i(b));
          // modulus of one spectrum, unit phase factor of the other (1 where it vanishes)
          const float m = which == 0 ? ml : mt;
          const float pr_ = which == 0 ? Ft.r(b) : Fl.r(b), pi_ = which == 0 ? Ft.i(b) : Fl.i(b);
          const float pm = which == 0 ? mt : ml;
          Fo.r(b) = pm > 0.0f ? m * (pr_ / pm) : m;
          Fo.i(b) = pm > 0.0f ? m * (pi_ / pm) : 0.0f;
        }
      inv(Fo, hp, wp, tw, T, xs);
      if (live) store_tile(dst + (long long)t * a.frame_elems, a, y0, x0, hp, wp, c, xs);
    }
  }
  // lanes past D add nothing; then the 64 lanes in butterfly order
  for (int v = 0; v < kVals; ++v) {
    float s = live ? acc[v] : 0.0f;
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0)
      a.partial[(((long long)t * a.n_tiles + tile) * a.n_chblk + chb) * kVals + v] = s;
  }
}

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

__global__ __launch_bounds__(kLanes) void diag_final_kernel(FinalArgs a) {
  const int t = blockIdx.x, lane = threadIdx.x;
  bool is_anchor = false;
  for (int j = 0; j < a.n_anchor; ++j) is_anchor |= a.anchors[j] == t;
  double s[kVals];
  for (int v = 0; v < kVals; ++v) s[v] = 0.0;
  if (!is_anchor)
    for (int it = lane; it < a.n_items; it += kLanes)
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

}  // namespace

size_t diag_workspace_bytes(int n_frames, int Hg, int Wg, int D, int tile_h, int tile_w) {
  const long long tiles = (long long)((Hg + tile_h - 1) / tile_h) * ((Wg + tile_w - 1) / tile_w);
  const long long chblk = (D + kLanes - 1) / kLanes;
  return align_up((size_t)(n_frames * tiles * chblk * kVals) * sizeof(float));
}

cast_status_t launch_diag(const float* ref, const float* approx, const float* theta,
                          const int* anchors, int n_anchor, int n_frames, int Hg, int Wg, int D,
                          const cast_diag_params_t& p, float* nrmse_out, float* band_out,
                          float* phase_err_out, float* r_phase_out, float* r_mag_out, void* ws,
                          hipStream_t stream) {
  DiagArgs a{};
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
  a.n_chblk = (D + kLanes - 1) / kLanes;
  a.n_anchor = n_anchor;
  a.n_frames = n_frames;
  a.n_bands = p.n_bands;
  a.eps = p.eps;
  for (int k = 0; k <= p.n_bands; ++k) a.edges[k] = (double)p.band_edges[k];
  for (int j = 0; j < n_anchor; ++j) a.anchors[j] = (short)anchors[j];
  hipLaunchKernelGGL(diag_tile_kernel, dim3(a.n_tiles, a.n_chblk, n_frames), dim3(kLanes), 0, stream, a);
  cast_status_t st = check_launch("diag_tile");
  if (st != CAST_OK) return st;
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
  hipLaunchKernelGGL(diag_final_kernel, dim3(n_frames), dim3(kLanes), 0, stream, f);
  return check_launch("diag_final");
}

}  // namespace cast
