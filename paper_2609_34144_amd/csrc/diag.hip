// Spectral diagnostics of reconstructed residuals on gfx950 (App. C eq:oracles,
// eq:bandenergy, eq:phaseerror; the relative error e_t of Sec. 3.1
// eq:sensitivity), with PAR's tile and FFT conventions (App. A.2).
//
// diag_tile   grid (tile, channel block of 256, frame); frames that are anchors
//             exit.  Each thread owns one channel of one tile of the skipped frame
//             t and transforms (orthonormal real 2-D DFT) the reference R_t, the
//             reconstruction R_hat_t, the anchor a of t's pair and the linear
//             interpolation (1 - alpha) R_a + alpha R_b.  It adds up
//             kappa |F_t - F_hat_t|^2 per radial band, kappa |F_t|^2 and the
//             energy-weighted circular distance of the transport phase, and writes
//             the oracle corrections of the linear interpolation
//             (|F_lin| e^{i Arg F_t} and |F_t| e^{i Arg F_lin}, inverted) when
//             asked.  The block sums its 256 threads in a fixed order into one
//             partial per (frame, tile, channel block).
// diag_final  one wave per frame: the partials in fixed order (fp64), then e_t,
//             the band fractions and the phase error.
//
// The tile edges are runtime values (1..8; edge tiles are smaller), the same for
// every thread of a block.  Each transform is a matrix DFT over the largest tile,
// held in registers, with zero rows and columns past the tile; its twiddles come
// from a constant table indexed by the (uniform) edge length, so they are scalar
// operands.  At most two spectra are live at once.
#include "cast_common.h"
#include "fft_tile.h"

namespace cast {

namespace {

constexpr int kDiagThreads = 256;
constexpr int kT = kParMaxTile;            // largest tile edge
constexpr int kNkx = kT / 2 + 1;           // stored columns of the largest tile
constexpr int kBins = kT * kNkx;
constexpr int kVals = kDiagMaxBands + 3;   // band energies, |F_t|^2, phase sum, weight sum
constexpr float kPi = 3.14159265358979323846f;

// cos and sin of 2 pi (k j mod n) / n for n = 1 .. 8 and k, j < 8, rounded from
// double, with the quarter turns exact (so the self-conjugate bins of a real
// tile come out exactly real); entries with k or j >= n meet zero data or give
// bins that are not used.
struct TwTable {
  float c[kT + 1][kT][kT];
  float s[kT + 1][kT][kT];
  constexpr TwTable() : c(), s() {
    for (int n = 1; n <= kT; ++n)
      for (int k = 0; k < kT; ++k)
        for (int j = 0; j < kT; ++j) {
          const int m = (k * j) % n;
          if (4 * m % n == 0) {   // m n / 4 turns: 0, 1/4, 1/2, 3/4
            const int q = 4 * m / n;
            c[n][k][j] = q == 0 ? 1.0f : (q == 2 ? -1.0f : 0.0f);
            s[n][k][j] = q == 1 ? 1.0f : (q == 3 ? -1.0f : 0.0f);
          } else {
            c[n][k][j] = (float)fft::tw_cos(m, n);
            s[n][k][j] = (float)fft::tw_sin(m, n);
          }
        }
  }
};
__constant__ TwTable kTw = TwTable();

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

using Spec = float[kT][kNkx];
using Row = float[kT];

// Orthonormal forward real 2-D DFT of a tile whose row y (zero past wp) is
// produced by row(y, v); rows y >= hp are zero.  Bins ky < hp, kx <= wp/2 of
// (Fr, Fi) are the transform; the others hold finite values of no meaning.
template <class RowFn>
__device__ __forceinline__ void fwd2(RowFn&& row, int hp, int wp, Spec& Fr, Spec& Fi) {
#pragma unroll
  for (int y = 0; y < kT; ++y) {
    Row v;
    if (y < hp) {
      row(y, v);
    } else {
#pragma unroll
      for (int x = 0; x < kT; ++x) v[x] = 0.0f;
    }
#pragma unroll
    for (int kx = 0; kx < kNkx; ++kx) {
      float re = 0.0f, im = 0.0f;
#pragma unroll
      for (int x = 0; x < kT; ++x) {
        re = fmaf(v[x], kTw.c[wp][kx][x], re);
        im = fmaf(-v[x], kTw.s[wp][kx][x], im);
      }
      Fr[y][kx] = re;
      Fi[y][kx] = im;
    }
  }
  const float sc = 1.0f / sqrtf((float)(hp * wp));
#pragma unroll
  for (int kx = 0; kx < kNkx; ++kx) {
    Row cr, ci;
#pragma unroll
    for (int y = 0; y < kT; ++y) { cr[y] = Fr[y][kx]; ci[y] = Fi[y][kx]; }
#pragma unroll
    for (int ky = 0; ky < kT; ++ky) {
      float re = 0.0f, im = 0.0f;
#pragma unroll
      for (int y = 0; y < kT; ++y) {   // (cr + i ci)(c - i s)
        const float c = kTw.c[hp][ky][y], s = kTw.s[hp][ky][y];
        re = fmaf(cr[y], c, fmaf(ci[y], s, re));
        im = fmaf(ci[y], c, fmaf(-cr[y], s, im));
      }
      Fr[ky][kx] = re * sc;
      Fi[ky][kx] = im * sc;
    }
  }
}

// Inverse of the Hermitian spectrum given by its stored bins (zero outside the
// tile's bins): x[y][x] = (hp wp)^-1/2 sum_{stored} kappa Re(F e^{+i phi}).  The
// column pass runs in place; each output row y < hp goes to out(y, v).
template <class OutFn>
__device__ __forceinline__ void inv2(Spec& Fr, Spec& Fi, int hp, int wp, OutFn&& out) {
#pragma unroll
  for (int kx = 0; kx < kNkx; ++kx) {
    Row cr, ci;
#pragma unroll
    for (int ky = 0; ky < kT; ++ky) { cr[ky] = Fr[ky][kx]; ci[ky] = Fi[ky][kx]; }
#pragma unroll
    for (int y = 0; y < kT; ++y) {
      float re = 0.0f, im = 0.0f;
#pragma unroll
      for (int ky = 0; ky < kT; ++ky) {   // (cr + i ci)(c + i s)
        const float c = kTw.c[hp][ky][y], s = kTw.s[hp][ky][y];
        re = fmaf(cr[ky], c, fmaf(-ci[ky], s, re));
        im = fmaf(ci[ky], c, fmaf(cr[ky], s, im));
      }
      Fr[y][kx] = re;
      Fi[y][kx] = im;
    }
  }
  const int nkx = wp / 2 + 1;
  const float sc = 1.0f / sqrtf((float)(hp * wp));
#pragma unroll
  for (int y = 0; y < kT; ++y) {
    if (y >= hp) continue;
    Row v;
#pragma unroll
    for (int x = 0; x < kT; ++x) {
      float acc = 0.0f;
#pragma unroll
      for (int kx = 0; kx < kNkx; ++kx) {
        const float kap = kx >= nkx ? 0.0f : ((kx == 0 || 2 * kx == wp) ? 1.0f : 2.0f);
        acc = fmaf(kap, fmaf(Fr[y][kx], kTw.c[wp][kx][x], -Fi[y][kx] * kTw.s[wp][kx][x]), acc);
      }
      v[x] = acc * sc;
    }
    out(y, v);
  }
}

__global__ __launch_bounds__(kDiagThreads) void diag_tile_kernel(DiagArgs a) {
  const int tile = blockIdx.x, chb = blockIdx.y, t = blockIdx.z;
  // the pair of frame t (eq:block), or nothing for an anchor
  int j = 0;
  while (j < a.n_anchor && a.anchors[j] < t) ++j;
  if (j < a.n_anchor && a.anchors[j] == t) return;
  const int pr = j == 0 ? 0 : (j == a.n_anchor ? a.n_anchor - 2 : j - 1);
  const int fa = a.anchors[pr], fb = a.anchors[pr + 1];
  const float alpha = (float)(t - fa) / (float)(fb - fa);

  const int ty = tile / a.n_tx, tx = tile - (tile / a.n_tx) * a.n_tx;
  const int y0 = ty * a.tile_h, x0 = tx * a.tile_w;
  const int hp = min(a.tile_h, a.Hg - y0), wp = min(a.tile_w, a.Wg - x0), nkx = wp / 2 + 1;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // per-bin weights of the tile (bin b = ky * kNkx + kx): kappa (0 outside the
  // tile's stored bins), and kappa times the indicator of each radial band
  __shared__ float s_kap[kBins];
  __shared__ float s_w[kDiagMaxBands][kBins];
  __shared__ float s_red[kDiagThreads / 64][kVals];
  if (tid < kBins) {
    const int ky = tid / kNkx, kx = tid - (tid / kNkx) * kNkx;
    const bool valid = ky < hp && kx < nkx;
    const float kap = valid ? ((kx == 0 || 2 * kx == wp) ? 1.0f : 2.0f) : 0.0f;
    // maximum physical radius of the tile's stored bins (for nu)
    double rmax = 0.0;
    for (int y = 0; y < hp; ++y)
      for (int x = 0; x < nkx; ++x) {
        const int ys = 2 * y <= hp ? y : y - hp;
        rmax = fmax(rmax, sqrt((double)ys * ys / ((double)hp * hp) + (double)x * x / ((double)wp * wp)));
      }
    const int kys = 2 * ky <= hp ? ky : ky - hp;
    const double nu = rmax > 0.0 ? sqrt((double)kys * kys / ((double)hp * hp) +
                                        (double)kx * kx / ((double)wp * wp)) / rmax : 0.0;
    int band = 0;
    while (band + 1 < a.n_bands && nu >= a.edges[band + 1]) ++band;
    s_kap[tid] = kap;
    for (int v = 0; v < kDiagMaxBands; ++v) s_w[v][tid] = v == band ? kap : 0.0f;
  }
  __syncthreads();

  // the lambdas below capture locals only (capturing the kernel argument by
  // reference would copy it to private memory)
  const float* const ref = a.ref;
  const float* const approx = a.approx;
  float* const r_phase = a.r_phase;
  float* const r_mag = a.r_mag;
  const long long frame_elems = a.frame_elems, Wg = a.Wg, D = a.D;
  const int c_raw = chb * kDiagThreads + tid;
  const bool live = c_raw < a.D;
  const int c = live ? c_raw : a.D - 1;
  // element offset of (y, x) of the tile in frame f, channel c
  auto off = [=](int f, int y, int x) -> long long {
    return (long long)f * frame_elems + ((long long)(y0 + y) * Wg + (x0 + x)) * D + c;
  };
  auto load_row = [=](const float* base, int f, int y, Row& v) {
#pragma unroll
    for (int x = 0; x < kT; ++x) v[x] = x < wp ? __builtin_nontemporal_load(base + off(f, y, x)) : 0.0f;
  };

  float acc[kVals];
#pragma unroll
  for (int v = 0; v < kVals; ++v) acc[v] = 0.0f;

  // F_t, and the error spectrum F_t - F_hat_t: band energies, reference energy
  Spec Tr, Ti, Or, Oi;
  fwd2([&](int y, Row& v) { load_row(ref, t, y, v); }, hp, wp, Tr, Ti);
  fwd2([&](int y, Row& v) { load_row(approx, t, y, v); }, hp, wp, Or, Oi);
#pragma unroll
  for (int ky = 0; ky < kT; ++ky)
#pragma unroll
    for (int kx = 0; kx < kNkx; ++kx) {
      const int b = ky * kNkx + kx;
      const float dr = Tr[ky][kx] - Or[ky][kx], di = Ti[ky][kx] - Oi[ky][kx];
      const float e = fmaf(dr, dr, di * di);
#pragma unroll
      for (int v = 0; v < kDiagMaxBands; ++v) acc[v] = fmaf(s_w[v][b], e, acc[v]);
      acc[kDiagMaxBands] = fmaf(s_kap[b], fmaf(Tr[ky][kx], Tr[ky][kx], Ti[ky][kx] * Ti[ky][kx]),
                                acc[kDiagMaxBands]);
    }

  // anchor a: transport phase error against theta
  if (a.theta != nullptr) {
    fwd2([&](int y, Row& v) { load_row(ref, fa, y, v); }, hp, wp, Or, Oi);
    const int nkx_out = a.tile_w / 2 + 1;
    const float* th_tile = a.theta + ((long long)pr * a.n_tiles + tile) * (a.tile_h * nkx_out);
#pragma unroll
    for (int ky = 0; ky < kT; ++ky)
#pragma unroll
      for (int kx = 0; kx < kNkx; ++kx) {
        if (ky >= hp || kx >= nkx) continue;   // uniform: bins of the tile only
        const float th = th_tile[ky * nkx_out + kx];
        const float at2 = fmaf(Tr[ky][kx], Tr[ky][kx], Ti[ky][kx] * Ti[ky][kx]);
        const float aa2 = fmaf(Or[ky][kx], Or[ky][kx], Oi[ky][kx] * Oi[ky][kx]);
        if (at2 > 0.0f && aa2 > 0.0f) {
          const float w = s_kap[ky * kNkx + kx] * at2;
          float x = atan2f(Ti[ky][kx], Tr[ky][kx]) - atan2f(Oi[ky][kx], Or[ky][kx]) - alpha * th;
          x = x - 2.0f * kPi * floorf((x + kPi) / (2.0f * kPi));
          acc[kDiagMaxBands + 1] = fmaf(w, fabsf(x), acc[kDiagMaxBands + 1]);
          acc[kDiagMaxBands + 2] += w;
        }
      }
  }

  // oracle corrections of the linear interpolation F_lin, the transform of
  // (1 - alpha) R_a + alpha R_b
  if (r_phase != nullptr || r_mag != nullptr) {
    fwd2([&](int y, Row& v) {
      Row vb;
      load_row(ref, fa, y, v);
      load_row(ref, fb, y, vb);
#pragma unroll
      for (int x = 0; x < kT; ++x) v[x] = (1.0f - alpha) * v[x] + alpha * vb[x];
    }, hp, wp, Or, Oi);
    // in place: T <- |F_lin| e^{i Arg F_t}, O <- |F_t| e^{i Arg F_lin} (a vanishing
    // spectrum gives phase factor 1); bins outside the tile are zeroed
#pragma unroll
    for (int ky = 0; ky < kT; ++ky)
#pragma unroll
      for (int kx = 0; kx < kNkx; ++kx) {
        const bool valid = ky < hp && kx < nkx;
        const float mt = sqrtf(fmaf(Tr[ky][kx], Tr[ky][kx], Ti[ky][kx] * Ti[ky][kx]));
        const float ml = sqrtf(fmaf(Or[ky][kx], Or[ky][kx], Oi[ky][kx] * Oi[ky][kx]));
        const float p_re = mt > 0.0f ? ml * (Tr[ky][kx] / mt) : ml;
        const float p_im = mt > 0.0f ? ml * (Ti[ky][kx] / mt) : 0.0f;
        const float m_re = ml > 0.0f ? mt * (Or[ky][kx] / ml) : mt;
        const float m_im = ml > 0.0f ? mt * (Oi[ky][kx] / ml) : 0.0f;
        Tr[ky][kx] = valid ? p_re : 0.0f;
        Ti[ky][kx] = valid ? p_im : 0.0f;
        Or[ky][kx] = valid ? m_re : 0.0f;
        Oi[ky][kx] = valid ? m_im : 0.0f;
      }
    if (r_phase != nullptr)
      inv2(Tr, Ti, hp, wp, [=](int y, const Row& v) {
#pragma unroll
        for (int x = 0; x < kT; ++x)
          if (live && x < wp) r_phase[off(t, y, x)] = v[x];
      });
    if (r_mag != nullptr)
      inv2(Or, Oi, hp, wp, [=](int y, const Row& v) {
#pragma unroll
        for (int x = 0; x < kT; ++x)
          if (live && x < wp) r_mag[off(t, y, x)] = v[x];
      });
  }

  // threads past D add nothing; then the block's 256 threads in a fixed order
#pragma unroll
  for (int v = 0; v < kVals; ++v) {
    float s = live ? acc[v] : 0.0f;
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    if (lane == 0) s_red[wave][v] = s;
  }
  __syncthreads();
  if (tid < kVals) {
    float s = 0.0f;
    for (int w = 0; w < kDiagThreads / 64; ++w) s += s_red[w][tid];
    a.partial[(((long long)t * a.n_tiles + tile) * a.n_chblk + chb) * kVals + tid] = s;
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
  a.n_chblk = (D + kDiagThreads - 1) / kDiagThreads;
  a.n_anchor = n_anchor;
  a.n_frames = n_frames;
  a.n_bands = p.n_bands;
  a.eps = p.eps;
  for (int k = 0; k <= p.n_bands; ++k) a.edges[k] = (double)p.band_edges[k];
  for (int j = 0; j < n_anchor; ++j) a.anchors[j] = (short)anchors[j];
  hipLaunchKernelGGL(diag_tile_kernel, dim3(a.n_tiles, a.n_chblk, n_frames), dim3(kDiagThreads), 0,
                     stream, a);
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
  hipLaunchKernelGGL(diag_final_kernel, dim3(n_frames), dim3(64), 0, stream, f);
  return check_launch("diag_final");
}

}  // namespace cast
