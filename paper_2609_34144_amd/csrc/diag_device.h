// Device code of the spectral diagnostics (App. C eq:oracles, eq:bandenergy,
// eq:phaseerror; the relative error e_t of Sec. 3.1 eq:sensitivity), with PAR's
// tile and FFT conventions (App. A.2).
//
// diag_tile<HP, WP>   one tile shape (HP x WP, edges 1..8), grid (tile of the
//             class, channel block of 256, frame); frames that are anchors exit.
//             Each thread owns one channel of one tile of the skipped frame t and
//             transforms (orthonormal real 2-D DFT, register-resident codelets)
//             the reference R_t, the reconstruction R_hat_t, the anchor a of t's
//             pair and the linear interpolation (1 - alpha) R_a + alpha R_b.  It
//             adds up kappa |F_t - F_hat_t|^2 per radial band, kappa |F_t|^2 and
//             the energy-weighted circular distance of the transport phase, and
//             writes the oracle corrections of the linear interpolation
//             (|F_lin| e^{i Arg F_t} and |F_t| e^{i Arg F_lin}, inverted) when
//             asked.  The block sums its 256 threads in a fixed order into one
//             partial per (frame, tile, channel block).
// A tiling has up to four tile shapes (full, right edge, bottom edge, corner):
// one launch each.  The 64 shapes are compiled in eight translation units, one
// per tile height.
#pragma once

#include "cast_common.h"
#include "fft_tile.h"

namespace cast {
namespace diagdev {

constexpr int kDiagThreads = 256;
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
  int ty0, tx0, ntx_c;     // the tile class of this launch: tiles (ty0 + i / ntx_c, tx0 + i % ntx_c)
  float eps;
  double edges[kDiagMaxBands + 1];
  short anchors[kParMaxAnchors];
};

typedef void (*DiagTileFn)(DiagArgs);

struct ProgArgs {
  const float* ref;
  float* p_out;            // [n_frames, n_tiles, tile_h * (tile_w / 2 + 1), D]
  long long frame_elems;
  int Hg, Wg, D, tile_h, tile_w, n_tx, n_tiles;
  int ty0, tx0, ntx_c;     // the tile class of this launch, as in DiagArgs
  short anchors[kParMaxAnchors];
};

typedef void (*DiagProgFn)(ProgArgs);

// Frame-wide buffer resource (a frame is below 4 GB); an element is addressed as
// (lane channel + tile row, in a VGPR) + (column within the tile, uniform, SGPR).
constexpr int kBufDword3 = 0x00020000;   // 32-bit data format, gfx9-family V#
constexpr int kNT = 2;                   // nontemporal cache policy (streaming stores)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t frame_rsrc(const float* base, long long frame,
                                                             long long frame_elems) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base) + frame * frame_elems, 0,
                                           (int)(unsigned)(frame_elems * 4), kBufDword3);
}

// The kernels of one tile height HP, for widths 1..8 (each row of the table is
// compiled in its own translation unit).
struct DiagRow {
  DiagTileFn k[8];
  DiagProgFn p[8];
};
void diag_row_1(DiagRow& r);
void diag_row_2(DiagRow& r);
void diag_row_3(DiagRow& r);
void diag_row_4(DiagRow& r);
void diag_row_5(DiagRow& r);
void diag_row_6(DiagRow& r);
void diag_row_7(DiagRow& r);
void diag_row_8(DiagRow& r);

// Orthonormal forward real 2-D DFT of an HP x WP tile whose row y is produced by
// row(y, v): F[ky][kx], ky < HP, kx <= WP / 2.
template <int HP, int WP, class RowFn>
__device__ __forceinline__ void fwd_tile(RowFn&& row, float (&Fr)[HP][WP / 2 + 1],
                                         float (&Fi)[HP][WP / 2 + 1]) {
  constexpr int NKX = WP / 2 + 1;
#pragma unroll
  for (int y = 0; y < HP; ++y) {
    float v[WP];
    row(y, v);
    float Xr[NKX], Xi[NKX];
    fft::rdft<WP>(v, Xr, Xi);
#pragma unroll
    for (int kx = 0; kx < NKX; ++kx) { Fr[y][kx] = Xr[kx]; Fi[y][kx] = Xi[kx]; }
  }
  const float sc = 1.0f / sqrtf((float)(HP * WP));
#pragma unroll
  for (int kx = 0; kx < NKX; ++kx) {
    float cr[HP], ci[HP];
#pragma unroll
    for (int y = 0; y < HP; ++y) { cr[y] = Fr[y][kx]; ci[y] = Fi[y][kx]; }
    fft::cdft<HP, false>(cr, ci);
#pragma unroll
    for (int ky = 0; ky < HP; ++ky) { Fr[ky][kx] = cr[ky] * sc; Fi[ky][kx] = ci[ky] * sc; }
  }
}

// Inverse of the Hermitian spectrum given by its stored bins: the column
// transforms in place, then each output row y goes to out(y, v) (the real
// inverse of the row, kappa-weighted real parts).
template <int HP, int WP, class OutFn>
__device__ __forceinline__ void inv_tile(float (&Fr)[HP][WP / 2 + 1], float (&Fi)[HP][WP / 2 + 1],
                                         OutFn&& out) {
  constexpr int NKX = WP / 2 + 1;
#pragma unroll
  for (int kx = 0; kx < NKX; ++kx) {
    float cr[HP], ci[HP];
#pragma unroll
    for (int ky = 0; ky < HP; ++ky) { cr[ky] = Fr[ky][kx]; ci[ky] = Fi[ky][kx]; }
    fft::cdft<HP, true>(cr, ci);
#pragma unroll
    for (int y = 0; y < HP; ++y) { Fr[y][kx] = cr[y]; Fi[y][kx] = ci[y]; }
  }
  const float sc = 1.0f / sqrtf((float)(HP * WP));
#pragma unroll
  for (int y = 0; y < HP; ++y) {
    float Xr[NKX], Xi[NKX], v[WP];
#pragma unroll
    for (int kx = 0; kx < NKX; ++kx) { Xr[kx] = Fr[y][kx]; Xi[kx] = Fi[y][kx]; }
    fft::c2r<WP>(Xr, Xi, v);
#pragma unroll
    for (int x = 0; x < WP; ++x) v[x] *= sc;
    out(y, v);
  }
}

template <int HP, int WP>
__global__ __launch_bounds__(kDiagThreads) void diag_tile(DiagArgs a) {
  constexpr int NKX = WP / 2 + 1, NB = HP * NKX;
  const int i_cls = blockIdx.x, chb = blockIdx.y, t = blockIdx.z;
  // the pair of frame t (eq:block), or nothing for an anchor
  int j = 0;
  while (j < a.n_anchor && a.anchors[j] < t) ++j;
  if (j < a.n_anchor && a.anchors[j] == t) return;
  const int pr = j == 0 ? 0 : (j == a.n_anchor ? a.n_anchor - 2 : j - 1);
  const int fa = a.anchors[pr], fb = a.anchors[pr + 1];
  const float alpha = (float)(t - fa) / (float)(fb - fa);

  const int ty = a.ty0 + i_cls / a.ntx_c, tx = a.tx0 + (i_cls - (i_cls / a.ntx_c) * a.ntx_c);
  const int tile = ty * a.n_tx + tx;
  const int y0 = ty * a.tile_h, x0 = tx * a.tile_w;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  // per-bin weights (bin b = ky * NKX + kx): kappa, and kappa times the
  // indicator of each radial band
  __shared__ float s_kap[NB];
  __shared__ float s_w[kDiagMaxBands][NB];
  __shared__ float s_red[kDiagThreads / 64][kVals];
  if (tid < NB) {
    const int ky = tid / NKX, kx = tid - (tid / NKX) * NKX;
    const float kap = (kx == 0 || 2 * kx == WP) ? 1.0f : 2.0f;
    // maximum physical radius of the tile's stored bins (for nu)
    double rmax = 0.0;
    for (int y = 0; y < HP; ++y)
      for (int x = 0; x < NKX; ++x) {
        const int ys = 2 * y <= HP ? y : y - HP;
        rmax = fmax(rmax, sqrt((double)ys * ys / ((double)HP * HP) + (double)x * x / ((double)WP * WP)));
      }
    const int kys = 2 * ky <= HP ? ky : ky - HP;
    const double nu = rmax > 0.0 ? sqrt((double)kys * kys / ((double)HP * HP) +
                                        (double)kx * kx / ((double)WP * WP)) / rmax : 0.0;
    int band = 0;
    while (band + 1 < a.n_bands && nu >= a.edges[band + 1]) ++band;
    s_kap[tid] = kap;
    for (int v = 0; v < kDiagMaxBands; ++v) s_w[v][tid] = v == band ? kap : 0.0f;
  }
  __syncthreads();

  // the lambdas below capture locals only (capturing the kernel argument by
  // reference would copy it to private memory)
  float* const r_phase = a.r_phase;
  float* const r_mag = a.r_mag;
  const int c_raw = chb * kDiagThreads + tid;
  const bool live = c_raw < a.D;
  const int c = live ? c_raw : a.D - 1;
  // byte offsets within a frame: lane channel + tile origin (VGPR), grid row and
  // tile column (uniform)
  const unsigned lane_off = (unsigned)c * 4u + (unsigned)(((long long)y0 * a.Wg + x0) * a.D * 4);
  const unsigned row_bytes = (unsigned)((long long)a.Wg * a.D * 4), col_bytes = (unsigned)a.D * 4u;
  auto load_row = [=](__amdgpu_buffer_rsrc_t r, int y, float (&v)[WP]) {
    const unsigned vo = lane_off + (unsigned)y * row_bytes;
#pragma unroll
    for (int x = 0; x < WP; ++x)
      v[x] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)vo, (int)(x * col_bytes), 0));
  };
  auto store_row = [=](__amdgpu_buffer_rsrc_t r, int y, const float (&v)[WP]) {
    const unsigned vo = lane_off + (unsigned)y * row_bytes;
#pragma unroll
    for (int x = 0; x < WP; ++x)
      __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v[x]), r, (int)vo, (int)(x * col_bytes), kNT);
  };
  const __amdgpu_buffer_rsrc_t r_ref_t = frame_rsrc(a.ref, t, a.frame_elems);
  const __amdgpu_buffer_rsrc_t r_app_t = frame_rsrc(a.approx, t, a.frame_elems);
  const __amdgpu_buffer_rsrc_t r_ref_a = frame_rsrc(a.ref, fa, a.frame_elems);
  const __amdgpu_buffer_rsrc_t r_ref_b = frame_rsrc(a.ref, fb, a.frame_elems);

  float acc[kVals];
#pragma unroll
  for (int v = 0; v < kVals; ++v) acc[v] = 0.0f;

  // F_t, and the error spectrum F_t - F_hat_t: band energies, reference energy
  float Tr[HP][NKX], Ti[HP][NKX], Or[HP][NKX], Oi[HP][NKX];
  fwd_tile<HP, WP>([&](int y, float (&v)[WP]) { load_row(r_ref_t, y, v); }, Tr, Ti);
  fwd_tile<HP, WP>([&](int y, float (&v)[WP]) { load_row(r_app_t, y, v); }, Or, Oi);
#pragma unroll
  for (int ky = 0; ky < HP; ++ky)
#pragma unroll
    for (int kx = 0; kx < NKX; ++kx) {
      const int b = ky * NKX + kx;
      const float dr = Tr[ky][kx] - Or[ky][kx], di = Ti[ky][kx] - Oi[ky][kx];
      const float e = fmaf(dr, dr, di * di);
#pragma unroll
      for (int v = 0; v < kDiagMaxBands; ++v) acc[v] = fmaf(s_w[v][b], e, acc[v]);
      acc[kDiagMaxBands] = fmaf(s_kap[b], fmaf(Tr[ky][kx], Tr[ky][kx], Ti[ky][kx] * Ti[ky][kx]),
                                acc[kDiagMaxBands]);
    }

  // anchor a: transport phase error against theta
  if (a.theta != nullptr) {
    fwd_tile<HP, WP>([&](int y, float (&v)[WP]) { load_row(r_ref_a, y, v); }, Or, Oi);
    const int nkx_out = a.tile_w / 2 + 1;
    const float* th_tile = a.theta + ((long long)pr * a.n_tiles + tile) * (a.tile_h * nkx_out);
#pragma unroll
    for (int ky = 0; ky < HP; ++ky)
#pragma unroll
      for (int kx = 0; kx < NKX; ++kx) {
        const float th = th_tile[ky * nkx_out + kx];
        const float at2 = fmaf(Tr[ky][kx], Tr[ky][kx], Ti[ky][kx] * Ti[ky][kx]);
        const float aa2 = fmaf(Or[ky][kx], Or[ky][kx], Oi[ky][kx] * Oi[ky][kx]);
        // Arg F_t - Arg F_a = Arg(F_t conj F_a) modulo 2 pi, which the wrap removes
        const float zr = fmaf(Tr[ky][kx], Or[ky][kx], Ti[ky][kx] * Oi[ky][kx]);
        const float zi = fmaf(Ti[ky][kx], Or[ky][kx], -Tr[ky][kx] * Oi[ky][kx]);
        const float w = at2 > 0.0f && aa2 > 0.0f ? ((kx == 0 || 2 * kx == WP) ? 1.0f : 2.0f) * at2 : 0.0f;
        float x = atan2f(zi, zr) - alpha * th;
        x = x - 2.0f * kPi * floorf((x + kPi) * (0.5f / kPi));
        acc[kDiagMaxBands + 1] = fmaf(w, fabsf(x), acc[kDiagMaxBands + 1]);
        acc[kDiagMaxBands + 2] += w;
      }
  }

  // oracle corrections of the linear interpolation F_lin, the transform of
  // (1 - alpha) R_a + alpha R_b
  if (r_phase != nullptr || r_mag != nullptr) {
    fwd_tile<HP, WP>([&](int y, float (&v)[WP]) {
      float vb[WP];
      load_row(r_ref_a, y, v);
      load_row(r_ref_b, y, vb);
#pragma unroll
      for (int x = 0; x < WP; ++x) v[x] = (1.0f - alpha) * v[x] + alpha * vb[x];
    }, Or, Oi);
    // in place: T <- |F_lin| e^{i Arg F_t}, O <- |F_t| e^{i Arg F_lin} (a vanishing
    // spectrum gives phase factor 1)
#pragma unroll
    for (int ky = 0; ky < HP; ++ky)
#pragma unroll
      for (int kx = 0; kx < NKX; ++kx) {
        const float mt = sqrtf(fmaf(Tr[ky][kx], Tr[ky][kx], Ti[ky][kx] * Ti[ky][kx]));
        const float ml = sqrtf(fmaf(Or[ky][kx], Or[ky][kx], Oi[ky][kx] * Oi[ky][kx]));
        // ratios of moduli (one reciprocal each, to about 1 ulp)
        const float rt = mt > 0.0f ? ml * __builtin_amdgcn_rcpf(mt) : 0.0f;
        const float rl = ml > 0.0f ? mt * __builtin_amdgcn_rcpf(ml) : 0.0f;
        const float p_re = mt > 0.0f ? rt * Tr[ky][kx] : ml;
        const float p_im = rt * Ti[ky][kx];
        const float m_re = ml > 0.0f ? rl * Or[ky][kx] : mt;
        const float m_im = rl * Oi[ky][kx];
        Tr[ky][kx] = p_re;
        Ti[ky][kx] = p_im;
        Or[ky][kx] = m_re;
        Oi[ky][kx] = m_im;
      }
    if (r_phase != nullptr) {
      const __amdgpu_buffer_rsrc_t r = frame_rsrc(r_phase, t, a.frame_elems);
      inv_tile<HP, WP>(Tr, Ti, [&](int y, const float (&v)[WP]) { if (live) store_row(r, y, v); });
    }
    if (r_mag != nullptr) {
      const __amdgpu_buffer_rsrc_t r = frame_rsrc(r_mag, t, a.frame_elems);
      inv_tile<HP, WP>(Or, Oi, [&](int y, const float (&v)[WP]) { if (live) store_row(r, y, v); });
    }
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

// Phase progress (App. C eq:phase_progress) of one tile shape: grid (tile of the
// class, channel block of 256, anchor pair (a, b)).  Each thread owns one channel
// of one tile and walks the frames a..b twice.  Frame by frame it transforms the
// tile, takes the phase Arg F_t of every stored bin and unwraps it along the
// frames, u_t = u_{t-1} + wrap_[-pi,pi)(Arg F_t - Arg F_{t-1}) with u_a = 0; the
// first walk ends with the displacement u_b, the second stores u_t / u_b for the
// interior frames.  Anchor frames, frames outside the pairs and slots past a
// smaller tile's bins are not written.
template <int HP, int WP>
__global__ __launch_bounds__(kDiagThreads) void diag_progress(ProgArgs a) {
  constexpr int NKX = WP / 2 + 1;
  const int i_cls = blockIdx.x, chb = blockIdx.y, pr = blockIdx.z;
  const int fa = a.anchors[pr], fb = a.anchors[pr + 1];
  const int ty = a.ty0 + i_cls / a.ntx_c, tx = a.tx0 + (i_cls - (i_cls / a.ntx_c) * a.ntx_c);
  const int tile = ty * a.n_tx + tx;
  const int y0 = ty * a.tile_h, x0 = tx * a.tile_w;
  const int c_raw = chb * kDiagThreads + (int)threadIdx.x;
  const bool live = c_raw < a.D;
  const int c = live ? c_raw : a.D - 1;
  const unsigned lane_off = (unsigned)c * 4u + (unsigned)(((long long)y0 * a.Wg + x0) * a.D * 4);
  const unsigned row_bytes = (unsigned)((long long)a.Wg * a.D * 4), col_bytes = (unsigned)a.D * 4u;
  const float* const ref = a.ref;
  const long long frame_elems = a.frame_elems;
  auto phases = [&](int t, float (&ph)[HP][NKX]) {
    const __amdgpu_buffer_rsrc_t r = frame_rsrc(ref, t, frame_elems);
    float Fr[HP][NKX], Fi[HP][NKX];
    fwd_tile<HP, WP>([&](int y, float (&v)[WP]) {
      const unsigned vo = lane_off + (unsigned)y * row_bytes;
#pragma unroll
      for (int x = 0; x < WP; ++x)
        v[x] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)vo, (int)(x * col_bytes), 0));
    }, Fr, Fi);
#pragma unroll
    for (int ky = 0; ky < HP; ++ky)
#pragma unroll
      for (int kx = 0; kx < NKX; ++kx) ph[ky][kx] = atan2f(Fi[ky][kx], Fr[ky][kx]);
  };
  auto wrap = [](float x) { return x - 2.0f * kPi * floorf((x + kPi) * (0.5f / kPi)); };
  float prev[HP][NKX], u[HP][NKX], den[HP][NKX];
  for (int pass = 0; pass < 2; ++pass) {
    phases(fa, prev);
#pragma unroll
    for (int ky = 0; ky < HP; ++ky)
#pragma unroll
      for (int kx = 0; kx < NKX; ++kx) u[ky][kx] = 0.0f;
    const int t_end = pass == 0 ? fb : fb - 1;
    for (int t = fa + 1; t <= t_end; ++t) {
      float ph[HP][NKX];
      phases(t, ph);
#pragma unroll
      for (int ky = 0; ky < HP; ++ky)
#pragma unroll
        for (int kx = 0; kx < NKX; ++kx) {
          u[ky][kx] += wrap(ph[ky][kx] - prev[ky][kx]);
          prev[ky][kx] = ph[ky][kx];
        }
      if (pass == 1 && live) {
        const int nkx_out = a.tile_w / 2 + 1;
        float* dst = a.p_out + ((long long)t * a.n_tiles + tile) * (long long)(a.tile_h * nkx_out) * a.D + c;
#pragma unroll
        for (int ky = 0; ky < HP; ++ky)
#pragma unroll
          for (int kx = 0; kx < NKX; ++kx)
            __builtin_nontemporal_store(u[ky][kx] / den[ky][kx], dst + (long long)(ky * nkx_out + kx) * a.D);
      }
    }
    if (pass == 0) {
#pragma unroll
      for (int ky = 0; ky < HP; ++ky)
#pragma unroll
        for (int kx = 0; kx < NKX; ++kx) den[ky][kx] = u[ky][kx];
    }
  }
}

}  // namespace diagdev
}  // namespace cast
