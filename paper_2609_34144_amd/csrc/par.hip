// Phase-Aware Reconstruction on gfx950 (Sec. 4.3; App. A.2; eq:block).
//
// Three stream-ordered kernels per call:
//   par_xspec  grid (tile, channel block of 64, anchor pair): every lane owns one
//              channel of one tile, transforms both anchors in registers and
//              writes its per-bin products F_b conj(F_a) and |F_b||F_a|; the 64
//              lanes are summed through LDS in fixed lane order into one partial
//              per (pair, tile, channel block).                        (eq:cross)
//   par_gate   grid (tile, pair): one lane per stored bin sums the partials in
//              fixed order, then computes eta, reliability, theta (representative
//              / mirror / self-conjugate), c_p, nu, g, and the per-target blend
//              coefficients A_t = (1-alpha) e^{i g alpha theta} / (Hp Wp) and
//              B_t = alpha e^{-i g (1-alpha) theta} / (Hp Wp).
//                                              (App. A.2, eq:confidence, eq:gate)
//   par_recon  grid (tile, channel block, pair): every lane re-transforms the two
//              anchors of its pair in registers, then for each target of the pair
//              blends the spectra (eq:fcpasm), inverts and stores / accumulates.
//
// HBM traffic is the anchors (read by xspec and again by recon; the second read
// is usually served by the Infinity Cache) plus the skipped frames written (or
// read and written in accumulate mode).  Tiles are at most 8x8; every tile shape
// (Hp, Wp) in [1,8]^2 has its own fully unrolled code path, selected per block.
#include "cast_common.h"
#include "fft_tile.h"

namespace cast {

namespace {

constexpr int kBins = kParBinsMax;     // 40 stored-bin slots: index ky*5 + kx
constexpr int kNkx = kParNkxMax;       // 5
constexpr int kVals = kBins * 3;       // (Re Z, Im Z, W) per slot
constexpr int kLdsStride = kVals + 1;  // odd row stride: conflict-free LDS transpose
constexpr int kChb = 64;               // channels per block (one wave)

struct ParArgs {
  float* theta_out;
  float* gate_out;
  float* conf_out;
  long long frame_elems;  // Hg * Wg * D
  int n_frames, Hg, Wg, D;
  int tile_h, tile_w, n_tx, n_tiles;
  int n_anchor, n_chblk, bins_out;
  float tau_low, tau_high, q, T, eta_rel, eta_abs, eps;
  int gate_mode, accumulate;
  short anchors[kParMaxAnchors];
};

struct TileGeom {
  int y0, x0, hp, wp;
};

__device__ __forceinline__ TileGeom tile_geom(const ParArgs& a, int tile) {
  TileGeom g;
  int ty = tile / a.n_tx, tx = tile - ty * a.n_tx;
  g.y0 = ty * a.tile_h;
  g.x0 = tx * a.tile_w;
  g.hp = min(a.tile_h, a.Hg - g.y0);
  g.wp = min(a.tile_w, a.Wg - g.x0);
  return g;
}

// Tiles of one shape form a rectangle in tile coordinates (the interior, the
// right edge column, the bottom edge row, the corner); a launch covers one.
struct TileClass {
  int ty0, tx0, ntx;
};

__device__ __forceinline__ int class_tile(const ParArgs& a, const TileClass& k, int b) {
  const int r = b / k.ntx;
  return (k.ty0 + r) * a.n_tx + k.tx0 + (b - r * k.ntx);
}

// Frame-wide buffer resource: every element access is (lane channel offset in a
// VGPR) + (token offset, uniform across the wave, in an SGPR); accesses outside
// the frame return 0 / are dropped by the hardware range check.
constexpr int kBufDword3 = 0x00020000;   // 32-bit data format, gfx9-family V#
constexpr int kNT = 2;                   // nontemporal cache policy (streaming stores)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t frame_rsrc(const float* base, long long frame,
                                                             long long frame_elems) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base) + frame * frame_elems, 0,
                                           (int)(unsigned)(frame_elems * 4), kBufDword3);
}
__device__ __forceinline__ float buf_ld(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0));
}
template <int AUX>
__device__ __forceinline__ void buf_st(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff,
                                       float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)voff, (int)soff, AUX);
}

// A stored column kx holds its own conjugates (kx = 0, and kx = W/2 for even W).
__host__ __device__ constexpr bool herm_col(int kx, int W) { return kx == 0 || (W % 2 == 0 && 2 * kx == W); }
// Number of stored rows that are kept for column kx (Hermitian columns keep ky <= H/2).
__host__ __device__ constexpr int col_rows(int kx, int H, int W) { return herm_col(kx, W) ? H / 2 + 1 : H; }
__host__ __device__ constexpr bool self_conj(int ky, int kx, int H, int W) {
  return herm_col(kx, W) && (ky == 0 || 2 * ky == H);
}

// Unnormalised forward 2-D real DFT of one channel of one tile, kept on the
// unique bins only: Hermitian columns ky <= HP/2, other columns all ky.
// `r` covers the frame, `tile0` is the byte offset of channel 0 of the tile's
// top-left token, `c4` the lane's channel byte offset (always in range).
template <int HP, int WP>
__device__ __forceinline__ void load_fwd(__amdgpu_buffer_rsrc_t r, unsigned tile0, unsigned WgD4,
                                         unsigned D4, unsigned c4, float (&fr)[HP][WP / 2 + 1],
                                         float (&fi)[HP][WP / 2 + 1]) {
  constexpr int NKX = WP / 2 + 1;
  float x[HP][WP];
  fft::static_for<0, HP>([&](auto yy) {
    constexpr int y = decltype(yy)::value;
    fft::static_for<0, WP>([&](auto xx) {
      constexpr int xi = decltype(xx)::value;
      x[y][xi] = buf_ld(r, c4, tile0 + y * WgD4 + xi * D4);
    });
  });
  float rr[HP][NKX], ri[HP][NKX];
  fft::static_for<0, HP>([&](auto yy) {
    constexpr int y = decltype(yy)::value;
    fft::rdft<WP>(x[y], rr[y], ri[y]);
  });
  fft::static_for<0, NKX>([&](auto kk) {
    constexpr int kx = decltype(kk)::value;
    if constexpr (herm_col(kx, WP)) {
      float col[HP], cr[HP / 2 + 1], ci[HP / 2 + 1];
      fft::static_for<0, HP>([&](auto yy) { col[decltype(yy)::value] = rr[decltype(yy)::value][kx]; });
      fft::rdft<HP>(col, cr, ci);
      fft::static_for<0, HP / 2 + 1>([&](auto yy) {
        constexpr int ky = decltype(yy)::value;
        fr[ky][kx] = cr[ky];
        fi[ky][kx] = ci[ky];
      });
    } else {
      float cr[HP], ci[HP];
      fft::static_for<0, HP>([&](auto yy) {
        constexpr int y = decltype(yy)::value;
        cr[y] = rr[y][kx];
        ci[y] = ri[y][kx];
      });
      fft::cdft<HP, false>(cr, ci);
      fft::static_for<0, HP>([&](auto yy) {
        constexpr int ky = decltype(yy)::value;
        fr[ky][kx] = cr[ky];
        fi[ky][kx] = ci[ky];
      });
    }
  });
}

// ---------------------------------------------------------------------------
// par_xspec
// ---------------------------------------------------------------------------
template <int HP, int WP>
__device__ __forceinline__ void xspec_body(const ParArgs& a, const float* __restrict__ resid,
                                           const TileGeom& g, int c_lane, int fa, int fb,
                                           float* lds_row) {
  constexpr int NKX = WP / 2 + 1;
  const bool valid = c_lane < a.D;
  const unsigned c4 = 4u * (unsigned)(valid ? c_lane : a.D - 1);
  const unsigned tile0 = 4u * (unsigned)((g.y0 * a.Wg + g.x0) * a.D);
  const unsigned WgD4 = 4u * (unsigned)(a.Wg * a.D), D4 = 4u * (unsigned)a.D;
  float ar[HP][NKX], ai[HP][NKX], br[HP][NKX], bi[HP][NKX];
  load_fwd<HP, WP>(frame_rsrc(resid, fa, a.frame_elems), tile0, WgD4, D4, c4, ar, ai);
  load_fwd<HP, WP>(frame_rsrc(resid, fb, a.frame_elems), tile0, WgD4, D4, c4, br, bi);
  const float live = valid ? 1.0f : 0.0f;   // lanes past D contribute nothing
  // every slot of the lane's LDS row is written (zeros where no unique bin lives)
  fft::static_for<0, kNkx * HP>([&](auto bb) {
    constexpr int ky = decltype(bb)::value / kNkx;
    constexpr int kx = decltype(bb)::value % kNkx;
    constexpr int s = (ky * kNkx + kx) * 3;
    if constexpr (kx < NKX && ky < col_rows(kx, HP, WP)) {
      const float xr = ar[ky][kx], xi = ai[ky][kx], yr = br[ky][kx], yi = bi[ky][kx];
      lds_row[s + 0] = live * (yr * xr + yi * xi);
      lds_row[s + 1] = self_conj(ky, kx, HP, WP) ? 0.0f : live * (yi * xr - yr * xi);
      lds_row[s + 2] = live * sqrtf((xr * xr + xi * xi) * (yr * yr + yi * yi));
    } else {
      lds_row[s + 0] = 0.0f;
      lds_row[s + 1] = 0.0f;
      lds_row[s + 2] = 0.0f;
    }
  });
  for (int s = HP * kNkx * 3; s < kVals; ++s) lds_row[s] = 0.0f;
}

template <int HP, int WP>
__global__ __launch_bounds__(64) void par_xspec_kernel(ParArgs a, TileClass k,
                                                        const float* __restrict__ resid,
                                                        float* __restrict__ partial) {
  __shared__ float lds[kChb * kLdsStride];
  const int tile = class_tile(a, k, blockIdx.x), chb = blockIdx.y, pair = blockIdx.z;
  const TileGeom g = tile_geom(a, tile);
  const int lane = threadIdx.x;
  const int c = chb * kChb + lane;
  const int fa = a.anchors[pair], fb = a.anchors[pair + 1];
  xspec_body<HP, WP>(a, resid, g, c, fa, fb, lds + lane * kLdsStride);
  __syncthreads();
  float* dst = partial + (((long long)pair * a.n_tiles + tile) * a.n_chblk + chb) * kVals;
  for (int v = lane; v < kVals; v += kChb) {
    float s0 = 0.0f, s1 = 0.0f, s2 = 0.0f, s3 = 0.0f;
#pragma unroll 16
    for (int l = 0; l < kChb; l += 4) {
      s0 += lds[(l + 0) * kLdsStride + v];
      s1 += lds[(l + 1) * kLdsStride + v];
      s2 += lds[(l + 2) * kLdsStride + v];
      s3 += lds[(l + 3) * kLdsStride + v];
    }
    dst[v] = (s0 + s1) + (s2 + s3);
  }
}

// ---------------------------------------------------------------------------
// par_gate
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Principal argument in (-pi, pi].
__device__ __forceinline__ float wrap_arg(float y, float x) {
  float t = atan2f(y, x);
  const float kPiF = 3.14159265358979323846f;
  return (t == -kPiF) ? kPiF : t;
}

__global__ __launch_bounds__(64) void par_gate_kernel(ParArgs a, const float* __restrict__ partial,
                                                       float4* __restrict__ coef) {
  const int tile = blockIdx.x, pair = blockIdx.y;
  const TileGeom g = tile_geom(a, tile);
  const int b = threadIdx.x;
  const int ky = b / kNkx, kx = b - (b / kNkx) * kNkx;
  const int H = g.hp, W = g.wp;
  const bool active = b < kBins && ky < H && kx <= W / 2;
  const bool hc = kx == 0 || (W % 2 == 0 && 2 * kx == W);
  int kind = 0;  // 0 representative, 1 mirror, 2 self-conjugate
  int sky = ky;  // row of the slot whose partial sums hold this bin's values
  if (hc) {
    int mky = (H - ky) % H;
    if (mky == ky) kind = 2;
    else if (2 * ky > H) { kind = 1; sky = mky; }
  }
  float zr = 0.0f, zi = 0.0f, w = 0.0f;
  if (active) {
    const float* src = partial + ((long long)pair * a.n_tiles + tile) * a.n_chblk * kVals +
                       (sky * kNkx + kx) * 3;
#pragma unroll 8
    for (int j = 0; j < a.n_chblk; ++j) {
      zr += src[(long long)j * kVals + 0];
      zi += src[(long long)j * kVals + 1];
      w += src[(long long)j * kVals + 2];
    }
    const float nrm = 1.0f / (float)(H * W);   // orthonormal scaling of both spectra
    zr *= nrm;
    zi *= nrm;
    w *= nrm;
    if (kind == 1) zi = -zi;                    // mirror = conjugate of its representative
  }
  const float wmax = wave_max(active ? w : 0.0f);
  const float eta = a.eta_rel * wmax + a.eta_abs;
  const float zabs = sqrtf(zr * zr + zi * zi);
  const bool rel = active && (w > eta) && (zabs > eta);
  float theta = 0.0f;
  if (rel && kind == 0) theta = wrap_arg(zi, zr);
  if (rel && kind == 1) theta = -wrap_arg(-zi, zr);
  const bool omega_plus = rel && !(ky == 0 && kx == 0);
  const float kappa = hc ? 1.0f : 2.0f;
  const float num = wave_sum(omega_plus ? kappa * zabs : 0.0f);
  const float den = wave_sum(omega_plus ? kappa * w : 0.0f);
  const int n_plus = __popcll(__ballot(omega_plus));
  const float conf = n_plus > 0 ? num / (den + a.eps) : 0.0f;
  // nu: physical radius of the bin over the largest stored radius of the tile
  const int kys = (2 * ky <= H) ? ky : ky - H;
  const float fy = (float)kys / (float)H, fx = (float)kx / (float)W;
  const float my = (float)(H / 2) / (float)H, mx = (float)(W / 2) / (float)W;
  const float rmax = sqrtf(my * my + mx * mx);
  const float nu = rmax > 0.0f ? sqrtf(fy * fy + fx * fx) / rmax : 0.0f;
  float gate;
  if (a.gate_mode == 1) gate = 1.0f;
  else if (a.gate_mode == 2) gate = 0.0f;
  else {
    const float tau = a.tau_low + (a.tau_high - a.tau_low) * powf(nu, a.q);
    gate = 1.0f / (1.0f + expf(-(conf - tau) / a.T));
  }
  // optional diagnostics, laid out per the caller's tile_h x (tile_w/2+1) rows
  const int nkx_out = a.tile_w / 2 + 1;
  if (b < kBins && ky < a.tile_h && kx < nkx_out) {
    const long long o = ((long long)pair * a.n_tiles + tile) * a.bins_out + ky * nkx_out + kx;
    if (a.theta_out) a.theta_out[o] = active ? theta : 0.0f;
    if (a.gate_out) a.gate_out[o] = active ? gate : 0.0f;
  }
  if (a.conf_out && b == 0) a.conf_out[(long long)pair * a.n_tiles + tile] = conf;
  if (b >= kBins) return;
  // blend coefficients for every target of this pair (eq:block composition)
  const int n_pairs = a.n_anchor - 1;
  const int fa = a.anchors[pair], fb = a.anchors[pair + 1];
  const float inv_gap = 1.0f / (float)(fb - fa);
  const float nrm = 1.0f / (float)(H * W);
  for (int part = 0; part < 3; ++part) {
    int t0, t1;
    if (part == 0) { t0 = fa + 1; t1 = fb; }
    else if (part == 1) { if (pair != 0) continue; t0 = 0; t1 = fa; }
    else { if (pair != n_pairs - 1) continue; t0 = fb + 1; t1 = a.n_frames; }
    for (int t = t0; t < t1; ++t) {
      const float alpha = (float)(t - fa) * inv_gap;
      float4 cf = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (active) {
        float sa, ca, sb, cb;
        sincosf(gate * alpha * theta, &sa, &ca);
        sincosf(-gate * (1.0f - alpha) * theta, &sb, &cb);
        const float wa = (1.0f - alpha) * nrm, wb = alpha * nrm;
        cf = make_float4(wa * ca, wa * sa, wb * cb, wb * sb);
      }
      coef[((long long)t * a.n_tiles + tile) * kBins + b] = cf;
    }
  }
}

// ---------------------------------------------------------------------------
// par_recon
// ---------------------------------------------------------------------------
// Number of unique stored bins of an HP x WP tile (Hermitian columns keep ky <= HP/2).
template <int HP, int WP>
constexpr int unique_bins() {
  int n = 0;
  for (int kx = 0; kx <= WP / 2; ++kx) n += col_rows(kx, HP, WP);
  return n;
}
// Slot of unique bin (ky, kx) in that enumeration (column-major over kx).
template <int HP, int WP>
constexpr int unique_slot(int ky, int kx) {
  int n = 0;
  for (int c = 0; c < kx; ++c) n += col_rows(c, HP, WP);
  return n + ky;
}

template <int HP, int WP, bool ACC>
__device__ __forceinline__ void recon_body(const ParArgs& a, const float* __restrict__ resid,
                                           float* __restrict__ out,
                                           const float4* __restrict__ coef, const TileGeom& g,
                                           int tile, int c_lane, int pair, float* fb_lds) {
  constexpr int NKX = WP / 2 + 1;
  constexpr int NU = unique_bins<HP, WP>();
  // Lanes past the last channel mirror channel D-1: same inputs, same results, and
  // they sit in the same wave as the lane that owns D-1, so their stores (and
  // read-modify-writes) coincide with it instruction by instruction.
  const unsigned c4 = 4u * (unsigned)(c_lane < a.D ? c_lane : a.D - 1);
  const unsigned tile0 = 4u * (unsigned)((g.y0 * a.Wg + g.x0) * a.D);
  const unsigned WgD4 = 4u * (unsigned)(a.Wg * a.D), D4 = 4u * (unsigned)a.D;
  const int fa = a.anchors[pair], fb = a.anchors[pair + 1];
  float ar[HP][NKX], ai[HP][NKX];
  {
    // F_b is parked in this lane's LDS column (LDS as extra per-lane storage: no
    // other lane reads it, so no barrier is needed)
    float br[HP][NKX], bi[HP][NKX];
    load_fwd<HP, WP>(frame_rsrc(resid, fb, a.frame_elems), tile0, WgD4, D4, c4, br, bi);
    fft::static_for<0, NKX>([&](auto kk) {
      constexpr int kx = decltype(kk)::value;
      fft::static_for<0, col_rows(kx, HP, WP)>([&](auto yy) {
        constexpr int ky = decltype(yy)::value;
        constexpr int u = unique_slot<HP, WP>(ky, kx);
        fb_lds[(2 * u) * kChb] = br[ky][kx];
        fb_lds[(2 * u + 1) * kChb] = bi[ky][kx];
      });
    });
  }
  load_fwd<HP, WP>(frame_rsrc(resid, fa, a.frame_elems), tile0, WgD4, D4, c4, ar, ai);
  (void)NU;
  const int n_pairs = a.n_anchor - 1;
  for (int part = 0; part < 3; ++part) {
    int t0, t1;
    if (part == 0) { t0 = fa + 1; t1 = fb; }
    else if (part == 1) { if (pair != 0) continue; t0 = 0; t1 = fa; }
    else { if (pair != n_pairs - 1) continue; t0 = fb + 1; t1 = a.n_frames; }
    for (int t = t0; t < t1; ++t) {
      const float4* __restrict__ cf = coef + ((long long)t * a.n_tiles + tile) * kBins;
      const __amdgpu_buffer_rsrc_t dst = frame_rsrc(out, t, a.frame_elems);
      // Recompute the uniform token offsets per target instead of keeping 64 of them
      // live across the target loop.
      unsigned wgd = __builtin_amdgcn_readfirstlane(WgD4), dd = __builtin_amdgcn_readfirstlane(D4);
      asm volatile("" : "+s"(wgd), "+s"(dd));
      // likewise re-read F_b from LDS per target rather than hoisting it into VGPRs
      const float* fbp = fb_lds;
      asm volatile("" : "+v"(fbp));
      // accumulate mode: fetch X_t first, all 64 loads in flight together (nothing
      // is stored to this frame before they are issued)
      float old[HP][WP];
      if constexpr (ACC) {
        fft::static_for<0, HP>([&](auto yy) {
          constexpr int y = decltype(yy)::value;
          fft::static_for<0, WP>([&](auto xx) {
            constexpr int xi = decltype(xx)::value;
            old[y][xi] = buf_ld(dst, c4, tile0 + y * wgd + xi * dd);
          });
        });
      }
      // eq:fcpasm blend and the column (y) inverse, one stored column at a time
      float gr[HP][NKX], gi[HP][NKX];
      fft::static_for<0, NKX>([&](auto kk) {
        constexpr int kx = decltype(kk)::value;
        auto fbr = [&](int u) { return fbp[(2 * u) * kChb]; };
        auto fbi = [&](int u) { return fbp[(2 * u + 1) * kChb]; };
        if constexpr (herm_col(kx, WP)) {
          float hr[HP / 2 + 1], hi[HP / 2 + 1], col[HP];
          fft::static_for<0, HP / 2 + 1>([&](auto yy) {
            constexpr int ky = decltype(yy)::value;
            constexpr int u = unique_slot<HP, WP>(ky, kx);
            const float4 k = cf[ky * kNkx + kx];
            if constexpr (self_conj(ky, kx, HP, WP)) {
              hr[ky] = k.x * ar[ky][kx] + k.z * fbr(u);
              hi[ky] = 0.0f;
            } else {
              const float b_r = fbr(u), b_i = fbi(u);
              hr[ky] = k.x * ar[ky][kx] - k.y * ai[ky][kx] + k.z * b_r - k.w * b_i;
              hi[ky] = k.x * ai[ky][kx] + k.y * ar[ky][kx] + k.z * b_i + k.w * b_r;
            }
          });
          fft::c2r<HP>(hr, hi, col);
          fft::static_for<0, HP>([&](auto yy) {
            constexpr int y = decltype(yy)::value;
            gr[y][kx] = col[y];
            gi[y][kx] = 0.0f;
          });
        } else {
          float hr[HP], hi[HP];
          fft::static_for<0, HP>([&](auto yy) {
            constexpr int ky = decltype(yy)::value;
            constexpr int u = unique_slot<HP, WP>(ky, kx);
            const float4 k = cf[ky * kNkx + kx];
            const float b_r = fbr(u), b_i = fbi(u);
            hr[ky] = k.x * ar[ky][kx] - k.y * ai[ky][kx] + k.z * b_r - k.w * b_i;
            hi[ky] = k.x * ai[ky][kx] + k.y * ar[ky][kx] + k.z * b_i + k.w * b_r;
          });
          fft::cdft<HP, true>(hr, hi);
          fft::static_for<0, HP>([&](auto yy) {
            constexpr int y = decltype(yy)::value;
            gr[y][kx] = hr[y];
            gi[y][kx] = hi[y];
          });
        }
      });
      // row (x) inverse real transforms and the store / accumulate
      fft::static_for<0, HP>([&](auto yy) {
        constexpr int y = decltype(yy)::value;
        float xv[WP];
        fft::c2r<WP>(gr[y], gi[y], xv);
        fft::static_for<0, WP>([&](auto xx) {
          constexpr int xi = decltype(xx)::value;
          const unsigned so = tile0 + y * wgd + xi * dd;
          if constexpr (ACC) buf_st<0>(dst, c4, so, old[y][xi] + xv[xi]);
          else buf_st<kNT>(dst, c4, so, xv[xi]);
        });
      });
    }
  }
}

template <int HP, int WP, bool ACC>
__global__ __launch_bounds__(64) void par_recon_kernel(ParArgs a, TileClass k,
                                                        const float* __restrict__ resid,
                                                        float* __restrict__ out,
                                                        const float4* __restrict__ coef) {
  __shared__ float fb_lds[2 * kBins * kChb];
  const int tile = class_tile(a, k, blockIdx.x), chb = blockIdx.y, pair = blockIdx.z;
  const TileGeom g = tile_geom(a, tile);
  recon_body<HP, WP, ACC>(a, resid, out, coef, g, tile, chb * kChb + threadIdx.x, pair,
                          fb_lds + threadIdx.x);
}

// Host-side table of the per-shape kernels, indexed [HP-1][WP-1].
typedef void (*XspecFn)(ParArgs, TileClass, const float*, float*);
typedef void (*ReconFn)(ParArgs, TileClass, const float*, float*, const float4*);

template <int HP, int WP>
struct ShapeKernels {
  static constexpr XspecFn xspec = par_xspec_kernel<HP, WP>;
  static constexpr ReconFn recon_w = par_recon_kernel<HP, WP, false>;
  static constexpr ReconFn recon_a = par_recon_kernel<HP, WP, true>;
};

#define CAST_SHAPE_ROW(H)                                                                   \
  {ShapeKernels<H, 1>::xspec, ShapeKernels<H, 2>::xspec, ShapeKernels<H, 3>::xspec,         \
   ShapeKernels<H, 4>::xspec, ShapeKernels<H, 5>::xspec, ShapeKernels<H, 6>::xspec,         \
   ShapeKernels<H, 7>::xspec, ShapeKernels<H, 8>::xspec}
const XspecFn kXspec[8][8] = {CAST_SHAPE_ROW(1), CAST_SHAPE_ROW(2), CAST_SHAPE_ROW(3),
                              CAST_SHAPE_ROW(4), CAST_SHAPE_ROW(5), CAST_SHAPE_ROW(6),
                              CAST_SHAPE_ROW(7), CAST_SHAPE_ROW(8)};
#undef CAST_SHAPE_ROW
#define CAST_SHAPE_ROW(H, F)                                                                \
  {ShapeKernels<H, 1>::F, ShapeKernels<H, 2>::F, ShapeKernels<H, 3>::F,                     \
   ShapeKernels<H, 4>::F, ShapeKernels<H, 5>::F, ShapeKernels<H, 6>::F,                     \
   ShapeKernels<H, 7>::F, ShapeKernels<H, 8>::F}
const ReconFn kReconW[8][8] = {CAST_SHAPE_ROW(1, recon_w), CAST_SHAPE_ROW(2, recon_w),
                               CAST_SHAPE_ROW(3, recon_w), CAST_SHAPE_ROW(4, recon_w),
                               CAST_SHAPE_ROW(5, recon_w), CAST_SHAPE_ROW(6, recon_w),
                               CAST_SHAPE_ROW(7, recon_w), CAST_SHAPE_ROW(8, recon_w)};
const ReconFn kReconA[8][8] = {CAST_SHAPE_ROW(1, recon_a), CAST_SHAPE_ROW(2, recon_a),
                               CAST_SHAPE_ROW(3, recon_a), CAST_SHAPE_ROW(4, recon_a),
                               CAST_SHAPE_ROW(5, recon_a), CAST_SHAPE_ROW(6, recon_a),
                               CAST_SHAPE_ROW(7, recon_a), CAST_SHAPE_ROW(8, recon_a)};
#undef CAST_SHAPE_ROW

struct ClassLaunch {
  int hp, wp, ntiles;
  TileClass k;
};

// Up to four tile classes: interior, right edge column, bottom edge row, corner.
int tile_classes(int Hg, int Wg, int th, int tw, ClassLaunch (&out)[4]) {
  const int nyf = Hg / th, hr = Hg % th, nxf = Wg / tw, wr = Wg % tw;
  const int ntx = nxf + (wr > 0);
  int n = 0;
  if (nyf > 0 && nxf > 0) out[n++] = {th, tw, nyf * nxf, {0, 0, nxf}};
  if (nyf > 0 && wr > 0) out[n++] = {th, wr, nyf, {0, nxf, 1}};
  if (hr > 0 && nxf > 0) out[n++] = {hr, tw, nxf, {nyf, 0, nxf}};
  if (hr > 0 && wr > 0) out[n++] = {hr, wr, 1, {nyf, nxf, 1}};
  (void)ntx;
  return n;
}

}  // namespace

ParPlan plan_par(int n_frames, int n_anchor, int Hg, int Wg, int D, const cast_par_params_t& p) {
  ParPlan pl{};
  pl.n_pairs = n_anchor - 1;
  pl.n_tiles_y = (Hg + p.tile_h - 1) / p.tile_h;
  pl.n_tiles_x = (Wg + p.tile_w - 1) / p.tile_w;
  pl.n_tiles = pl.n_tiles_y * pl.n_tiles_x;
  pl.chb = kChb;
  pl.n_chblk = (D + kChb - 1) / kChb;
  pl.bins_out = p.tile_h * (p.tile_w / 2 + 1);
  size_t partial = (size_t)pl.n_pairs * pl.n_tiles * pl.n_chblk * kVals * sizeof(float);
  size_t coef = (size_t)n_frames * pl.n_tiles * kBins * 4 * sizeof(float);
  pl.off_partial = 0;
  pl.off_coef = align_up(partial);
  pl.total = pl.off_coef + align_up(coef);
  return pl;
}

cast_status_t launch_par(const float* resid, const int* anchors, int n_anchor, int n_frames,
                         int Hg, int Wg, int D, const cast_par_params_t& p, float* out,
                         float* theta_out, float* gate_out, float* conf_out, const ParPlan& pl,
                         void* ws, hipStream_t stream) {
  ParArgs a{};
  float* partial = reinterpret_cast<float*>(static_cast<char*>(ws) + pl.off_partial);
  float4* coef = reinterpret_cast<float4*>(static_cast<char*>(ws) + pl.off_coef);
  a.theta_out = theta_out;
  a.gate_out = gate_out;
  a.conf_out = conf_out;
  a.frame_elems = (long long)Hg * Wg * D;
  a.n_frames = n_frames;
  a.Hg = Hg;
  a.Wg = Wg;
  a.D = D;
  a.tile_h = p.tile_h;
  a.tile_w = p.tile_w;
  a.n_tx = pl.n_tiles_x;
  a.n_tiles = pl.n_tiles;
  a.n_anchor = n_anchor;
  a.n_chblk = pl.n_chblk;
  a.bins_out = pl.bins_out;
  a.tau_low = p.tau_low;
  a.tau_high = p.tau_high;
  a.q = p.q;
  a.T = p.T;
  a.eta_rel = p.eta_rel;
  a.eta_abs = p.eta_abs;
  a.eps = p.eps;
  a.gate_mode = p.gate_mode;
  a.accumulate = p.accumulate;
  for (int j = 0; j < n_anchor; ++j) a.anchors[j] = (short)anchors[j];

  ClassLaunch cls[4];
  const int ncls = tile_classes(Hg, Wg, p.tile_h, p.tile_w, cls);
  cast_status_t st;
  for (int j = 0; j < ncls; ++j) {
    dim3 grid(cls[j].ntiles, pl.n_chblk, pl.n_pairs);
    hipLaunchKernelGGL(kXspec[cls[j].hp - 1][cls[j].wp - 1], grid, dim3(kChb), 0, stream, a,
                       cls[j].k, resid, partial);
    st = check_launch("par_xspec");
    if (st != CAST_OK) return st;
  }
  hipLaunchKernelGGL(par_gate_kernel, dim3(pl.n_tiles, pl.n_pairs), dim3(64), 0, stream, a,
                     (const float*)partial, coef);
  st = check_launch("par_gate");
  if (st != CAST_OK) return st;
  for (int j = 0; j < ncls; ++j) {
    dim3 grid(cls[j].ntiles, pl.n_chblk, pl.n_pairs);
    ReconFn fn = p.accumulate ? kReconA[cls[j].hp - 1][cls[j].wp - 1]
                              : kReconW[cls[j].hp - 1][cls[j].wp - 1];
    hipLaunchKernelGGL(fn, grid, dim3(kChb), 0, stream, a, cls[j].k, resid, out,
                       (const float4*)coef);
    st = check_launch("par_recon");
    if (st != CAST_OK) return st;
  }
  return CAST_OK;
}

}  // namespace cast
