// Device code of Phase-Aware Reconstruction, shared by the translation units
// that instantiate it (per-shape kernels and the fused 8x8-tiling kernels).
// See par.hip for the algorithm and the launch structure.
#pragma once
#include "cast_common.h"
#include "fft_tile.h"

namespace cast {
namespace pardev {


constexpr int kBins = kParBinsMax;     // 40 stored-bin slots: index ky*5 + kx
constexpr int kNkx = kParNkxMax;       // 5
constexpr int kVals = kBins * 3;       // (Re Z, Im Z, W) per slot
constexpr int kChb = 64;               // channels per block (one wave)
constexpr int kXsStride = kChb + 2;    // LDS row of one bin slot: 64 lane values + pad (8-byte rows)
typedef float f32x2 __attribute__((ext_vector_type(2)));

struct ParArgs {
  float* theta_out;
  float* gate_out;
  float* conf_out;
  long long frame_elems;  // Hg * Wg * D
  int n_frames, Hg, Wg, D;
  int tile_h, tile_w, n_tx, n_tiles;
  int n_anchor, n_chblk, bins_out;
  float tau_low, tau_high, q, T, eta_rel, eta_abs, eps;
  int gate_mode, accumulate, update_anchors;
  short anchors[kParMaxAnchors];
  // the fused reconstruction launch takes the pairs in this order: most targets
  // first, so the blocks that walk the longest target lists start first and the
  // launch ends on short ones
  short recon_order[kParMaxAnchors];
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
template <int AUX = 0>
__device__ __forceinline__ float buf_ld(__amdgpu_buffer_rsrc_t r, unsigned voff, unsigned soff) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, AUX));
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
// load_tile reads the tile's HP x WP values of one channel: `r` covers the frame,
// `tile0` is the byte offset of channel 0 of the tile's top-left token, `c4` the
// lane's channel byte offset (always in range); fwd_tile transforms them.
template <int HP, int WP>
__device__ __forceinline__ void load_tile(__amdgpu_buffer_rsrc_t r, unsigned tile0, unsigned WgD4,
                                          unsigned D4, unsigned c4, float (&x)[HP][WP]) {
  fft::static_for<0, HP>([&](auto yy) {
    constexpr int y = decltype(yy)::value;
    fft::static_for<0, WP>([&](auto xx) {
      constexpr int xi = decltype(xx)::value;
      x[y][xi] = buf_ld(r, c4, tile0 + y * WgD4 + xi * D4);
    });
  });
}

// Forward transform of loaded tile values (unique bins, as above).
template <int HP, int WP>
__device__ __forceinline__ void fwd_tile(const float (&x)[HP][WP], float (&fr)[HP][WP / 2 + 1],
                                         float (&fi)[HP][WP / 2 + 1]) {
  constexpr int NKX = WP / 2 + 1;
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
// One block of the cross-spectrum pass: tile `tile`, channel block `chb`, pair.
// Every lane transforms both anchors of its channel (all their loads in flight
// together); the per-bin products Re(F_b conj F_a), Im(F_b conj F_a) and
// |F_b||F_a| are summed over the 64 lanes through LDS, one quantity at a time (40
// rows of 64 lane values plus pad, 10.6 KB, so that LDS does not limit the number
// of resident blocks), in fixed lane order.
template <int HP, int WP>
__device__ __forceinline__ void xspec_block(const ParArgs& a, int tile, int chb, int pair,
                                            const float* __restrict__ resid,
                                            float* __restrict__ partial, float* lds) {
  constexpr int NKX = WP / 2 + 1;
  const TileGeom g = tile_geom(a, tile);
  const int lane = threadIdx.x;
  const int c_lane = chb * kChb + lane;
  const int fa = a.anchors[pair], fb = a.anchors[pair + 1];
  const bool valid = c_lane < a.D;
  const unsigned c4 = 4u * (unsigned)(valid ? c_lane : a.D - 1);
  const unsigned tile0 = 4u * (unsigned)((g.y0 * a.Wg + g.x0) * a.D);
  const unsigned WgD4 = 4u * (unsigned)(a.Wg * a.D), D4 = 4u * (unsigned)a.D;
  float ar[HP][NKX], ai[HP][NKX], br[HP][NKX], bi[HP][NKX];
  {
    float xa[HP][WP], xb[HP][WP];
    load_tile<HP, WP>(frame_rsrc(resid, fa, a.frame_elems), tile0, WgD4, D4, c4, xa);
    load_tile<HP, WP>(frame_rsrc(resid, fb, a.frame_elems), tile0, WgD4, D4, c4, xb);
    fwd_tile<HP, WP>(xa, ar, ai);
    fwd_tile<HP, WP>(xb, br, bi);
  }
  const float live = valid ? 1.0f : 0.0f;   // lanes past D contribute nothing
  float* dst = partial + (((long long)pair * a.n_tiles + tile) * a.n_chblk + chb) * kVals;
  fft::static_for<0, 3>([&](auto qq) {
    constexpr int q = decltype(qq)::value;
    // the lane's value of quantity q at every slot (zero where no unique bin lives)
    fft::static_for<0, kNkx * HP>([&](auto bb) {
      constexpr int ky = decltype(bb)::value / kNkx;
      constexpr int kx = decltype(bb)::value % kNkx;
      constexpr int s = ky * kNkx + kx;
      float* cell = lds + s * kXsStride + lane;
      if constexpr (kx < NKX && ky < col_rows(kx, HP, WP)) {
        const float xr = ar[ky][kx], xi = ai[ky][kx], yr = br[ky][kx], yi = bi[ky][kx];
        if constexpr (q == 0) *cell = live * (yr * xr + yi * xi);
        else if constexpr (q == 1) *cell = self_conj(ky, kx, HP, WP) ? 0.0f : live * (yi * xr - yr * xi);
        else *cell = live * sqrtf((xr * xr + xi * xi) * (yr * yr + yi * yi));
      } else {
        *cell = 0.0f;
      }
    });
    for (int s = HP * kNkx; s < kBins; ++s) lds[s * kXsStride + lane] = 0.0f;
    __syncthreads();
    if (lane < kBins) {
      // slot `lane`'s 64 lane values are one contiguous row: 8-byte reads, all in
      // flight together; partial sum g takes the lanes l = g mod 4 in order
      const f32x2* rowp = reinterpret_cast<const f32x2*>(lds + lane * kXsStride);
      f32x2 v[kChb / 2];
#pragma unroll
      for (int k = 0; k < kChb / 2; ++k) v[k] = rowp[k];
      float s0 = 0.0f, s1 = 0.0f, s2 = 0.0f, s3 = 0.0f;
#pragma unroll
      for (int k = 0; k < kChb / 2; k += 2) {
        s0 += v[k].x;
        s1 += v[k].y;
        s2 += v[k + 1].x;
        s3 += v[k + 1].y;
      }
      dst[lane * 3 + q] = (s0 + s1) + (s2 + s3);
    }
    __syncthreads();
  });
}

// ---------------------------------------------------------------------------
// The gate of one stored bin (App. A.2, eq:confidence, eq:gate), one lane per bin
// slot b of a wave: from the channel sums (Z, W) of the bin's slot, eta over the
// tile's stored bins, reliability, theta (representative / mirror /
// self-conjugate), c_p over the tile, nu and g.  Every lane of the wave takes part
// (wave reductions); lanes outside the tile's bins pass active = false.
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

// Which slot holds bin b's sums: Hermitian columns store their rows ky <= H/2;
// a mirror row reads its representative's slot and conjugates it.
struct BinSlot {
  int ky, kx, sky, kind;   // kind 0 representative, 1 mirror, 2 self-conjugate
  bool active, hc;
};
__device__ __forceinline__ BinSlot bin_slot(int b, int H, int W) {
  BinSlot r;
  r.ky = b / kNkx;
  r.kx = b - r.ky * kNkx;
  r.active = b < kBins && r.ky < H && r.kx <= W / 2;
  r.hc = r.kx == 0 || (W % 2 == 0 && 2 * r.kx == W);
  r.kind = 0;
  r.sky = r.ky;
  if (r.hc) {
    const int mky = (H - r.ky) % H;
    if (mky == r.ky) r.kind = 2;
    else if (2 * r.ky > H) { r.kind = 1; r.sky = mky; }
  }
  return r;
}

struct BinGate {
  float theta, gate, conf;
};
// zr, zi, w: the slot's sums over all channels of F_b conj(F_a) and |F_b||F_a|
// (unnormalised transforms).
__device__ __forceinline__ BinGate bin_gate(const ParArgs& a, const BinSlot& s, int H, int W,
                                            float zr, float zi, float w) {
  if (s.active) {
    const float nrm = 1.0f / (float)(H * W);   // orthonormal scaling of both spectra
    zr *= nrm;
    zi *= nrm;
    w *= nrm;
    if (s.kind == 1) zi = -zi;                  // mirror = conjugate of its representative
  } else {
    zr = zi = w = 0.0f;
  }
  const float wmax = wave_max(s.active ? w : 0.0f);
  const float eta = a.eta_rel * wmax + a.eta_abs;
  const float zabs = sqrtf(zr * zr + zi * zi);
  const bool rel = s.active && (w > eta) && (zabs > eta);
  BinGate r;
  r.theta = 0.0f;
  if (rel && s.kind == 0) r.theta = wrap_arg(zi, zr);
  if (rel && s.kind == 1) r.theta = -wrap_arg(-zi, zr);
  const bool omega_plus = rel && !(s.ky == 0 && s.kx == 0);
  const float kappa = s.hc ? 1.0f : 2.0f;
  const float num = wave_sum(omega_plus ? kappa * zabs : 0.0f);
  const float den = wave_sum(omega_plus ? kappa * w : 0.0f);
  const int n_plus = __popcll(__ballot(omega_plus));
  r.conf = n_plus > 0 ? num / (den + a.eps) : 0.0f;
  // nu: physical radius of the bin over the largest stored radius of the tile
  const int kys = (2 * s.ky <= H) ? s.ky : s.ky - H;
  const float fy = (float)kys / (float)H, fx = (float)s.kx / (float)W;
  const float my = (float)(H / 2) / (float)H, mx = (float)(W / 2) / (float)W;
  const float rmax = sqrtf(my * my + mx * mx);
  const float nu = rmax > 0.0f ? sqrtf(fy * fy + fx * fx) / rmax : 0.0f;
  if (a.gate_mode == 1) r.gate = 1.0f;
  else if (a.gate_mode == 2) r.gate = 0.0f;
  else {
    const float tau = a.tau_low + (a.tau_high - a.tau_low) * powf(nu, a.q);
    r.gate = 1.0f / (1.0f + expf(-(r.conf - tau) / a.T));
  }
  return r;
}

// Blend coefficients of target t of pair (fa, fb) for one bin (eq:fcpasm with
// the orthonormal normalisation folded in): A_t = (1-alpha) e^{i g alpha theta} /
// (H W), B_t = alpha e^{-i g (1-alpha) theta} / (H W), alpha = (t - fa)/(fb - fa).
__device__ __forceinline__ float4 blend_coef(int t, int fa, int fb, float theta, float gate,
                                             int H, int W, bool active) {
  if (!active) return make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  const float alpha = (float)(t - fa) * (1.0f / (float)(fb - fa));
  const float nrm = 1.0f / (float)(H * W);
  float sa, ca, sb, cb;
  sincosf(gate * alpha * theta, &sa, &ca);
  sincosf(-gate * (1.0f - alpha) * theta, &sb, &cb);
  const float wa = (1.0f - alpha) * nrm, wb = alpha * nrm;
  return make_float4(wa * ca, wa * sa, wb * cb, wb * sb);
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

// The anchor case of eq:block on one (tile, channel): out[f] = R_f, or += R_f.
// NTT: the read-modify-write of out streams (nontemporal load and store).
template <int HP, int WP, bool ACC, bool NTT>
__device__ __forceinline__ void anchor_tile_update(const ParArgs& a, const float* __restrict__ resid,
                                                   float* __restrict__ out, int f, unsigned tile0,
                                                   unsigned WgD4, unsigned D4, unsigned c4) {
  const __amdgpu_buffer_rsrc_t src = frame_rsrc(resid, f, a.frame_elems);
  const __amdgpu_buffer_rsrc_t dst = frame_rsrc(out, f, a.frame_elems);
  fft::static_for<0, HP>([&](auto yy) {
    constexpr int y = decltype(yy)::value;
    float v[WP], o[WP];
    fft::static_for<0, WP>([&](auto xx) {
      constexpr int xi = decltype(xx)::value;
      v[xi] = buf_ld(src, c4, tile0 + y * WgD4 + xi * D4);
      if constexpr (ACC) o[xi] = buf_ld<NTT ? kNT : 0>(dst, c4, tile0 + y * WgD4 + xi * D4);
    });
    fft::static_for<0, WP>([&](auto xx) {
      constexpr int xi = decltype(xx)::value;
      if constexpr (ACC) buf_st<NTT ? kNT : 0>(dst, c4, tile0 + y * WgD4 + xi * D4, o[xi] + v[xi]);
      else buf_st<kNT>(dst, c4, tile0 + y * WgD4 + xi * D4, v[xi]);
    });
  });
}

// NTT (accumulate mode): the targets' read-modify-write streams past the caches
// (nontemporal loads and stores).  With several anchor pairs this pass reads every
// interior anchor once per adjacent pair, and streaming the targets keeps those
// anchors in the Infinity Cache for the second read.
//
// INL: the wave computes its tile's gate itself (bin_gate, one lane per stored bin,
// from the cross-spectrum partials) and each target's blend coefficients into
// coef_lds, instead of reading those of par_gate.  For grids that the chip holds
// in one round, where the gate launch would be a serial step of its own.
template <int HP, int WP, bool ACC, bool NTT, bool INL = false>
__device__ __forceinline__ void recon_body(const ParArgs& a, const float* __restrict__ resid,
                                           float* __restrict__ out,
                                           const float4* __restrict__ coef, const TileGeom& g,
                                           int tile, int c_lane, int pair, float* fb_lds,
                                           const float* __restrict__ partial = nullptr,
                                           float4* coef_lds = nullptr) {
  constexpr int NKX = WP / 2 + 1;
  constexpr int NU = unique_bins<HP, WP>();
  // INL: this lane's bin slot and its gate (lanes past the tile's bins: inactive)
  BinSlot bs{};
  BinGate bg{};
  if constexpr (INL) {
    bs = bin_slot((int)(threadIdx.x & 63), HP, WP);
    float zr = 0.0f, zi = 0.0f, w = 0.0f;
    if (bs.active) {
      const float* src = partial + ((long long)pair * a.n_tiles + tile) * a.n_chblk * kVals +
                         (bs.sky * kNkx + bs.kx) * 3;
#pragma unroll 8
      for (int j = 0; j < a.n_chblk; ++j) {
        zr += src[(long long)j * kVals + 0];
        zi += src[(long long)j * kVals + 1];
        w += src[(long long)j * kVals + 2];
      }
    }
    bg = bin_gate(a, bs, HP, WP, zr, zi, w);
  }
  // Lanes past the last channel mirror channel D-1: same inputs, same results, and
  // they sit in the same wave as the lane that owns D-1, so their stores (and
  // read-modify-writes) coincide with it instruction by instruction.
  const unsigned c4 = 4u * (unsigned)(c_lane < a.D ? c_lane : a.D - 1);
  const unsigned tile0 = 4u * (unsigned)((g.y0 * a.Wg + g.x0) * a.D);
  const unsigned WgD4 = 4u * (unsigned)(a.Wg * a.D), D4 = 4u * (unsigned)a.D;
  const int fa = a.anchors[pair], fb = a.anchors[pair + 1];
  if (a.update_anchors) {
    // pair p updates its left anchor, the last pair its right one too, so every
    // anchor slot is written once (out does not overlap resid)
    anchor_tile_update<HP, WP, ACC, NTT>(a, resid, out, fa, tile0, WgD4, D4, c4);
    if (pair == a.n_anchor - 2) anchor_tile_update<HP, WP, ACC, NTT>(a, resid, out, fb, tile0, WgD4, D4, c4);
  }
  float ar[HP][NKX], ai[HP][NKX];
  {
    // both anchors' loads in flight together; F_b is parked in this lane's LDS
    // column (LDS as extra per-lane storage: no other lane reads it, so no barrier
    // is needed)
    float xa[HP][WP], xb[HP][WP];
    load_tile<HP, WP>(frame_rsrc(resid, fb, a.frame_elems), tile0, WgD4, D4, c4, xb);
    load_tile<HP, WP>(frame_rsrc(resid, fa, a.frame_elems), tile0, WgD4, D4, c4, xa);
    float br[HP][NKX], bi[HP][NKX];
    fwd_tile<HP, WP>(xb, br, bi);
    fft::static_for<0, NKX>([&](auto kk) {
      constexpr int kx = decltype(kk)::value;
      fft::static_for<0, col_rows(kx, HP, WP)>([&](auto yy) {
        constexpr int ky = decltype(yy)::value;
        constexpr int u = unique_slot<HP, WP>(ky, kx);
        fb_lds[(2 * u) * kChb] = br[ky][kx];
        fb_lds[(2 * u + 1) * kChb] = bi[ky][kx];
      });
    });
    fwd_tile<HP, WP>(xa, ar, ai);
  }
  (void)NU;
  const int n_pairs = a.n_anchor - 1;
  for (int part = 0; part < 3; ++part) {
    int t0, t1;
    if (part == 0) { t0 = fa + 1; t1 = fb; }
    else if (part == 1) { if (pair != 0) continue; t0 = 0; t1 = fa; }
    else { if (pair != n_pairs - 1) continue; t0 = fb + 1; t1 = a.n_frames; }
    for (int t = t0; t < t1; ++t) {
      const float4* __restrict__ cf = coef + ((long long)t * a.n_tiles + tile) * kBins;
      if constexpr (INL) {
        // this target's coefficients, one bin per lane, into LDS for every lane
        const int b = (int)(threadIdx.x & 63);
        if (b < kBins) coef_lds[b] = blend_coef(t, fa, fb, bg.theta, bg.gate, HP, WP, bs.active);
        __syncthreads();
      }
      auto coef_at = [&](int u) -> float4 {
        if constexpr (INL) return coef_lds[u];
        else return cf[u];
      };
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
            old[y][xi] = buf_ld<NTT ? kNT : 0>(dst, c4, tile0 + y * wgd + xi * dd);
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
            const float4 k = coef_at(ky * kNkx + kx);
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
            const float4 k = coef_at(ky * kNkx + kx);
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
          if constexpr (ACC) buf_st<NTT ? kNT : 0>(dst, c4, so, old[y][xi] + xv[xi]);
          else buf_st<kNT>(dst, c4, so, xv[xi]);
        });
      });
    }
  }
}

// One block of the reconstruction pass: tile `tile`, channel block `chb`, pair.
template <int HP, int WP, bool ACC, bool NTT, bool INL = false>
__device__ __forceinline__ void recon_block(const ParArgs& a, int tile, int chb, int pair,
                                            const float* __restrict__ resid, float* __restrict__ out,
                                            const float4* __restrict__ coef, float* fb_lds,
                                            const float* __restrict__ partial = nullptr,
                                            float4* coef_lds = nullptr) {
  const TileGeom g = tile_geom(a, tile);
  recon_body<HP, WP, ACC, NTT, INL>(a, resid, out, coef, g, tile, chb * kChb + threadIdx.x, pair,
                                    fb_lds + threadIdx.x, partial, coef_lds);
}

// ---------------------------------------------------------------------------
// Fused launches for the default 8x8 tiling: one grid covers the interior, the
// right edge column (8 x WR), the bottom edge row (HR x 8) and the corner
// (HR x WR); each block takes its class from blockIdx.x (uniform branch) and runs
// that shape's fully unrolled code.  HR / WR = 8 mean "no remainder".
// ---------------------------------------------------------------------------
struct ClassSet {
  TileClass k[4];   // interior, right column, bottom row, corner
  int end[4];       // cumulative block counts along grid.x
};

template <int HR, int WR, class F>
__device__ __forceinline__ void for_class(const ParArgs& a, const ClassSet& cs, int b, F&& f) {
  if (b < cs.end[0]) {
    f(std::integral_constant<int, 8>{}, std::integral_constant<int, 8>{}, class_tile(a, cs.k[0], b));
    return;
  }
  if constexpr (WR < 8) {
    if (b < cs.end[1]) {
      f(std::integral_constant<int, 8>{}, std::integral_constant<int, WR>{}, class_tile(a, cs.k[1], b - cs.end[0]));
      return;
    }
  }
  if constexpr (HR < 8) {
    if (b < cs.end[2]) {
      f(std::integral_constant<int, HR>{}, std::integral_constant<int, 8>{}, class_tile(a, cs.k[2], b - cs.end[1]));
      return;
    }
  }
  if constexpr (HR < 8 && WR < 8) f(std::integral_constant<int, HR>{}, std::integral_constant<int, WR>{}, class_tile(a, cs.k[3], b - cs.end[2]));
}

// The fused launches run a 1-D grid of ntiles * n_chblk * n_pairs blocks, pairs one
// after another.  Block b runs on XCD b % 8; within one pair's range the blocks of
// one XCD take a contiguous run of the work in the order tile (fastest), channel
// block, so each XCD sweeps its own part of the frames.
__device__ __forceinline__ void fused_block_work(int b, int ntiles, int n_chblk,
                                                 int& tile_b, int& chb, int& pair) {
  const int per = ntiles * n_chblk;
  pair = b / per;
  const int idx = b - pair * per;
  const int x = idx & 7, j = idx >> 3;
  const int q = per >> 3, r = per & 7;
  const int w = x * q + min(x, r) + j;
  tile_b = w % ntiles;
  chb = w / ntiles;
}

template <int HR, int WR>
__global__ __launch_bounds__(64) void par_xspec_fused(ParArgs a, ClassSet cs,
                                                       const float* __restrict__ resid,
                                                       float* __restrict__ partial) {
  __shared__ __attribute__((aligned(16))) float lds[kBins * kXsStride];
  int tile_b, chb, pair;
  fused_block_work(blockIdx.x, cs.end[3], a.n_chblk, tile_b, chb, pair);
  for_class<HR, WR>(a, cs, tile_b, [&](auto hp, auto wp, int tile) {
    xspec_block<decltype(hp)::value, decltype(wp)::value>(a, tile, chb, pair, resid, partial, lds);
  });
}

template <int HR, int WR, bool ACC, bool NTT, bool INL>
__global__ __launch_bounds__(64) void par_recon_fused(ParArgs a, ClassSet cs,
                                                       const float* __restrict__ resid,
                                                       float* __restrict__ out,
                                                       const float4* __restrict__ coef,
                                                       const float* __restrict__ partial) {
  __shared__ float fb_lds[2 * kBins * kChb];
  __shared__ float4 coef_lds[INL ? kBins : 1];
  int tile_b, chb, pair;
  fused_block_work(blockIdx.x, cs.end[3], a.n_chblk, tile_b, chb, pair);
  pair = a.recon_order[pair];
  for_class<HR, WR>(a, cs, tile_b, [&](auto hp, auto wp, int tile) {
    recon_block<decltype(hp)::value, decltype(wp)::value, ACC, NTT, INL>(
        a, tile, chb, pair, resid, out, coef, fb_lds, partial, coef_lds);
  });
}

typedef void (*XspecFusedFn)(ParArgs, ClassSet, const float*, float*);
typedef void (*ReconFusedFn)(ParArgs, ClassSet, const float*, float*, const float4*, const float*);

// The fused kernels of one bottom-remainder height HR, for WR = 1..8
// (each row is compiled in its own translation unit).
struct FusedRow {
  XspecFusedFn xspec[8];
  ReconFusedFn recon_w[8], recon_a[8], recon_as[8];   // write, accumulate, accumulate streaming
  ReconFusedFn inl_w[8], inl_a[8], inl_as[8];         // the same with the gate computed inline
};

void fused_row_1(FusedRow& r);
void fused_row_2(FusedRow& r);
void fused_row_3(FusedRow& r);
void fused_row_4(FusedRow& r);
void fused_row_5(FusedRow& r);
void fused_row_6(FusedRow& r);
void fused_row_7(FusedRow& r);
void fused_row_8(FusedRow& r);

}  // namespace pardev
}  // namespace cast
