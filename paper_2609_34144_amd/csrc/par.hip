// Phase-Aware Reconstruction on gfx950 (Sec. 4.3; App. A.2; eq:block).
//
// Three stream-ordered kernels per call:
//   par_xspec  grid (tile, channel block of 64, anchor pair): every lane owns one
//              channel of one tile, transforms both anchors in registers and
//              writes its per-bin products F_b conj(F_a) and |F_b||F_a|; the 64
//              lanes are summed through LDS in fixed lane order into one partial
//              per (pair, tile, channel block).                        (eq:cross)
//   par_gate   grid (tile, pair, chunk of kGateTargets targets), four waves: one
//              lane per stored bin; each wave sums a quarter of the channel blocks'
//              partials, wave 0 adds the four in wave order, then computes eta,
//              reliability, theta (representative / mirror / self-conjugate), c_p,
//              nu, g; the waves share the blend coefficients of the chunk's targets
//              A_t = (1-alpha) e^{i g alpha theta} / (Hp Wp) and
//              B_t = alpha e^{-i g (1-alpha) theta} / (Hp Wp).
//                                              (App. A.2, eq:confidence, eq:gate)
//   par_recon  grid (tile, channel block, pair): every lane re-transforms the two
//              anchors of its pair in registers, then for each target of the pair
//              blends the spectra (eq:fcpasm), inverts and stores / accumulates.
//
// HBM traffic is the anchors (read by xspec and again by recon; the second read
// is usually served by the Infinity Cache) plus the skipped frames written (or
// read and written in accumulate mode).  Tiles are at most 8x8; every tile shape
// (Hp, Wp) in [1,8]^2 has its own fully unrolled code path.  With the default
// 8x8 tiling each pass is one launch over all tile classes (interior, right
// column, bottom row, corner; kernels in par_fused.hip), so small edge classes do
// not each pay a launch and a drain; other tilings launch per class.  The fused
// launches are 1-D grids that give each XCD a contiguous part of each pair's
// (tile, channel block) range (fused_block_work), so the waves of one XCD sweep
// neighbouring tiles of the same frames.
#include <algorithm>

#include "par_device.h"

namespace cast {

using namespace pardev;

namespace {

template <int HP, int WP>
__global__ __launch_bounds__(64) void par_xspec_kernel(ParArgs a, TileClass k,
                                                        const float* __restrict__ resid,
                                                        float* __restrict__ partial) {
  __shared__ __attribute__((aligned(16))) float lds[kBins * kXsStride];
  xspec_block<HP, WP>(a, class_tile(a, k, blockIdx.x), blockIdx.y, blockIdx.z, resid, partial, lds);
}

constexpr int kGateTargets = 8;   // targets per gate block
constexpr int kGateWaves = 4;     // waves per gate block
constexpr int kInlineBlocksPerCU = 7;   // resident reconstruction blocks with the gate inline

__global__ __launch_bounds__(64 * kGateWaves) void par_gate_kernel(ParArgs a,
                                                                    const float* __restrict__ partial,
                                                                    float4* __restrict__ coef) {
  __shared__ float part[kGateWaves][3][64];
  __shared__ float2 tg[64];
  const int tile = blockIdx.x, pair = blockIdx.y;
  const TileGeom g = tile_geom(a, tile);
  const int wv = threadIdx.x >> 6, b = threadIdx.x & 63;
  const int H = g.hp, W = g.wp;
  const BinSlot bs = bin_slot(b, H, W);
  // wave wv sums its quarter of the channel blocks' partials, in block order
  {
    float zr = 0.0f, zi = 0.0f, w = 0.0f;
    if (bs.active) {
      const float* src = partial + ((long long)pair * a.n_tiles + tile) * a.n_chblk * kVals +
                         (bs.sky * kNkx + bs.kx) * 3;
      const int j0 = a.n_chblk * wv / kGateWaves, j1 = a.n_chblk * (wv + 1) / kGateWaves;
#pragma unroll 4
      for (int j = j0; j < j1; ++j) {
        zr += src[(long long)j * kVals + 0];
        zi += src[(long long)j * kVals + 1];
        w += src[(long long)j * kVals + 2];
      }
    }
    part[wv][0][b] = zr;
    part[wv][1][b] = zi;
    part[wv][2][b] = w;
  }
  __syncthreads();
  if (wv == 0) {
    float zr = 0.0f, zi = 0.0f, w = 0.0f;
    if (bs.active) {
#pragma unroll
      for (int q = 0; q < kGateWaves; ++q) {
        zr += part[q][0][b];
        zi += part[q][1][b];
        w += part[q][2][b];
      }
    }
    const BinGate bg = bin_gate(a, bs, H, W, zr, zi, w);
    // optional diagnostics, laid out per the caller's tile_h x (tile_w/2+1) rows
    // (written by the first target chunk)
    const int nkx_out = a.tile_w / 2 + 1;
    if (blockIdx.z == 0 && b < kBins && bs.ky < a.tile_h && bs.kx < nkx_out) {
      const long long o = ((long long)pair * a.n_tiles + tile) * a.bins_out + bs.ky * nkx_out + bs.kx;
      if (a.theta_out) a.theta_out[o] = bs.active ? bg.theta : 0.0f;
      if (a.gate_out) a.gate_out[o] = bs.active ? bg.gate : 0.0f;
    }
    if (a.conf_out && b == 0 && blockIdx.z == 0) a.conf_out[(long long)pair * a.n_tiles + tile] = bg.conf;
    tg[b] = make_float2(bg.theta, bg.gate);
  }
  __syncthreads();
  if (b >= kBins) return;
  const float theta = tg[b].x, gate = tg[b].y;
  // blend coefficients of this chunk of the pair's targets (eq:block composition):
  // target k of the pair is fa+1+k for the interior, then (first pair) the frames
  // before the first anchor, then (last pair) the frames after the last anchor
  const int n_pairs = a.n_anchor - 1;
  const int fa = a.anchors[pair], fb = a.anchors[pair + 1];
  const int n_in = fb - fa - 1, n_lo = pair == 0 ? fa : 0;
  const int n_hi = pair == n_pairs - 1 ? a.n_frames - fb - 1 : 0;
  const int k0 = blockIdx.z * kGateTargets, k1 = min(k0 + kGateTargets, n_in + n_lo + n_hi);
  for (int k = k0 + wv; k < k1; k += kGateWaves) {
    const int t = k < n_in ? fa + 1 + k : (k < n_in + n_lo ? k - n_in : fb + 1 + (k - n_in - n_lo));
    coef[((long long)t * a.n_tiles + tile) * kBins + b] = blend_coef(t, fa, fb, theta, gate, H, W,
                                                                      bs.active);
  }
}

template <int HP, int WP, bool ACC>
__global__ __launch_bounds__(64) void par_recon_kernel(ParArgs a, TileClass k,
                                                        const float* __restrict__ resid,
                                                        float* __restrict__ out,
                                                        const float4* __restrict__ coef) {
  __shared__ float fb_lds[2 * kBins * kChb];
  recon_block<HP, WP, ACC, false>(a, class_tile(a, k, blockIdx.x), blockIdx.y, blockIdx.z, resid,
                                  out, coef, fb_lds);
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

// Table of fused-kernel rows, filled on first use (the rows live in their own
// translation units).
const FusedRow& fused_row(int hr) {
  static const FusedRow* rows = [] {
    static FusedRow r[8];
    fused_row_1(r[0]);
    fused_row_2(r[1]);
    fused_row_3(r[2]);
    fused_row_4(r[3]);
    fused_row_5(r[4]);
    fused_row_6(r[5]);
    fused_row_7(r[6]);
    fused_row_8(r[7]);
    return r;
  }();
  return rows[hr - 1];
}

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

// K_f = N_cur (every frame an anchor, nothing to reconstruct) with the anchor
// update: out[a] = R_a or out[a] += R_a, four consecutive elements per thread.
constexpr int kUpdThreads = 256;
__global__ __launch_bounds__(kUpdThreads) void par_anchor_update_kernel(ParArgs a,
                                                                        const float* __restrict__ resid,
                                                                        float* __restrict__ out) {
  const long long f = a.anchors[blockIdx.y];
  const long long e0 = ((long long)blockIdx.x * kUpdThreads + threadIdx.x) * 4;
  const float* src = resid + f * a.frame_elems;
  float* dst = out + f * a.frame_elems;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const long long e = e0 + k;
    if (e < a.frame_elems) dst[e] = a.accumulate ? dst[e] + src[e] : src[e];
  }
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
  a.update_anchors = p.update_anchors;
  for (int j = 0; j < n_anchor; ++j) a.anchors[j] = (short)anchors[j];
  // gate grid: (tile, pair, chunk of kGateTargets targets of the pair); the frames
  // each pair's reconstruction blocks write (targets, and anchors when updated)
  // order the fused reconstruction launch, most first (ties by pair index)
  int max_targets = 0;
  int work[kParMaxAnchors];
  for (int pr = 0; pr + 1 < n_anchor; ++pr) {
    int n = anchors[pr + 1] - anchors[pr] - 1;
    if (pr == 0) n += anchors[0];
    if (pr + 2 == n_anchor) n += n_frames - anchors[n_anchor - 1] - 1;
    max_targets = n > max_targets ? n : max_targets;
    work[pr] = n + (p.update_anchors ? (pr + 2 == n_anchor ? 2 : 1) : 0);
    a.recon_order[pr] = (short)pr;
  }
  std::stable_sort(a.recon_order, a.recon_order + (n_anchor - 1),
                   [&](short x, short y) { return work[x] > work[y]; });
  const dim3 gate_grid(pl.n_tiles, pl.n_pairs,
                       max_targets > 0 ? (max_targets + kGateTargets - 1) / kGateTargets : 1);

  cast_status_t st;
  if (p.tile_h == 8 && p.tile_w == 8) {
    // default tiling: one fused launch per pass covers every tile class
    const int nyf = Hg / 8, hr = Hg % 8, nxf = Wg / 8, wr = Wg % 8;
    ClassSet cs{};
    cs.k[0] = {0, 0, nxf};
    cs.k[1] = {0, nxf, 1};
    cs.k[2] = {nyf, 0, nxf};
    cs.k[3] = {nyf, nxf, 1};
    cs.end[0] = nyf * nxf;
    cs.end[1] = cs.end[0] + (wr > 0 ? nyf : 0);
    cs.end[2] = cs.end[1] + (hr > 0 ? nxf : 0);
    cs.end[3] = cs.end[2] + (hr > 0 && wr > 0 ? 1 : 0);
    const FusedRow& row = fused_row(hr > 0 ? hr : 8);
    const int wi = (wr > 0 ? wr : 8) - 1;
    const dim3 grid((unsigned)cs.end[3] * pl.n_chblk * pl.n_pairs);
    hipLaunchKernelGGL(row.xspec[wi], grid, dim3(kChb), 0, stream, a, cs, resid, partial);
    st = check_launch("par_xspec");
    if (st != CAST_OK) return st;
    // When the reconstruction grid fits in one round of resident blocks (kInlineBlocksPerCU
    // per compute unit: the register file allows 8, LDS with the coefficients 7), each
    // block computes its tile's gate itself, and the gate launch, a serial step of
    // its own, goes; the debug outputs come from the gate launch.
    const int cus = device_cu_count();
    const bool inl = theta_out == nullptr && gate_out == nullptr && conf_out == nullptr && cus > 0 &&
                     (long long)grid.x <= (long long)kInlineBlocksPerCU * cus;
    if (!inl) {
      hipLaunchKernelGGL(par_gate_kernel, gate_grid, dim3(64 * kGateWaves), 0, stream, a,
                         (const float*)partial, coef);
      st = check_launch("par_gate");
      if (st != CAST_OK) return st;
    }
    // accumulate mode with several pairs: stream the targets (see recon_body)
    const ReconFusedFn rf = !p.accumulate ? (inl ? row.inl_w[wi] : row.recon_w[wi])
                            : (pl.n_pairs > 1 ? (inl ? row.inl_as[wi] : row.recon_as[wi])
                                              : (inl ? row.inl_a[wi] : row.recon_a[wi]));
    hipLaunchKernelGGL(rf, grid, dim3(kChb), 0, stream, a, cs, resid, out, (const float4*)coef,
                       (const float*)partial);
    return check_launch("par_recon");
  }
  // other tilings: one launch per tile class and pass
  ClassLaunch cls[4];
  const int ncls = tile_classes(Hg, Wg, p.tile_h, p.tile_w, cls);
  for (int j = 0; j < ncls; ++j) {
    dim3 grid(cls[j].ntiles, pl.n_chblk, pl.n_pairs);
    hipLaunchKernelGGL(kXspec[cls[j].hp - 1][cls[j].wp - 1], grid, dim3(kChb), 0, stream, a,
                       cls[j].k, resid, partial);
    st = check_launch("par_xspec");
    if (st != CAST_OK) return st;
  }
  hipLaunchKernelGGL(par_gate_kernel, gate_grid, dim3(64 * kGateWaves), 0, stream, a,
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

cast_status_t launch_par_anchor_update(const float* resid, const int* anchors, int n_anchor,
                                       int Hg, int Wg, int D, int accumulate, float* out,
                                       hipStream_t stream) {
  ParArgs a{};
  a.frame_elems = (long long)Hg * Wg * D;
  a.n_anchor = n_anchor;
  a.accumulate = accumulate;
  for (int j = 0; j < n_anchor; ++j) a.anchors[j] = (short)anchors[j];
  const long long per_block = 4LL * kUpdThreads;
  dim3 grid((unsigned)((a.frame_elems + per_block - 1) / per_block), (unsigned)n_anchor);
  hipLaunchKernelGGL(par_anchor_update_kernel, grid, dim3(kUpdThreads), 0, stream, a, resid, out);
  return check_launch("par_anchor_update");
}

}  // namespace cast
