// Internal declarations shared by the libcast translation units (not installed).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/cast.h"

namespace cast {

// ---------------------------------------------------------------------------
// Error reporting (thread-local detail string, see cast_last_error_detail)
// ---------------------------------------------------------------------------
cast_status_t fail(cast_status_t st, const char* fmt, ...);
cast_status_t check_launch(const char* what);

constexpr size_t kWsAlign = 256;
inline size_t align_up(size_t x, size_t a = kWsAlign) { return (x + a - 1) / a * a; }

// ---------------------------------------------------------------------------
// bf16 <-> fp32 on the device (bf16 = upper half of binary32)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// ---------------------------------------------------------------------------
// Routing plan: how the pooled-mean scan is split (shared by the workspace
// query and the launch so both agree).
// ---------------------------------------------------------------------------
struct RoutePlan {
  int D;            // H * dh
  int ngrp;         // channel groups of kMeansCh
  int segs;         // n_a + M pooled rows
  size_t off_means, total;
};
constexpr int kMeansWaves = 8;      // waves per pooled-mean block
constexpr int kMeansCh = 128;       // channels per pooled-mean block (16 lanes x 8 bf16)
constexpr int kRankMaxM = 256;      // TopK by counting larger keys up to this many chunks
constexpr int kRouteMaxM = 4096;    // bitonic keys live in 32 KB of LDS

RoutePlan plan_route(int n_a, int S, int H, int dh, int M, int Bv);

// Pooled means of n_a frames of q (S tokens) and M chunks of k (Bv tokens):
// means [n_a + M, D] fp32 (q_bar rows first).  n_a may be 0.
cast_status_t launch_pool_means(const void* q, const void* k, int n_a, int S, int M, int Bv,
                                const RoutePlan& p, float* means, hipStream_t stream);

cast_status_t launch_route(const void* q, const void* k, int n_a, int S, int H, int dh, int M,
                           int Bv, int k_eff, float scale, float* scores_out, int32_t* idx_out,
                           const RoutePlan& plan, void* ws, hipStream_t stream);

// ---------------------------------------------------------------------------
// Reconstruction-coupled routing
// ---------------------------------------------------------------------------
constexpr int kCoupledMaxAnchors = 512;
constexpr int kCoupledMaxMask = 32768;   // n_a * M retain flags held in LDS by the solver

struct CoupledPlan {
  RoutePlan qk, v;      // pooled-mean scans of (Q, K) and of V
  size_t off_means_qk, off_means_v, off_u, total;
};
CoupledPlan plan_coupled(int n_a, int S, int H, int dh, int M, int Bv);

cast_status_t launch_coupled(const void* q, const void* k, const void* v, const float* gram,
                             const int* anchors, int n_a, int n_frames, int S, int H, int dh,
                             int M, int Bv, int k_eff, float scale, const cast_coupled_params_t& prm,
                             float* u_out, int32_t* idx_out, const CoupledPlan& plan, void* ws,
                             hipStream_t stream);

cast_status_t launch_wo_gram(const void* w_o, int D, int H, int dh, float* gram, hipStream_t stream);

// ---------------------------------------------------------------------------
// Attention
// ---------------------------------------------------------------------------
constexpr int kAttnMaxKeff = 1024;   // routed chunks per (anchor, head)
// Key split of the routed attention.  With U = n_a H ceil(S / 256) work units
// (anchor, head, 256-query tile) on C compute units, the last U mod C units (all
// of them when U < C) form a partial round; when it is at most half full they run
// as `split` pieces over disjoint key ranges (at most 8, each at least 16 key
// tiles), which the pieces' partial outputs need `bytes` of workspace for.
struct AttnSplitPlan {
  int n_full, n_split, split;
  size_t bytes;
};
AttnSplitPlan attn_split_plan(int n_a, int S, int H, int dh, long long L, int cus);
// compute units of the current device (cached per device), 0 if they cannot be read
int device_cu_count();

cast_status_t launch_anchor_attn(const void* q, const void* k_hist, const void* v_hist,
                                 const int32_t* idx, int k_eff, const void* k_cur,
                                 const void* v_cur, int n0, int n_a, int S, int H, int dh, int M,
                                 int Bv, float scale, void* out, float* lse_out,
                                 const AttnSplitPlan& plan, void* workspace, hipStream_t stream);

// ---------------------------------------------------------------------------
// PAR
// ---------------------------------------------------------------------------
constexpr int kParMaxTile = 8;
constexpr int kParMaxAnchors = 512;
constexpr int kParMaxFrames = 4096;
constexpr int kParNkxMax = kParMaxTile / 2 + 1;           // 5 stored columns
constexpr int kParBinsMax = kParMaxTile * kParNkxMax;     // 40 stored bins

struct ParPlan {
  int n_pairs, n_tiles, n_tiles_y, n_tiles_x;
  int chb;              // channels per xspec block
  int n_chblk;          // channel blocks for the cross-spectrum partial sums
  int bins_out;         // tile_h * (tile_w/2 + 1), debug-output row length
  size_t off_partial, off_coef, total;
};
ParPlan plan_par(int n_frames, int n_anchor, int Hg, int Wg, int D, const cast_par_params_t& p);

cast_status_t launch_par(const float* resid, const int* anchors, int n_anchor, int n_frames,
                         int Hg, int Wg, int D, const cast_par_params_t& p, float* out,
                         float* theta_out, float* gate_out, float* conf_out,
                         const ParPlan& plan, void* ws, hipStream_t stream);
// K_f = N_cur with the anchor update: out[a] = R_a or out[a] += R_a for every frame
cast_status_t launch_par_anchor_update(const float* resid, const int* anchors, int n_anchor,
                                       int Hg, int Wg, int D, int accumulate, float* out,
                                       hipStream_t stream);

// ---------------------------------------------------------------------------
// Control-aware frame selection
// ---------------------------------------------------------------------------
constexpr int kSelectMaxFrames = 4096;
int select_splits(int S, int D);   // partial sums per (branch, frame)
cast_status_t launch_frame_select(const void* cam, const void* act, int dtype, int n_cur, int S,
                                  int D, const int* anchors_prev, int n_prev, int k_f,
                                  const cast_select_params_t& p, int32_t* ages, float* r_out,
                                  float* score_out, int32_t* anchors_out, float* partial,
                                  hipStream_t stream);

// ---------------------------------------------------------------------------
// Spectral diagnostics
// ---------------------------------------------------------------------------
constexpr int kDiagMaxBands = 8;
size_t diag_workspace_bytes(int n_frames, int Hg, int Wg, int D, int tile_h, int tile_w);
cast_status_t launch_diag(const float* ref, const float* approx, const float* theta,
                          const int* anchors, int n_anchor, int n_frames, int Hg, int Wg, int D,
                          const cast_diag_params_t& p, float* nrmse_out, float* band_out,
                          float* phase_err_out, float* r_phase_out, float* r_mag_out, void* ws,
                          hipStream_t stream);
cast_status_t launch_phase_progress(const float* ref, const int* anchors, int n_anchor, int Hg,
                                    int Wg, int D, int tile_h, int tile_w, float* p_out,
                                    hipStream_t stream);

}  // namespace cast
