// C ABI entry points of libcast: argument validation, workspace sizing and
// dispatch to the kernel launchers.  Every entry point validates all of its
// arguments before anything is enqueued and reports failures as a status plus
// a thread-local detail string.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>

#include "cast_common.h"

namespace cast {

static thread_local char g_detail[512] = "";

cast_status_t fail(cast_status_t st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_detail, sizeof(g_detail), fmt, ap);
  va_end(ap);
  return st;
}

cast_status_t check_launch(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(CAST_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return CAST_OK;
}

static bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

static cast_status_t check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return CAST_OK;
  if (ws == nullptr) return fail(CAST_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
  if (!aligned(ws, kWsAlign)) return fail(CAST_ERR_WORKSPACE, "workspace must be %zu-byte aligned", kWsAlign);
  if (have < need) return fail(CAST_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return CAST_OK;
}

static bool dh_ok(int dh) { return dh == 32 || dh == 64 || dh == 128; }

// Scratch of cast_par_reconstruct_noalloc: one copy per GPU the library runs on,
// held until the process ends.  In host code `scratch` names a host-side stand-in,
// not device memory: kernels get the device address that hipGetSymbolAddress
// returns for the current device, looked up once per device and kept.
constexpr size_t kParStaticScratchBytes = CAST_PAR_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kParStaticScratchBytes];

static cast_status_t static_scratch_ptr(void** out) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* ptrs[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(CAST_ERR_HIP, "par (static scratch): hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(CAST_ERR_UNSUPPORTED, "par (static scratch): device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(mu);
  if (ptrs[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(CAST_ERR_HIP, "par (static scratch): hipGetSymbolAddress: %s", hipGetErrorString(e));
    ptrs[dev] = p;
  }
  *out = ptrs[dev];
  return CAST_OK;
}

}  // namespace cast

using namespace cast;

extern "C" {

const char* cast_status_string(int s) {
  switch (s) {
    case CAST_OK: return "CAST_OK";
    case CAST_ERR_NULL: return "CAST_ERR_NULL";
    case CAST_ERR_SHAPE: return "CAST_ERR_SHAPE";
    case CAST_ERR_ANCHORS: return "CAST_ERR_ANCHORS";
    case CAST_ERR_UNSUPPORTED: return "CAST_ERR_UNSUPPORTED";
    case CAST_ERR_WORKSPACE: return "CAST_ERR_WORKSPACE";
    case CAST_ERR_HIP: return "CAST_ERR_HIP";
    default: return "CAST_ERR_UNKNOWN";
  }
}

const char* cast_last_error_detail(void) { return g_detail; }

int cast_abi_version(void) { return CAST_ABI_VERSION; }

// ------------------------------------------------------------------ routing

static cast_status_t route_shape_check(int n_a, int S, int H, int dh, int M, int Bv) {
  if (n_a < 1 || S < 1 || H < 1 || M < 0 || Bv < 1)
    return fail(CAST_ERR_SHAPE, "route: need n_a>=1, S>=1, H>=1, M>=0, Bv>=1 (got %d %d %d %d %d)",
                n_a, S, H, M, Bv);
  if (!dh_ok(dh)) return fail(CAST_ERR_UNSUPPORTED, "route: dh must be 32, 64 or 128 (got %d)", dh);
  if (M > kRouteMaxM) return fail(CAST_ERR_UNSUPPORTED, "route: M=%d exceeds %d chunks", M, kRouteMaxM);
  if ((long long)S * H * dh >= (1LL << 31) || (long long)Bv * H * dh >= (1LL << 31))
    return fail(CAST_ERR_UNSUPPORTED, "route: one frame or chunk must hold < 2^31 elements");
  if ((long long)M * Bv >= (1LL << 31) || (long long)n_a * S >= (1LL << 31))
    return fail(CAST_ERR_UNSUPPORTED, "route: token counts must stay below 2^31");
  return CAST_OK;
}

size_t cast_route_kv_workspace_bytes(int n_a, int S, int H, int dh, int M, int Bv) {
  if (route_shape_check(n_a, S, H, dh, M, Bv) != CAST_OK || M == 0) return 0;
  return plan_route(n_a, S, H, dh, M, Bv).total;
}

cast_status_t cast_route_kv(const void* q, const void* k_hist, int n_a, int S, int H, int dh,
                            int M, int Bv, int topk, float scale, float* scores_out,
                            int32_t* idx_out, int* k_eff_out, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  if (k_eff_out == nullptr) return fail(CAST_ERR_NULL, "route: k_eff_out is NULL");
  cast_status_t st = route_shape_check(n_a, S, H, dh, M, Bv);
  if (st != CAST_OK) return st;
  if (topk < 1) return fail(CAST_ERR_SHAPE, "route: topk must be >= 1 (got %d)", topk);
  if (M == 0) { *k_eff_out = 0; return CAST_OK; }          // routing bypassed (App. B.3)
  if (q == nullptr || k_hist == nullptr || idx_out == nullptr)
    return fail(CAST_ERR_NULL, "route: q, k_hist and idx_out are required");
  if (!aligned(q, 16) || !aligned(k_hist, 16))
    return fail(CAST_ERR_SHAPE, "route: q and k_hist must be 16-byte aligned");
  if (!aligned(idx_out, 4) || !aligned(scores_out, 4))
    return fail(CAST_ERR_SHAPE, "route: idx_out and scores_out must be 4-byte aligned");
  RoutePlan plan = plan_route(n_a, S, H, dh, M, Bv);
  st = check_ws(workspace, workspace_bytes, plan.total);
  if (st != CAST_OK) return st;
  int k_eff = topk < M ? topk : M;
  st = launch_route(q, k_hist, n_a, S, H, dh, M, Bv, k_eff, scale, scores_out, idx_out, plan,
                    workspace, stream);
  if (st != CAST_OK) return st;
  *k_eff_out = k_eff;
  return CAST_OK;
}

// ------------------------------------------------- coupled routing (NEXT)

void cast_coupled_params_default(cast_coupled_params_t* p) {
  if (p == nullptr) return;
  p->l_anc = 1.0f;
  p->l_rec = 1.0f;
  p->passes = 2;
  p->tol = 1e-6f;
  p->eps = 1e-8f;
}

cast_status_t cast_wo_gram(const void* w_o, int D, int H, int dh, float* gram_out,
                           hipStream_t stream) {
  if (H < 1 || !dh_ok(dh) || (long long)H * dh != D)
    return fail(CAST_ERR_SHAPE, "wo_gram: need H>=1, dh in {32,64,128}, D == H*dh (got %d %d %d)",
                D, H, dh);
  if ((long long)D * D >= (1LL << 31))
    return fail(CAST_ERR_UNSUPPORTED, "wo_gram: D*D must stay below 2^31");
  if (w_o == nullptr || gram_out == nullptr) return fail(CAST_ERR_NULL, "wo_gram: null pointer");
  if (!aligned(w_o, 16) || !aligned(gram_out, 16))
    return fail(CAST_ERR_SHAPE, "wo_gram: pointers must be 16-byte aligned");
  return launch_wo_gram(w_o, D, H, dh, gram_out, stream);
}

size_t cast_route_coupled_workspace_bytes(int n_a, int S, int H, int dh, int M, int Bv) {
  if (route_shape_check(n_a, S, H, dh, M, Bv) != CAST_OK || M == 0) return 0;
  return plan_coupled(n_a, S, H, dh, M, Bv).total;
}

cast_status_t cast_route_coupled(const void* q, const void* k_hist, const void* v_hist,
                                 const float* gram, const int* anchors, int n_a, int n_frames,
                                 int S, int H, int dh, int M, int Bv, int topk, float scale,
                                 const cast_coupled_params_t* params, float* u_out,
                                 int32_t* idx_out, int* k_eff_out, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  if (k_eff_out == nullptr) return fail(CAST_ERR_NULL, "coupled: k_eff_out is NULL");
  cast_status_t st = route_shape_check(n_a, S, H, dh, M, Bv);
  if (st != CAST_OK) return st;
  if (topk < 1) return fail(CAST_ERR_SHAPE, "coupled: topk must be >= 1 (got %d)", topk);
  if (params == nullptr) return fail(CAST_ERR_NULL, "coupled: params is NULL");
  if (!(params->l_anc >= 0.0f) || !(params->l_rec >= 0.0f) || !(params->tol >= 0.0f) ||
      !(params->eps >= 0.0f) || params->passes < 0 || params->passes > 1000)
    return fail(CAST_ERR_SHAPE, "coupled: weights, tol, eps must be >= 0 and 0 <= passes <= 1000");
  if (anchors == nullptr) return fail(CAST_ERR_NULL, "coupled: anchors is NULL");
  if (n_a > kCoupledMaxAnchors)
    return fail(CAST_ERR_UNSUPPORTED, "coupled: n_a=%d exceeds %d anchors", n_a, kCoupledMaxAnchors);
  if (n_frames < n_a || n_frames > 32767)
    return fail(CAST_ERR_SHAPE, "coupled: n_frames=%d must be in [n_a, 32767]", n_frames);
  for (int j = 0; j < n_a; ++j) {
    if (anchors[j] < 0 || anchors[j] >= n_frames || (j > 0 && anchors[j] <= anchors[j - 1]))
      return fail(CAST_ERR_ANCHORS, "coupled: anchors must be strictly increasing in [0, n_frames)");
  }
  if (M == 0) { *k_eff_out = 0; return CAST_OK; }
  if ((long long)n_a * M > kCoupledMaxMask)
    return fail(CAST_ERR_UNSUPPORTED, "coupled: n_a*M=%lld exceeds %d", (long long)n_a * M,
                kCoupledMaxMask);
  if (q == nullptr || k_hist == nullptr || v_hist == nullptr || gram == nullptr || idx_out == nullptr)
    return fail(CAST_ERR_NULL, "coupled: q, k_hist, v_hist, gram and idx_out are required");
  if (!aligned(q, 16) || !aligned(k_hist, 16) || !aligned(v_hist, 16) || !aligned(gram, 16))
    return fail(CAST_ERR_SHAPE, "coupled: q, k_hist, v_hist, gram must be 16-byte aligned");
  if (!aligned(idx_out, 4) || !aligned(u_out, 4))
    return fail(CAST_ERR_SHAPE, "coupled: idx_out and u_out must be 4-byte aligned");
  CoupledPlan plan = plan_coupled(n_a, S, H, dh, M, Bv);
  st = check_ws(workspace, workspace_bytes, plan.total);
  if (st != CAST_OK) return st;
  const int k_eff = topk < M ? topk : M;
  st = launch_coupled(q, k_hist, v_hist, gram, anchors, n_a, n_frames, S, H, dh, M, Bv, k_eff,
                      scale, *params, u_out, idx_out, plan, workspace, stream);
  if (st != CAST_OK) return st;
  *k_eff_out = k_eff;
  return CAST_OK;
}

// ---------------------------------------------------------------- attention

size_t cast_anchor_attn_workspace_bytes(int n_a, int S, int H, int dh, int k_eff, int n0, int Bv) {
  if (n_a < 1 || S < 1 || H < 1 || !dh_ok(dh) || k_eff < 0 || n0 < 0 || Bv < 1) return 0;
  const long long L = (long long)n0 + (long long)k_eff * Bv;
  if (L < 1) return 0;
  return attn_split_plan(n_a, S, H, dh, L, device_cu_count()).bytes;
}

cast_status_t cast_anchor_attn(const void* q, const void* k_hist, const void* v_hist,
                               const int32_t* idx, int k_eff, const void* k_cur,
                               const void* v_cur, int n0, int n_a, int S, int H, int dh, int M,
                               int Bv, float scale, void* out, float* lse_out,
                               void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (n_a < 1 || S < 1 || H < 1 || M < 0 || Bv < 1 || n0 < 0 || k_eff < 0)
    return fail(CAST_ERR_SHAPE, "attn: need n_a,S,H,Bv>=1 and M,n0,k_eff>=0");
  if (!dh_ok(dh)) return fail(CAST_ERR_UNSUPPORTED, "attn: dh must be 32, 64 or 128 (got %d)", dh);
  if (k_eff > M) return fail(CAST_ERR_SHAPE, "attn: k_eff=%d exceeds M=%d", k_eff, M);
  if (k_eff > kAttnMaxKeff)
    return fail(CAST_ERR_UNSUPPORTED, "attn: k_eff=%d exceeds %d routed chunks", k_eff, kAttnMaxKeff);
  long long L = (long long)n0 + (long long)k_eff * Bv;
  if (L < 1) return fail(CAST_ERR_SHAPE, "attn: nothing to attend to (n0 = 0 and k_eff = 0)");
  if (L * (long long)Bv >= (1LL << 40) || L >= (1LL << 31) || L >= (1LL << 24) * (long long)Bv)
    return fail(CAST_ERR_UNSUPPORTED, "attn: key sequence too long for the row indexing");
  if (!(scale > 0.0f) || scale > 3.0e38f)
    return fail(CAST_ERR_SHAPE, "attn: scale must be finite and > 0");
  if ((long long)M * Bv >= (1LL << 31) || (long long)n_a * S >= (1LL << 31))
    return fail(CAST_ERR_UNSUPPORTED, "attn: token counts must stay below 2^31");
  if ((long long)M * Bv * H * dh * 2 >= (1LL << 32) || (long long)n0 * H * dh * 2 >= (1LL << 32))
    return fail(CAST_ERR_UNSUPPORTED, "attn: K/V history and current tensors must each be < 4 GiB");
  if (q == nullptr || out == nullptr) return fail(CAST_ERR_NULL, "attn: q and out are required");
  if (k_eff > 0 && (k_hist == nullptr || v_hist == nullptr || idx == nullptr))
    return fail(CAST_ERR_NULL, "attn: k_hist, v_hist and idx are required when k_eff > 0");
  if (n0 > 0 && (k_cur == nullptr || v_cur == nullptr))
    return fail(CAST_ERR_NULL, "attn: k_cur and v_cur are required when n0 > 0");
  const void* ptrs[] = {q, k_hist, v_hist, k_cur, v_cur, out};
  for (const void* p : ptrs)
    if (p != nullptr && !aligned(p, 16)) return fail(CAST_ERR_SHAPE, "attn: tensors must be 16-byte aligned");
  if (!aligned(idx, 4) || !aligned(lse_out, 4))
    return fail(CAST_ERR_SHAPE, "attn: idx and lse_out must be 4-byte aligned");
  // no workspace: every unit runs whole
  AttnSplitPlan plan{(int)((long long)n_a * H * ((S + 255) / 256)), 0, 1, 0};
  if (workspace != nullptr) {
    if (!aligned(workspace, kWsAlign))
      return fail(CAST_ERR_WORKSPACE, "attn: workspace must be %zu-byte aligned", kWsAlign);
    plan = attn_split_plan(n_a, S, H, dh, L, device_cu_count());
    if (workspace_bytes < plan.bytes)
      return fail(CAST_ERR_WORKSPACE, "attn: workspace has %zu bytes, %zu needed", workspace_bytes, plan.bytes);
  }
  return launch_anchor_attn(q, k_hist, v_hist, idx, k_eff, k_cur, v_cur, n0, n_a, S, H, dh, M,
                            Bv, scale, out, lse_out, plan, workspace, stream);
}

// ---------------------------------------------------------------------- PAR

void cast_par_params_default(cast_par_params_t* p) {
  if (p == nullptr) return;
  p->tile_h = 8;
  p->tile_w = 8;
  p->tau_low = 0.25f;
  p->tau_high = 0.75f;
  p->q = 2.0f;
  p->T = 0.10f;
  p->eta_rel = 1e-6f;
  p->eta_abs = 1e-8f;
  p->eps = 1e-8f;
  p->gate_mode = 0;
  p->accumulate = 0;
  p->update_anchors = 0;
}

static cast_status_t par_shape_check(int n_frames, int n_anchor, int Hg, int Wg, int D,
                                     const cast_par_params_t* p) {
  if (p == nullptr) return fail(CAST_ERR_NULL, "par: params is NULL");
  if (n_frames < 1 || Hg < 1 || Wg < 1 || D < 1 || n_anchor < 1)
    return fail(CAST_ERR_SHAPE, "par: need n_frames, n_anchor, Hg, Wg, D >= 1");
  if (n_frames > kParMaxFrames) return fail(CAST_ERR_UNSUPPORTED, "par: n_frames > %d", kParMaxFrames);
  if (n_anchor > kParMaxAnchors) return fail(CAST_ERR_UNSUPPORTED, "par: n_anchor > %d", kParMaxAnchors);
  if (n_anchor > n_frames) return fail(CAST_ERR_ANCHORS, "par: more anchors than frames");
  if (p->tile_h < 1 || p->tile_h > kParMaxTile || p->tile_w < 1 || p->tile_w > kParMaxTile)
    return fail(CAST_ERR_UNSUPPORTED, "par: tile edges must be in [1, %d]", kParMaxTile);
  if (p->gate_mode < 0 || p->gate_mode > 2) return fail(CAST_ERR_SHAPE, "par: gate_mode must be 0, 1 or 2");
  if (p->accumulate != 0 && p->accumulate != 1) return fail(CAST_ERR_SHAPE, "par: accumulate must be 0 or 1");
  if (p->update_anchors != 0 && p->update_anchors != 1)
    return fail(CAST_ERR_SHAPE, "par: update_anchors must be 0 or 1");
  if (!(p->T > 0.0f) || !(p->q > 0.0f) || !(p->tau_high >= p->tau_low))
    return fail(CAST_ERR_SHAPE, "par: eq:gate needs q > 0, T > 0, tau_high >= tau_low");
  if ((long long)Hg * Wg * D >= (1LL << 30))
    return fail(CAST_ERR_UNSUPPORTED, "par: one frame must hold < 2^30 elements (4 GiB)");
  return CAST_OK;
}

size_t cast_par_workspace_bytes(int n_frames, int n_anchor, int Hg, int Wg, int D,
                                const cast_par_params_t* params) {
  if (par_shape_check(n_frames, n_anchor, Hg, Wg, D, params) != CAST_OK) return 0;
  if (n_anchor == n_frames || n_anchor < 2) return 0;
  return plan_par(n_frames, n_anchor, Hg, Wg, D, *params).total;
}

}  // extern "C"

// The validation and dispatch of cast_par_reconstruct.  With `static_scratch`
// the workspace is this device's static scratch array (found on first use) and
// a plan larger than it is rejected.
static cast_status_t par_reconstruct(const float* resid, const int* anchors, int n_anchor,
                                     int n_frames, int Hg, int Wg, int D,
                                     const cast_par_params_t* params, float* out,
                                     float* theta_out, float* gate_out, float* conf_out,
                                     void* workspace, size_t workspace_bytes, bool static_scratch,
                                     hipStream_t stream) {
  if (anchors == nullptr) return fail(CAST_ERR_NULL, "par: anchors is NULL");
  cast_status_t st = par_shape_check(n_frames, n_anchor, Hg, Wg, D, params);
  if (st != CAST_OK) return st;
  for (int j = 0; j < n_anchor; ++j) {
    if (anchors[j] < 0 || anchors[j] >= n_frames)
      return fail(CAST_ERR_ANCHORS, "par: anchor %d = %d outside [0, %d)", j, anchors[j], n_frames);
    if (j > 0 && anchors[j] <= anchors[j - 1])
      return fail(CAST_ERR_ANCHORS, "par: anchors must be strictly increasing (index %d)", j);
  }
  const bool bypass = n_anchor == n_frames;                 // K_f = N_cur (App. A.1)
  if (bypass && !params->update_anchors) return CAST_OK;
  if (!bypass && n_anchor < 2) return fail(CAST_ERR_ANCHORS, "par: reconstruction needs K_f >= 2 anchors");
  if (resid == nullptr || out == nullptr) return fail(CAST_ERR_NULL, "par: resid and out are required");
  if (!aligned(resid, 4) || !aligned(out, 4) || !aligned(theta_out, 4) || !aligned(gate_out, 4) ||
      !aligned(conf_out, 4))
    return fail(CAST_ERR_SHAPE, "par: misaligned buffers");
  if (params->update_anchors) {
    // anchor slots of out are written while other blocks read the anchors of resid
    const unsigned long long bytes = (unsigned long long)n_frames * Hg * Wg * D * sizeof(float);
    const unsigned long long r0 = (unsigned long long)(uintptr_t)resid, o0 = (unsigned long long)(uintptr_t)out;
    if (r0 < o0 + bytes && o0 < r0 + bytes)
      return fail(CAST_ERR_SHAPE, "par: update_anchors needs out not to overlap resid");
  }
  if (bypass)
    return launch_par_anchor_update(resid, anchors, n_anchor, Hg, Wg, D, params->accumulate, out, stream);
  ParPlan plan = plan_par(n_frames, n_anchor, Hg, Wg, D, *params);
  if (static_scratch) {
    if (plan.total > kParStaticScratchBytes)
      return fail(CAST_ERR_WORKSPACE,
                  "par (static scratch): these sizes need %zu bytes of scratch, the static "
                  "scratch holds %zu; use cast_par_reconstruct with a workspace",
                  plan.total, kParStaticScratchBytes);
    st = static_scratch_ptr(&workspace);
    if (st != CAST_OK) return st;
    workspace_bytes = kParStaticScratchBytes;
  }
  st = check_ws(workspace, workspace_bytes, plan.total);
  if (st != CAST_OK) return st;
  return launch_par(resid, anchors, n_anchor, n_frames, Hg, Wg, D, *params, out, theta_out,
                    gate_out, conf_out, plan, workspace, stream);
}

extern "C" {

cast_status_t cast_par_reconstruct(const float* resid, const int* anchors, int n_anchor,
                                   int n_frames, int Hg, int Wg, int D,
                                   const cast_par_params_t* params, float* out,
                                   float* theta_out, float* gate_out, float* conf_out,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  return par_reconstruct(resid, anchors, n_anchor, n_frames, Hg, Wg, D, params, out, theta_out,
                         gate_out, conf_out, workspace, workspace_bytes, false, stream);
}

cast_status_t cast_par_reconstruct_noalloc(const float* resid, const int* anchors, int n_anchor,
                                           int n_frames, int Hg, int Wg, int D,
                                           const cast_par_params_t* params, float* out,
                                           float* theta_out, float* gate_out, float* conf_out,
                                           hipStream_t stream) {
  return par_reconstruct(resid, anchors, n_anchor, n_frames, Hg, Wg, D, params, out, theta_out,
                         gate_out, conf_out, nullptr, 0, true, stream);
}

size_t cast_par_static_scratch_bytes(void) { return kParStaticScratchBytes; }

// ---------------------------------------------------------------------------
// Control-aware frame selection
// ---------------------------------------------------------------------------
void cast_select_params_default(cast_select_params_t* p) {
  if (p == nullptr) return;
  p->lambda_cov = 0.5f;
  p->eps = 1e-8f;
}

static cast_status_t select_shape_check(int n_cur, int S, int D) {
  if (n_cur < 1 || S < 1 || D < 1) return fail(CAST_ERR_SHAPE, "frame_select: need n_cur, S, D >= 1");
  if (n_cur > kSelectMaxFrames)
    return fail(CAST_ERR_UNSUPPORTED, "frame_select: n_cur > %d", kSelectMaxFrames);
  if ((long long)S * D >= (1LL << 40)) return fail(CAST_ERR_UNSUPPORTED, "frame_select: frame too large");
  return CAST_OK;
}

size_t cast_frame_select_workspace_bytes(int n_cur, int S, int D) {
  if (select_shape_check(n_cur, S, D) != CAST_OK) return 0;
  return align_up((size_t)2 * n_cur * select_splits(S, D) * sizeof(float));
}

cast_status_t cast_frame_select(const void* delta_cam, const void* delta_act, int dtype,
                                int n_cur, int S, int D, const int* anchors_prev, int n_prev,
                                int k_f, const cast_select_params_t* params, int32_t* ages,
                                float* r_out, float* score_out, int32_t* anchors_out,
                                void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (params == nullptr || anchors_prev == nullptr || ages == nullptr || anchors_out == nullptr)
    return fail(CAST_ERR_NULL, "frame_select: params, anchors_prev, ages and anchors_out are required");
  cast_status_t st = select_shape_check(n_cur, S, D);
  if (st != CAST_OK) return st;
  if (dtype != 0 && dtype != 1) return fail(CAST_ERR_SHAPE, "frame_select: dtype must be 0 (fp32) or 1 (bf16)");
  if (!(params->lambda_cov >= 0.0f) || !(params->eps >= 0.0f) || params->lambda_cov > 1e30f || params->eps > 1e30f)
    return fail(CAST_ERR_SHAPE, "frame_select: lambda_cov and eps must be finite and >= 0");
  if (k_f < 1 || k_f > n_cur) return fail(CAST_ERR_SHAPE, "frame_select: k_f must be in [1, n_cur]");
  if (n_prev < 1 || n_prev > n_cur) return fail(CAST_ERR_ANCHORS, "frame_select: n_prev must be in [1, n_cur]");
  for (int j = 0; j < n_prev; ++j) {
    if (anchors_prev[j] < 0 || anchors_prev[j] >= n_cur)
      return fail(CAST_ERR_ANCHORS, "frame_select: anchor %d = %d outside [0, %d)", j, anchors_prev[j], n_cur);
    if (j > 0 && anchors_prev[j] <= anchors_prev[j - 1])
      return fail(CAST_ERR_ANCHORS, "frame_select: anchors must be strictly increasing (index %d)", j);
  }
  const size_t esz = dtype == 0 ? 4 : 2;
  if (!aligned(ages, 4) || !aligned(anchors_out, 4) || !aligned(r_out, 4) || !aligned(score_out, 4) ||
      !aligned(delta_cam, esz) || !aligned(delta_act, esz))
    return fail(CAST_ERR_SHAPE, "frame_select: misaligned buffers");
  if (delta_cam != nullptr || delta_act != nullptr) {
    st = check_ws(workspace, workspace_bytes, cast_frame_select_workspace_bytes(n_cur, S, D));
    if (st != CAST_OK) return st;
  }
  return launch_frame_select(delta_cam, delta_act, dtype, n_cur, S, D, anchors_prev, n_prev, k_f,
                             *params, ages, r_out, score_out, anchors_out,
                             static_cast<float*>(workspace), stream);
}

// ---------------------------------------------------------------------------
// Spectral diagnostics
// ---------------------------------------------------------------------------
void cast_diag_params_default(cast_diag_params_t* p) {
  if (p == nullptr) return;
  p->tile_h = 8;
  p->tile_w = 8;
  p->n_bands = 3;
  for (int k = 0; k < 9; ++k) p->band_edges[k] = 0.0f;
  p->band_edges[1] = 1.0f / 3.0f;
  p->band_edges[2] = 2.0f / 3.0f;
  p->band_edges[3] = 1.0f;
  p->eps = 1e-8f;
}

static cast_status_t diag_check(int n_frames, int Hg, int Wg, int D, const cast_diag_params_t* p) {
  if (p == nullptr) return fail(CAST_ERR_NULL, "diag: params is NULL");
  if (n_frames < 1 || Hg < 1 || Wg < 1 || D < 1) return fail(CAST_ERR_SHAPE, "diag: sizes must be >= 1");
  if (n_frames > kParMaxFrames) return fail(CAST_ERR_UNSUPPORTED, "diag: n_frames > %d", kParMaxFrames);
  if (p->tile_h < 1 || p->tile_h > kParMaxTile || p->tile_w < 1 || p->tile_w > kParMaxTile)
    return fail(CAST_ERR_UNSUPPORTED, "diag: tile edges must be in [1, %d]", kParMaxTile);
  if (p->n_bands < 1 || p->n_bands > kDiagMaxBands)
    return fail(CAST_ERR_SHAPE, "diag: n_bands must be in [1, %d]", kDiagMaxBands);
  if (p->band_edges[0] != 0.0f || p->band_edges[p->n_bands] != 1.0f)
    return fail(CAST_ERR_SHAPE, "diag: band edges must start at 0 and end at 1");
  for (int k = 0; k < p->n_bands; ++k)
    if (!(p->band_edges[k + 1] > p->band_edges[k])) return fail(CAST_ERR_SHAPE, "diag: band edges must increase");
  if (!(p->eps >= 0.0f)) return fail(CAST_ERR_SHAPE, "diag: eps must be >= 0");
  if ((long long)Hg * Wg * D >= (1LL << 30)) return fail(CAST_ERR_UNSUPPORTED, "diag: frame too large");
  return CAST_OK;
}

size_t cast_spectral_diagnostics_workspace_bytes(int n_frames, int Hg, int Wg, int D,
                                                 const cast_diag_params_t* params) {
  if (diag_check(n_frames, Hg, Wg, D, params) != CAST_OK) return 0;
  return diag_workspace_bytes(n_frames, Hg, Wg, D, params->tile_h, params->tile_w);
}

cast_status_t cast_spectral_diagnostics(const float* ref, const float* approx, const float* theta,
                                        const int* anchors, int n_anchor, int n_frames, int Hg,
                                        int Wg, int D, const cast_diag_params_t* params,
                                        float* nrmse_out, float* band_out, float* phase_err_out,
                                        float* r_phase_out, float* r_mag_out, void* workspace,
                                        size_t workspace_bytes, hipStream_t stream) {
  if (ref == nullptr || approx == nullptr || anchors == nullptr)
    return fail(CAST_ERR_NULL, "diag: ref, approx and anchors are required");
  cast_status_t st = diag_check(n_frames, Hg, Wg, D, params);
  if (st != CAST_OK) return st;
  if (n_anchor < 2 || n_anchor > n_frames || n_anchor > kParMaxAnchors)
    return fail(CAST_ERR_ANCHORS, "diag: need 2 <= n_anchor <= min(n_frames, %d)", kParMaxAnchors);
  for (int j = 0; j < n_anchor; ++j) {
    if (anchors[j] < 0 || anchors[j] >= n_frames)
      return fail(CAST_ERR_ANCHORS, "diag: anchor %d = %d outside [0, %d)", j, anchors[j], n_frames);
    if (j > 0 && anchors[j] <= anchors[j - 1])
      return fail(CAST_ERR_ANCHORS, "diag: anchors must be strictly increasing (index %d)", j);
  }
  const void* bufs[] = {ref, approx, theta, nrmse_out, band_out, phase_err_out, r_phase_out, r_mag_out};
  for (const void* b : bufs)
    if (!aligned(b, 4)) return fail(CAST_ERR_SHAPE, "diag: misaligned buffers");
  st = check_ws(workspace, workspace_bytes, diag_workspace_bytes(n_frames, Hg, Wg, D, params->tile_h, params->tile_w));
  if (st != CAST_OK) return st;
  return launch_diag(ref, approx, theta, anchors, n_anchor, n_frames, Hg, Wg, D, *params,
                     nrmse_out, band_out, phase_err_out, r_phase_out, r_mag_out, workspace, stream);
}

cast_status_t cast_phase_progress(const float* ref, const int* anchors, int n_anchor, int n_frames,
                                  int Hg, int Wg, int D, const cast_diag_params_t* params,
                                  float* p_out, hipStream_t stream) {
  if (ref == nullptr || anchors == nullptr || p_out == nullptr)
    return fail(CAST_ERR_NULL, "progress: ref, anchors and p_out are required");
  cast_status_t st = diag_check(n_frames, Hg, Wg, D, params);
  if (st != CAST_OK) return st;
  if (n_anchor < 2 || n_anchor > n_frames || n_anchor > kParMaxAnchors)
    return fail(CAST_ERR_ANCHORS, "progress: need 2 <= n_anchor <= min(n_frames, %d)", kParMaxAnchors);
  for (int j = 0; j < n_anchor; ++j) {
    if (anchors[j] < 0 || anchors[j] >= n_frames)
      return fail(CAST_ERR_ANCHORS, "progress: anchor %d = %d outside [0, %d)", j, anchors[j], n_frames);
    if (j > 0 && anchors[j] <= anchors[j - 1])
      return fail(CAST_ERR_ANCHORS, "progress: anchors must be strictly increasing (index %d)", j);
  }
  if (!aligned(ref, 4) || !aligned(p_out, 4)) return fail(CAST_ERR_SHAPE, "progress: misaligned buffers");
  return launch_phase_progress(ref, anchors, n_anchor, Hg, Wg, D, params->tile_h, params->tile_w,
                               p_out, stream);
}

}  // extern "C"
