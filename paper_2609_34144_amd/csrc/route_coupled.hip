// Reconstruction-coupled historical routing on gfx950 (Sec. 4.4 eq:pooled,
// eq:omission, eq:abc, eq:risk, eq:objective, eq:topk; App. B eq:abcclosed,
// eq:boundarycoeff, eq:gain, eq:boundarygain, Algorithm 1).
//
// route_means (route_kv.hip)   token means of Q and K, then of V
// coupled_omission  grid (anchor x head, range of 16 blocks): scores over the M
//                   blocks, softmax, o_bar, then for each block of the range
//                   u = (pi/(1-pi+eps))^2 d^T G_h d with d = o_bar - v_bar[m]
//                   (G_h = P_h^T P_h, so ||P_h d||^2 costs dh^2, not D dh)
// coupled_refine    one workgroup per head (heads never interact): masks start as
//                   TopK(u), then Algorithm 1's directional passes; every TopK is a
//                   bitonic sort of 64-bit keys (ordered value bits, inverted block
//                   index) in LDS; the head's objective J is kept up to date by the
//                   accepted gain differences
// wo_gram           G_h from the bf16 output projection (weights only, once per model)
// All reductions run in a fixed order and nothing is atomic: results are
// bit-identical across runs.
#include "cast_common.h"

namespace cast {

namespace {

constexpr int kOmM = 16;          // blocks per omission workgroup (4 per wave)
constexpr int kThreads = 256;
constexpr int kRefineThreads = 64;   // the solver runs in one wave per head
constexpr int kRefineCacheU = 8192;  // u of one head (n_a * M floats) staged in LDS up to this

struct CoupledArgs {
  const float* means_qk;   // [n_a + M, D]: q_bar rows, then k_bar rows
  const float* means_v;    // [M, D]
  const float* gram;       // [H, dh, dh]
  float* u;                // [n_a, H, M] (workspace)
  float* u_out;            // optional copy of u
  int32_t* idx_out;        // [n_a, H, k_eff]
  int n_a, H, M, D, k_eff, n_frames, passes;
  float scale, l_anc, l_rec, tol, eps;
  short anchors[kCoupledMaxAnchors];
};

// Sum of one value per thread of the workgroup, in a fixed order; every thread
// gets the result.  `red` holds kThreads floats; the call contains barriers.
__device__ float block_sum(float v, float* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  const float r = red[0];
  __syncthreads();
  return r;
}

// Sum over the 64 lanes of a wave by a fixed butterfly: every lane gets the same
// (order-independent of the schedule) result.
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ float block_max(float v, float* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + s]);
    __syncthreads();
  }
  const float r = red[0];
  __syncthreads();
  return r;
}

// ---------------------------------------------------------------------------
// omission proxy u (eq:pooled, eq:omission)
// ---------------------------------------------------------------------------
template <int DH>
__global__ __launch_bounds__(kThreads) void coupled_omission_kernel(CoupledArgs a) {
  extern __shared__ float sm[];
  float* e = sm;               // [M] scores, then unnormalised probabilities
  float* qs = e + a.M;         // [DH]
  float* ob = qs + DH;         // [DH]
  float* red = ob + DH;        // [kThreads]
  float* dv = red + kThreads;  // [kOmM][DH] difference vectors, kOmM / 4 per wave
  const int ih = blockIdx.x, i = ih / a.H, h = ih - (ih / a.H) * a.H;
  const int m0 = blockIdx.y * kOmM;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  for (int d = tid; d < DH; d += kThreads) qs[d] = a.means_qk[(long long)i * a.D + h * DH + d];
  __syncthreads();
  // scores: one wave per block, lanes over the channels
  float lmax = -INFINITY;
  for (int m = wave; m < a.M; m += kThreads / 64) {
    const float* kb = a.means_qk + (long long)(a.n_a + m) * a.D + h * DH;
    float s = 0.0f;
    for (int d = lane; d < DH; d += 64) s = fmaf(qs[d], kb[d], s);
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
    s *= a.scale;
    if (lane == 0) e[m] = s;
    lmax = fmaxf(lmax, s);
  }
  __syncthreads();
  const float smax = block_max(lmax, red);
  float lsum = 0.0f;
  for (int m = tid; m < a.M; m += kThreads) {
    const float x = expf(e[m] - smax);
    e[m] = x;
    lsum += x;
  }
  const float ssum = block_sum(lsum, red);
  // o_bar = sum_m pi_m v_bar_m: thread -> (channel, part of the blocks), parts
  // combined in a fixed order
  {
    constexpr int NP = kThreads / DH;
    const int d = tid % DH, part = tid / DH;
    float acc = 0.0f;
    for (int m = part; m < a.M; m += NP)
      acc = fmaf(e[m], a.means_v[(long long)m * a.D + h * DH + d], acc);
    red[tid] = acc;
    __syncthreads();
    if (tid < DH) {
      float o = 0.0f;
      for (int p = 0; p < NP; ++p) o += red[p * DH + tid];
      ob[tid] = o / ssum;
    }
    __syncthreads();
  }
  // u for the blocks of this range: wave w takes the 4 blocks m0 + 4w .. +3 at
  // once, so every G element loaded serves 4 difference vectors
  constexpr int MW = kOmM / 4;
  const float* G = a.gram + (long long)h * DH * DH;   // symmetric: row l of column c = G[c][l]
  float* dw = dv + wave * MW * DH;                    // [MW][DH]
  const int mw0 = m0 + MW * wave;
#pragma unroll
  for (int j = 0; j < MW; ++j) {
    const int m = min(mw0 + j, a.M - 1);
    for (int c = lane; c < DH; c += 64) dw[j * DH + c] = ob[c] - a.means_v[(long long)m * a.D + h * DH + c];
  }
  __syncthreads();
  float y1[MW], y2[MW];
#pragma unroll
  for (int j = 0; j < MW; ++j) { y1[j] = 0.0f; y2[j] = 0.0f; }
  const int l1 = lane < DH ? lane : 0;
#pragma unroll 4
  for (int c = 0; c < DH; ++c) {
    const float g1 = G[c * DH + l1];
    const float g2 = DH > 64 ? G[c * DH + lane + 64] : 0.0f;
#pragma unroll
    for (int j = 0; j < MW; ++j) {
      const float dc = dw[j * DH + c];
      y1[j] = fmaf(g1, dc, y1[j]);
      if (DH > 64) y2[j] = fmaf(g2, dc, y2[j]);
    }
  }
#pragma unroll
  for (int j = 0; j < MW; ++j) {
    const int m = mw0 + j;
    float part = lane < DH ? dw[j * DH + lane] * y1[j] : 0.0f;
    if (DH > 64) part += dw[j * DH + lane + 64] * y2[j];
    for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o);
    if (m < a.M && lane == 0) {
      const float pi = e[m] / ssum;
      const float cf = pi / (1.0f - pi + a.eps);
      const float u = cf * cf * part;
      const long long o = ((long long)i * a.H + h) * a.M + m;
      a.u[o] = u;
      if (a.u_out) a.u_out[o] = u;
    }
  }
}

// ---------------------------------------------------------------------------
// Algorithm 1 (eq:gain, eq:boundarygain, eq:topk)
// ---------------------------------------------------------------------------
// In-LDS bitonic sort of P (power of two) 64-bit keys into descending order by
// the nthr threads of the workgroup.
__device__ void bitonic_desc(unsigned long long* key, int P, int nthr) {
  for (int kk = 2; kk <= P; kk <<= 1) {
    for (int j = kk >> 1; j > 0; j >>= 1) {
      for (int x = threadIdx.x; x < P; x += nthr) {
        const int y = x ^ j;
        if (y > x) {
          const unsigned long long p = key[x], q = key[y];
          const bool desc = (x & kk) == 0;
          if (desc ? (p < q) : (p > q)) { key[x] = q; key[y] = p; }
        }
      }
      __syncthreads();
    }
  }
}

// 64-bit key of value v of block m: larger v first, then lower m.
__device__ __forceinline__ unsigned long long order_key(float v, int m) {
  uint32_t b = __float_as_uint(v);
  if ((b << 1) == 0u) b = 0u;   // -0 and +0 compare equal
  const uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((unsigned long long)ord << 32) | (uint32_t)(~(uint32_t)m);
}

struct Coeffs {
  // interval (rows j, j+1): A = B, C from the closed form of eq:abcclosed
  // boundary sides (eq:boundarycoeff): rows (ra, rb) and sums over their frames
  int has_l, has_r;
  float al, bl, cl, ar, br, cr;
};

// One wave per head: the solver is a chain of small sorts and sums, and with a
// single wave every barrier is immediate and every sum a shuffle butterfly.
template <bool CACHE_U>
__global__ __launch_bounds__(kRefineThreads) void coupled_refine_kernel(CoupledArgs a) {
  extern __shared__ unsigned long long keys[];        // [P]
  const int M = a.M, n_a = a.n_a, k = a.k_eff, h = blockIdx.x;
  int P = 2;
  while (P < M) P <<= 1;
  float* g = reinterpret_cast<float*>(keys + P);      // [M] gains of the visited row
  uint32_t* xm = reinterpret_cast<uint32_t*>(g + M);  // [n_a * M] retain bits
  const int nwords = (n_a * M + 31) / 32;
  float* su = reinterpret_cast<float*>(xm + nwords);  // [n_a * M] u of this head (CACHE_U)
  __shared__ Coeffs cf;
  __shared__ float pair_ab[kCoupledMaxAnchors], pair_c[kCoupledMaxAnchors];
  const int tid = threadIdx.x;
  // u is read at every step of the solver: staged in LDS when it fits
  if constexpr (CACHE_U)
    for (int x = tid; x < n_a * M; x += kRefineThreads) {
      const int i = x / M, m = x - (x / M) * M;
      su[x] = a.u[((long long)i * a.H + h) * M + m];
    }
  auto U = [&](int i, int m) -> float {
    if constexpr (CACHE_U) return su[i * M + m];
    else return a.u[((long long)i * a.H + h) * M + m];
  };
  auto X = [&](int i, int m) -> float {
    const int bit = i * M + m;
    return (xm[bit >> 5] >> (bit & 31)) & 1u ? 1.0f : 0.0f;
  };

  // ---- coefficients
  for (int j = tid; j + 1 < n_a; j += kRefineThreads) {
    const float n = (float)(a.anchors[j + 1] - a.anchors[j]);
    pair_ab[j] = (n - 1.0f) * (2.0f * n - 1.0f) / (6.0f * n);
    pair_c[j] = (n * n - 1.0f) / (6.0f * n);
  }
  if (tid == 0) {
    Coeffs c{};
    if (n_a >= 2) {
      const int a0 = a.anchors[0], a1 = a.anchors[1];
      const int b0 = a.anchors[n_a - 2], b1 = a.anchors[n_a - 1];
      for (int t = 0; t < a0; ++t) {
        const float al = (float)(t - a0) / (float)(a1 - a0);
        c.al += (1.0f - al) * (1.0f - al);
        c.bl += al * al;
        c.cl += fabsf(al * (1.0f - al));
      }
      for (int t = b1 + 1; t < a.n_frames; ++t) {
        const float al = (float)(t - b0) / (float)(b1 - b0);
        c.ar += (1.0f - al) * (1.0f - al);
        c.br += al * al;
        c.cr += fabsf(al * (1.0f - al));
      }
      c.has_l = a0 > 0;
      c.has_r = b1 < a.n_frames - 1;
    }
    cf = c;
  }
  for (int w = tid; w < nwords; w += kRefineThreads) xm[w] = 0u;
  __syncthreads();

  // TopK of the values in g[0..M): leaves the winners first in keys[], returns
  // their sum (the same on every thread)
  auto topk_sum = [&]() -> float {
    if (M <= kRefineThreads) {
      // one value per lane: its rank is the number of larger keys (the keys are
      // distinct, so the ranks are too); the winners are stored in rank order
      const bool in = tid < M;
      const float gv = in ? g[tid] : 0.0f;
      const unsigned long long km = in ? order_key(gv, tid) : 0ull;
      int rank = 0;
      for (int j = 0; j < M; ++j) rank += __shfl(km, j) > km ? 1 : 0;
      const bool win = in && rank < k;
      if (win) keys[rank] = km;
      return wave_sum(win ? gv : 0.0f);
    }
    for (int m = tid; m < P; m += kRefineThreads) keys[m] = m < M ? order_key(g[m], m) : 0ull;
    __syncthreads();
    bitonic_desc(keys, P, kRefineThreads);
    float s = 0.0f;
    for (int x = tid; x < k; x += kRefineThreads) s += g[~(uint32_t)(keys[x] & 0xffffffffull)];
    return wave_sum(s);
  };
  // row i's mask := the k winners left in keys[]
  auto apply_topk = [&](int i) {
    const int b0 = i * M, b1 = b0 + M;
    for (int w = (b0 >> 5) + tid; w <= ((b1 - 1) >> 5); w += kRefineThreads) {   // one owner per word
      uint32_t word = xm[w];
      for (int bb = 0; bb < 32; ++bb) {
        const int bit = (w << 5) + bb;
        if (bit >= b0 && bit < b1) word &= ~(1u << bb);
      }
      xm[w] = word;
    }
    __syncthreads();
    if (tid == 0) {
      for (int x = 0; x < k; ++x) {
        const int bit = b0 + (int)~(uint32_t)(keys[x] & 0xffffffffull);
        xm[bit >> 5] |= 1u << (bit & 31);
      }
    }
    __syncthreads();
  };

  // ---- initial masks: TopK(u) per anchor
  for (int i = 0; i < n_a; ++i) {
    for (int m = tid; m < M; m += kRefineThreads) g[m] = U(i, m);
    __syncthreads();
    topk_sum();
    apply_topk(i);
  }

  // ---- objective J of the head (eq:objective with eq:risk and eq:boundaryrisk)
  auto risk = [&](int ra, int rb, float A, float B, float C, int m) -> float {
    const float ua = U(ra, m), ub = U(rb, m), oa = 1.0f - X(ra, m), ob = 1.0f - X(rb, m);
    return A * oa * ua + B * ob * ub + 2.0f * C * oa * ob * sqrtf(ua) * sqrtf(ub);
  };
  float jpart = 0.0f;
  for (int m = tid; m < M; m += kRefineThreads) {
    float anc = 0.0f, rec = 0.0f;
    for (int i = 0; i < n_a; ++i) anc += (1.0f - X(i, m)) * U(i, m);
    for (int j = 0; j + 1 < n_a; ++j) rec += risk(j, j + 1, pair_ab[j], pair_ab[j], pair_c[j], m);
    if (cf.has_l) rec += risk(0, 1, cf.al, cf.bl, cf.cl, m);
    if (cf.has_r) rec += risk(n_a - 2, n_a - 1, cf.ar, cf.br, cf.cr, m);
    jpart += a.l_anc * anc + a.l_rec * rec;
  }
  float J = wave_sum(jpart);

  // ---- directional passes
  for (int s = 0; s < a.passes && k < M; ++s) {
    bool changed = false;
    for (int v = 0; v < n_a; ++v) {
      const int i = (s % 2 == 0) ? v : n_a - 1 - v;
      float oldpart = 0.0f;
      for (int m = tid; m < M; m += kRefineThreads) {
        const float ui = U(i, m), si = sqrtf(ui);
        float G = a.l_anc * ui, rec = 0.0f;
        if (i > 0)
          rec += pair_ab[i - 1] * ui + 2.0f * pair_c[i - 1] * (1.0f - X(i - 1, m)) * sqrtf(U(i - 1, m)) * si;
        if (i + 1 < n_a)
          rec += pair_ab[i] * ui + 2.0f * pair_c[i] * (1.0f - X(i + 1, m)) * si * sqrtf(U(i + 1, m));
        if (cf.has_l) {
          if (i == 0) rec += cf.al * ui + 2.0f * cf.cl * (1.0f - X(1, m)) * si * sqrtf(U(1, m));
          if (i == 1) rec += cf.bl * ui + 2.0f * cf.cl * (1.0f - X(0, m)) * si * sqrtf(U(0, m));
        }
        if (cf.has_r) {
          if (i == n_a - 2) rec += cf.ar * ui + 2.0f * cf.cr * (1.0f - X(n_a - 1, m)) * si * sqrtf(U(n_a - 1, m));
          if (i == n_a - 1) rec += cf.br * ui + 2.0f * cf.cr * (1.0f - X(n_a - 2, m)) * si * sqrtf(U(n_a - 2, m));
        }
        G += a.l_rec * rec;
        g[m] = G;
        oldpart += X(i, m) * G;
      }
      const float g_old = wave_sum(oldpart);
      const float g_new = topk_sum();
      const float gain = g_new - g_old;
      if (gain > a.tol * fmaxf(J, 1e-8f)) {   // uniform: every thread holds the same sums
        apply_topk(i);
        J -= gain;
        changed = true;
      }
    }
    if (!changed) break;
  }

  // ---- ascending block indices of every mask
  if (tid == 0) {
    for (int i = 0; i < n_a; ++i) {
      int32_t* dst = a.idx_out + ((long long)i * a.H + h) * k;
      int r = 0;
      for (int m = 0; m < M && r < k; ++m)
        if (X(i, m) != 0.0f) dst[r++] = m;
    }
  }
}

// ---------------------------------------------------------------------------
// Gram matrices of the head slices of W_O
// ---------------------------------------------------------------------------
template <int DH>
__global__ __launch_bounds__(kThreads) void wo_gram_kernel(const uint16_t* __restrict__ w, int D,
                                                           float* __restrict__ gram) {
  constexpr int RB = 16;                 // G rows per workgroup
  constexpr int NB = DH * RB / kThreads; // outputs per thread
  constexpr int CH = 64;                 // W rows staged per step
  __shared__ float tile[CH][DH];
  const int h = blockIdx.x, rb = blockIdx.y, tid = threadIdx.x;
  const int ra = rb * RB + tid / (kThreads / RB);         // this thread's G row
  const int c0 = tid % (kThreads / RB);                   // first column, stride kThreads / RB
  float acc[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) acc[j] = 0.0f;
  for (int r0 = 0; r0 < D; r0 += CH) {
    for (int x = tid; x < CH * DH; x += kThreads) {
      const int rr = x / DH, cc = x - (x / DH) * DH;
      const int r = r0 + rr;
      tile[rr][cc] = r < D ? __uint_as_float((uint32_t)w[(long long)r * D + h * DH + cc] << 16) : 0.0f;
    }
    __syncthreads();
    for (int rr = 0; rr < CH; ++rr) {
      const float av = tile[rr][ra];
#pragma unroll
      for (int j = 0; j < NB; ++j) acc[j] = fmaf(av, tile[rr][c0 + j * (kThreads / RB)], acc[j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < NB; ++j)
    gram[((long long)h * DH + ra) * DH + c0 + j * (kThreads / RB)] = acc[j];
}

}  // namespace

CoupledPlan plan_coupled(int n_a, int S, int H, int dh, int M, int Bv) {
  CoupledPlan p{};
  p.qk = plan_route(n_a, S, H, dh, M, Bv);
  p.v = plan_route(0, S, H, dh, M, Bv);
  const size_t D = (size_t)H * dh;
  p.off_means_qk = 0;
  p.off_means_v = p.off_means_qk + align_up((size_t)(n_a + M) * D * sizeof(float));
  p.off_u = p.off_means_v + align_up((size_t)M * D * sizeof(float));
  p.total = p.off_u + align_up((size_t)n_a * H * M * sizeof(float));
  return p;
}

cast_status_t launch_coupled(const void* q, const void* k, const void* v, const float* gram,
                             const int* anchors, int n_a, int n_frames, int S, int H, int dh,
                             int M, int Bv, int k_eff, float scale, const cast_coupled_params_t& prm,
                             float* u_out, int32_t* idx_out, const CoupledPlan& p, void* ws,
                             hipStream_t stream) {
  char* base = static_cast<char*>(ws);
  CoupledArgs a{};
  a.means_qk = reinterpret_cast<float*>(base + p.off_means_qk);
  a.means_v = reinterpret_cast<float*>(base + p.off_means_v);
  a.gram = gram;
  a.u = reinterpret_cast<float*>(base + p.off_u);
  a.u_out = u_out;
  a.idx_out = idx_out;
  a.n_a = n_a;
  a.H = H;
  a.M = M;
  a.D = H * dh;
  a.k_eff = k_eff;
  a.n_frames = n_frames;
  a.passes = prm.passes;
  a.scale = scale;
  a.l_anc = prm.l_anc;
  a.l_rec = prm.l_rec;
  a.tol = prm.tol;
  a.eps = prm.eps;
  for (int j = 0; j < n_a; ++j) a.anchors[j] = (short)anchors[j];
  cast_status_t st = launch_pool_means(q, k, n_a, S, M, Bv, p.qk,
                                       const_cast<float*>(a.means_qk), stream);
  if (st != CAST_OK) return st;
  st = launch_pool_means(v, v, 0, S, M, Bv, p.v, const_cast<float*>(a.means_v), stream);
  if (st != CAST_OK) return st;
  const dim3 grid(n_a * H, (M + kOmM - 1) / kOmM);
  const size_t shm = (size_t)(M + 2 * dh + kThreads + kOmM * dh) * sizeof(float);
  switch (dh) {
    case 32: hipLaunchKernelGGL(coupled_omission_kernel<32>, grid, dim3(kThreads), shm, stream, a); break;
    case 64: hipLaunchKernelGGL(coupled_omission_kernel<64>, grid, dim3(kThreads), shm, stream, a); break;
    default: hipLaunchKernelGGL(coupled_omission_kernel<128>, grid, dim3(kThreads), shm, stream, a); break;
  }
  st = check_launch("coupled_omission");
  if (st != CAST_OK) return st;
  int P = 2;
  while (P < M) P <<= 1;
  const size_t shm2 = (size_t)P * 8 + (size_t)M * 4 + (size_t)((n_a * M + 31) / 32) * 4;
  if (n_a * M <= kRefineCacheU)
    hipLaunchKernelGGL(coupled_refine_kernel<true>, dim3(H), dim3(kRefineThreads),
                       shm2 + (size_t)n_a * M * 4, stream, a);
  else
    hipLaunchKernelGGL(coupled_refine_kernel<false>, dim3(H), dim3(kRefineThreads), shm2, stream, a);
  return check_launch("coupled_refine");
}

cast_status_t launch_wo_gram(const void* w_o, int D, int H, int dh, float* gram, hipStream_t stream) {
  const uint16_t* w = static_cast<const uint16_t*>(w_o);
  const dim3 grid(H, dh / 16);
  switch (dh) {
    case 32: hipLaunchKernelGGL(wo_gram_kernel<32>, grid, dim3(kThreads), 0, stream, w, D, gram); break;
    case 64: hipLaunchKernelGGL(wo_gram_kernel<64>, grid, dim3(kThreads), 0, stream, w, D, gram); break;
    default: hipLaunchKernelGGL(wo_gram_kernel<128>, grid, dim3(kThreads), 0, stream, w, D, gram); break;
  }
  return check_launch("wo_gram");
}

}  // namespace cast
