// Control-aware frame selection on gfx950 (Sec. 3.1 eq:sensitivity; Sec. 4.2
// eq:debt, eq:score; App. A.1 eq:normalization and the scheduling rules).
//
// frame_sq      HBM scan: every (control branch, frame) is cut into spans of
//               kSpan elements; a 256-thread block sums the squares of one span
//               in fp32 (four 16-byte loads in flight per thread when the frames
//               allow them) and writes one partial, so the sums are bit-identical
//               across runs.
// frame_select  one block: per present branch r_i = sqrt(sum / (S D)) (partials
//               added in fp64 by one wave per frame, fixed order), min / max over
//               the chunk, the normalised responses and their mean d_i; ages after
//               the block's anchors, coverage debt h_i / ceil(N / K_f), score
//               d_i + lambda D_i (lambda D_i without a fresh response); the K_f
//               best frames by rank counting under (score descending, frame
//               ascending), written in ascending frame order.  Every float operation after r is one
//               correctly rounded fp32 operation (no contraction), so the
//               decision is reproducible on the host in fp32.
#include "cast_common.h"

namespace cast {

namespace {

constexpr int kSqThreads = 256;
constexpr int kSpan = 32768;          // elements per partial (128 per thread)
constexpr int kUnroll = 4;            // independent 16-byte loads in flight per thread
constexpr int kSelThreads = 1024;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

struct SqArgs {
  const void* src[2];     // present branches only, in order
  long long frame_elems;  // S * D
  int n_split;
};

template <int DT, bool VEC>
__global__ __launch_bounds__(kSqThreads) void frame_sq_kernel(SqArgs a, float* __restrict__ partial) {
  const int split = blockIdx.x, f = blockIdx.y, z = blockIdx.z;
  const long long e0 = (long long)split * kSpan;
  const long long e1 = min(e0 + kSpan, a.frame_elems);
  float acc = 0.0f;
  if constexpr (DT == 0) {
    const float* x = static_cast<const float*>(a.src[z]) + (long long)f * a.frame_elems;
    if constexpr (VEC) {
      const f32x4* x4 = reinterpret_cast<const f32x4*>(x);
      const long long q1 = e1 / 4;
      float pa[kUnroll] = {};
      for (long long e = e0 / 4 + threadIdx.x; e < q1; e += kUnroll * kSqThreads) {
        f32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const long long eu = e + u * kSqThreads;
          v[u] = eu < q1 ? __builtin_nontemporal_load(x4 + eu) : f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          pa[u] = fmaf(v[u].x, v[u].x, pa[u]);
          pa[u] = fmaf(v[u].y, v[u].y, pa[u]);
          pa[u] = fmaf(v[u].z, v[u].z, pa[u]);
          pa[u] = fmaf(v[u].w, v[u].w, pa[u]);
        }
      }
      acc = (pa[0] + pa[1]) + (pa[2] + pa[3]);
    } else {
      for (long long e = e0 + threadIdx.x; e < e1; e += kSqThreads) acc = fmaf(x[e], x[e], acc);
    }
  } else {
    const uint16_t* x = static_cast<const uint16_t*>(a.src[z]) + (long long)f * a.frame_elems;
    if constexpr (VEC) {
      const u32x4* x8 = reinterpret_cast<const u32x4*>(x);
      const long long q1 = e1 / 8;
      float pa[kUnroll] = {};
      for (long long e = e0 / 8 + threadIdx.x; e < q1; e += kUnroll * kSqThreads) {
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const long long eu = e + u * kSqThreads;
          v[u] = eu < q1 ? __builtin_nontemporal_load(x8 + eu) : u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const float lo = bf16lo(w[k]), hi = bf16hi(w[k]);
            pa[u] = fmaf(lo, lo, pa[u]);
            pa[u] = fmaf(hi, hi, pa[u]);
          }
        }
      }
      acc = (pa[0] + pa[1]) + (pa[2] + pa[3]);
    } else {
      for (long long e = e0 + threadIdx.x; e < e1; e += kSqThreads) {
        const float v = __uint_as_float((uint32_t)x[e] << 16);
        acc = fmaf(v, v, acc);
      }
    }
  }
  // fixed-order block sum: butterfly in each wave, then the 4 wave sums in order
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
  __shared__ float ws[kSqThreads / 64];
  if ((threadIdx.x & 63) == 0) ws[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0)
    partial[((long long)z * gridDim.y + f) * a.n_split + split] = (ws[0] + ws[1]) + (ws[2] + ws[3]);
}

struct SelArgs {
  const float* partial;   // [n_present, n_cur, n_split]
  int32_t* ages;
  float* r_out;           // [2, n_cur] rows by branch (cam, act), or null
  float* score_out;
  int32_t* anchors_out;
  double inv_elems;       // 1 / (S D)
  int n_split, n_cur, k_f, n_present;
  int row_of[2];          // r_out row of present branch z
  float lambda_cov, eps;
  uint32_t prev_mask[kSelectMaxFrames / 32];   // anchors the block ran with
};

__global__ __launch_bounds__(kSelThreads) void frame_select_kernel(SelArgs a) {
  __shared__ float r[2][kSelectMaxFrames];
  __shared__ float sc[kSelectMaxFrames];
  __shared__ unsigned char sel[kSelectMaxFrames];
  __shared__ float red[2][kSelThreads / 64];
  __shared__ float lohi[2][2];
  const int tid = threadIdx.x, n = a.n_cur;

  // r per present branch: one wave per (branch, frame) adds its partials in fp64,
  // lane l taking partials l, l + 64, ..., then a fixed butterfly
  const int wave = tid >> 6, lane = tid & 63;
  for (int item = wave; item < a.n_present * n; item += kSelThreads / 64) {
    const int z = item / n, i = item - z * n;
    const float* p = a.partial + (long long)item * a.n_split;
    double sum = 0.0;
    for (int k = lane; k < a.n_split; k += 64) sum += (double)p[k];
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) {
      const float ri = (float)sqrt(sum * a.inv_elems);
      r[z][i] = ri;
      if (a.r_out) a.r_out[(long long)a.row_of[z] * n + i] = ri;
    }
  }
  __syncthreads();
  // min and max over the chunk, per branch (exact in any order)
  for (int z = 0; z < a.n_present; ++z) {
    float lo = INFINITY, hi = -INFINITY;
    for (int i = tid; i < n; i += kSelThreads) {
      lo = fminf(lo, r[z][i]);
      hi = fmaxf(hi, r[z][i]);
    }
    for (int o = 32; o > 0; o >>= 1) {
      lo = fminf(lo, __shfl_xor(lo, o));
      hi = fmaxf(hi, __shfl_xor(hi, o));
    }
    if ((tid & 63) == 0) { red[0][tid >> 6] = lo; red[1][tid >> 6] = hi; }
    __syncthreads();
    if (tid == 0) {
      lo = red[0][0];
      hi = red[1][0];
      for (int w = 1; w < kSelThreads / 64; ++w) {
        lo = fminf(lo, red[0][w]);
        hi = fmaxf(hi, red[1][w]);
      }
      lohi[z][0] = lo;
      lohi[z][1] = hi;
    }
    __syncthreads();
  }
  // sensitivity, ages, debt and score per frame
  const int h_cov = (n + a.k_f - 1) / a.k_f;
  for (int i = tid; i < n; i += kSelThreads) {
    float d = 0.0f;
    for (int z = 0; z < a.n_present; ++z) {
      const float lo = lohi[z][0], hi = lohi[z][1];
      const float nz = __fdiv_rn(__fsub_rn(r[z][i], lo), __fadd_rn(__fsub_rn(hi, lo), a.eps));
      d = __fadd_rn(d, nz);
    }
    if (a.n_present == 2) d = __fmul_rn(d, 0.5f);
    const bool was_anchor = (a.prev_mask[i >> 5] >> (i & 31)) & 1u;
    const int h = was_anchor ? 0 : a.ages[i] + 1;
    a.ages[i] = h;
    const float debt = __fdiv_rn((float)h, (float)h_cov);
    const float ld = __fmul_rn(a.lambda_cov, debt);
    const float s = a.n_present > 0 ? __fadd_rn(d, ld) : ld;
    sc[i] = s;
    if (a.score_out) a.score_out[i] = s;
  }
  __syncthreads();
  // TopK under (score descending, frame ascending) by rank counting
  for (int i = tid; i < n; i += kSelThreads) {
    const float si = sc[i];
    int rank = 0;
    for (int j = 0; j < n; ++j) {
      const float sj = sc[j];
      rank += (sj > si) || (sj == si && j < i);
    }
    sel[i] = rank < a.k_f;
  }
  __syncthreads();
  for (int i = tid; i < n; i += kSelThreads) {
    if (!sel[i]) continue;
    int pos = 0;
    for (int j = 0; j < i; ++j) pos += sel[j];
    if (pos < a.k_f) a.anchors_out[pos] = i;   // (NaN scores could select more)
  }
}

}  // namespace

int select_splits(int S, int D) {
  const long long e = (long long)S * D;
  return (int)((e + kSpan - 1) / kSpan);
}

cast_status_t launch_frame_select(const void* cam, const void* act, int dtype, int n_cur, int S,
                                  int D, const int* anchors_prev, int n_prev, int k_f,
                                  const cast_select_params_t& p, int32_t* ages, float* r_out,
                                  float* score_out, int32_t* anchors_out, float* partial,
                                  hipStream_t stream) {
  SqArgs q{};
  int n_present = 0;
  int row_of[2] = {0, 0};
  if (cam) { row_of[n_present] = 0; q.src[n_present++] = cam; }
  if (act) { row_of[n_present] = 1; q.src[n_present++] = act; }
  q.frame_elems = (long long)S * D;
  q.n_split = select_splits(S, D);
  if (n_present > 0) {
    const int esz = dtype == 0 ? 4 : 2;
    bool vec = q.frame_elems % (16 / esz) == 0;
    for (int z = 0; z < n_present; ++z) vec = vec && ((uintptr_t)q.src[z] % 16 == 0);
    dim3 grid(q.n_split, n_cur, n_present);
    if (dtype == 0) {
      if (vec) hipLaunchKernelGGL((frame_sq_kernel<0, true>), grid, dim3(kSqThreads), 0, stream, q, partial);
      else hipLaunchKernelGGL((frame_sq_kernel<0, false>), grid, dim3(kSqThreads), 0, stream, q, partial);
    } else {
      if (vec) hipLaunchKernelGGL((frame_sq_kernel<1, true>), grid, dim3(kSqThreads), 0, stream, q, partial);
      else hipLaunchKernelGGL((frame_sq_kernel<1, false>), grid, dim3(kSqThreads), 0, stream, q, partial);
    }
    cast_status_t st = check_launch("frame_sq");
    if (st != CAST_OK) return st;
  }
  SelArgs s{};
  s.partial = partial;
  s.ages = ages;
  s.r_out = r_out;
  s.score_out = score_out;
  s.anchors_out = anchors_out;
  s.inv_elems = 1.0 / (double)q.frame_elems;
  s.n_split = q.n_split;
  s.n_cur = n_cur;
  s.k_f = k_f;
  s.n_present = n_present;
  s.row_of[0] = row_of[0];
  s.row_of[1] = row_of[1];
  s.lambda_cov = p.lambda_cov;
  s.eps = p.eps;
  for (int j = 0; j < n_prev; ++j) s.prev_mask[anchors_prev[j] >> 5] |= 1u << (anchors_prev[j] & 31);
  hipLaunchKernelGGL(frame_select_kernel, dim3(1), dim3(kSelThreads), 0, stream, s);
  return check_launch("frame_select");
}

}  // namespace cast
