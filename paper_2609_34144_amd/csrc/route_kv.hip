// Pooled chunk scores and TopK routing on gfx950 (Sec. 4.4 eq:pooled, eq:topk).
//
// route_pool      HBM scan: every anchor frame of Q and every history chunk of K is
//                 cut into token splits; a 64-lane block sums one split for 512
//                 channels (8 bf16 per lane, 16-byte coalesced loads) in fp32.
// route_finalize  fixed-order sum of the splits -> pooled means q_bar, k_bar (fp32).
// route_topk      one block per (anchor, head): scores s = scale * q_bar . k_bar for
//                 all M chunks, a bitonic sort of 64-bit keys (score order, then
//                 lower chunk index) in LDS, and a second sort that emits the k_eff
//                 winners in ascending chunk order.
// No atomics anywhere: results are bit-identical across runs.
#include "cast_common.h"

namespace cast {

namespace {

__global__ __launch_bounds__(kPoolThreads) void route_pool_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, int n_a, int S, int Bv,
    int D, int spq, int tq, int spk, int tk, float* __restrict__ partial) {
  const int item = blockIdx.x, grp = blockIdx.y;
  const int c = (grp * kPoolThreads + threadIdx.x) * 8;
  const int nq = n_a * spq;
  const uint16_t* base;
  int t0, t1;
  if (item < nq) {
    const int seg = item / spq, sp = item - (item / spq) * spq;
    base = q + (long long)seg * S * D;
    t0 = sp * tq;
    t1 = min(S, t0 + tq);
  } else {
    const int it = item - nq;
    const int seg = it / spk, sp = it - (it / spk) * spk;
    base = k + (long long)seg * Bv * D;
    t0 = sp * tk;
    t1 = min(Bv, t0 + tk);
  }
  if (c >= D) return;
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4* p = reinterpret_cast<const u32x4*>(base + (long long)t0 * D + c);
  const long long stride = D / 8;
  const int n = t1 - t0;
  auto add = [&](const u32x4& v) {
    acc[0] += bf16lo(v.x); acc[1] += bf16hi(v.x);
    acc[2] += bf16lo(v.y); acc[3] += bf16hi(v.y);
    acc[4] += bf16lo(v.z); acc[5] += bf16hi(v.z);
    acc[6] += bf16lo(v.w); acc[7] += bf16hi(v.w);
  };
  int t = 0;
  for (; t + 8 <= n; t += 8) {
    u32x4 v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p + u * stride);
#pragma unroll
    for (int u = 0; u < 8; ++u) add(v[u]);
    p += 8 * stride;
  }
  for (; t < n; ++t) {
    add(__builtin_nontemporal_load(p));
    p += stride;
  }
  float4* o = reinterpret_cast<float4*>(partial + (long long)item * D + c);
  o[0] = make_float4(acc[0], acc[1], acc[2], acc[3]);
  o[1] = make_float4(acc[4], acc[5], acc[6], acc[7]);
}

__global__ __launch_bounds__(256) void route_finalize_kernel(const float* __restrict__ partial,
                                                             int n_a, int D, int spq, int spk,
                                                             int S, int Bv, float* __restrict__ means) {
  const int seg = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= D) return;
  int nsp, first;
  float len;
  if (seg < n_a) { nsp = spq; first = seg * spq; len = (float)S; }
  else { nsp = spk; first = n_a * spq + (seg - n_a) * spk; len = (float)Bv; }
  float s = 0.0f;
#pragma unroll 8
  for (int j = 0; j < nsp; ++j) s += partial[(long long)(first + j) * D + c];
  means[(long long)seg * D + c] = s / len;
}

// In-LDS bitonic sort of P (power of two) 64-bit keys into descending order.
__device__ void bitonic_desc(unsigned long long* key, int P) {
  for (int kk = 2; kk <= P; kk <<= 1) {
    for (int j = kk >> 1; j > 0; j >>= 1) {
      for (int x = threadIdx.x; x < P; x += blockDim.x) {
        const int y = x ^ j;
        if (y > x) {
          const unsigned long long a = key[x], b = key[y];
          const bool desc = (x & kk) == 0;
          if (desc ? (a < b) : (a > b)) { key[x] = b; key[y] = a; }
        }
      }
      __syncthreads();
    }
  }
}

template <int DH>
__global__ __launch_bounds__(256) void route_topk_kernel(const float* __restrict__ means, int n_a,
                                                         int H, int M, int P, int k_eff, float scale,
                                                         float* __restrict__ scores_out,
                                                         int32_t* __restrict__ idx_out) {
  extern __shared__ unsigned long long keys[];
  __shared__ float qs[DH];
  const int i = blockIdx.x / H, h = blockIdx.x - (blockIdx.x / H) * H;
  const int D = H * DH;
  for (int d = threadIdx.x; d < DH; d += blockDim.x) qs[d] = means[(long long)i * D + h * DH + d];
  __syncthreads();
  for (int m = threadIdx.x; m < P; m += blockDim.x) {
    unsigned long long key = 0ull;
    if (m < M) {
      const float4* kr = reinterpret_cast<const float4*>(means + (long long)(n_a + m) * D + h * DH);
      float s = 0.0f;
#pragma unroll 8
      for (int d4 = 0; d4 < DH / 4; ++d4) {
        const float4 v = kr[d4];
        s = fmaf(qs[4 * d4 + 0], v.x, s);
        s = fmaf(qs[4 * d4 + 1], v.y, s);
        s = fmaf(qs[4 * d4 + 2], v.z, s);
        s = fmaf(qs[4 * d4 + 3], v.w, s);
      }
      s = s * scale;
      if (scores_out) scores_out[((long long)i * H + h) * M + m] = s;
      uint32_t b = __float_as_uint(s);
      if ((b << 1) == 0u) b = 0u;   // -0 and +0 compare equal: give them one key
      const uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);   // monotone in s
      key = ((unsigned long long)ord << 32) | (uint32_t)(~(uint32_t)m);   // ties: lower m first
    }
    keys[m] = key;
  }
  __syncthreads();
  bitonic_desc(keys, P);
  // the k_eff best, re-keyed so that a descending sort lists them by ascending index
  for (int x = threadIdx.x; x < P; x += blockDim.x) {
    unsigned long long k2 = 0ull;
    if (x < k_eff) {
      const uint32_t m = ~(uint32_t)(keys[x] & 0xffffffffull);
      k2 = (unsigned long long)(~m);
    }
    keys[x] = k2;
  }
  __syncthreads();
  bitonic_desc(keys, P);
  int32_t* dst = idx_out + ((long long)i * H + h) * k_eff;
  for (int x = threadIdx.x; x < k_eff; x += blockDim.x) {
    uint32_t m = ~(uint32_t)(keys[x] & 0xffffffffull);
    dst[x] = (int32_t)(m < (uint32_t)M ? m : (uint32_t)(M - 1));
  }
}

}  // namespace

RoutePlan plan_route(int n_a, int S, int H, int dh, int M, int Bv) {
  RoutePlan p{};
  p.D = H * dh;
  p.ngrp = (p.D + kPoolChannels - 1) / kPoolChannels;
  // aim for ~4096 scan blocks in total; splits are at least 32 tokens long
  const long long tokens = (long long)n_a * S + (long long)M * Bv;
  long long tps = (tokens * p.ngrp + 4095) / 4096;
  if (tps < 32) tps = 32;
  p.spq = (int)((S + tps - 1) / tps);
  p.tq = (S + p.spq - 1) / p.spq;
  p.spk = (int)((Bv + tps - 1) / tps);
  p.tk = (Bv + p.spk - 1) / p.spk;
  p.items = n_a * p.spq + M * p.spk;
  size_t partial = (size_t)p.items * p.D * sizeof(float);
  size_t means = (size_t)(n_a + M) * p.D * sizeof(float);
  p.off_partial = 0;
  p.off_means = align_up(partial);
  p.off_scores = p.off_means + align_up(means);
  p.total = p.off_scores;
  return p;
}

cast_status_t launch_pool_means(const void* q, const void* k, int n_a, int S, int M, int Bv,
                                const RoutePlan& p, float* partial, float* means,
                                hipStream_t stream) {
  if (p.items <= 0) return CAST_OK;
  hipLaunchKernelGGL(route_pool_kernel, dim3(p.items, p.ngrp), dim3(kPoolThreads), 0, stream,
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), n_a, S, Bv,
                     p.D, p.spq, p.tq, p.spk, p.tk, partial);
  cast_status_t st = check_launch("route_pool");
  if (st != CAST_OK) return st;
  hipLaunchKernelGGL(route_finalize_kernel, dim3((p.D + 255) / 256, n_a + M), dim3(256), 0, stream,
                     partial, n_a, p.D, p.spq, p.spk, S, Bv, means);
  return check_launch("route_finalize");
}

cast_status_t launch_route(const void* q, const void* k, int n_a, int S, int H, int dh, int M,
                           int Bv, int k_eff, float scale, float* scores_out, int32_t* idx_out,
                           const RoutePlan& p, void* ws, hipStream_t stream) {
  float* partial = reinterpret_cast<float*>(static_cast<char*>(ws) + p.off_partial);
  float* means = reinterpret_cast<float*>(static_cast<char*>(ws) + p.off_means);
  cast_status_t st = launch_pool_means(q, k, n_a, S, M, Bv, p, partial, means, stream);
  if (st != CAST_OK) return st;
  int P = 2;
  while (P < M) P <<= 1;
  const size_t shm = (size_t)P * sizeof(unsigned long long);
  switch (dh) {
    case 32:
      hipLaunchKernelGGL(route_topk_kernel<32>, dim3(n_a * H), dim3(256), shm, stream, means, n_a, H,
                         M, P, k_eff, scale, scores_out, idx_out);
      break;
    case 64:
      hipLaunchKernelGGL(route_topk_kernel<64>, dim3(n_a * H), dim3(256), shm, stream, means, n_a, H,
                         M, P, k_eff, scale, scores_out, idx_out);
      break;
    default:
      hipLaunchKernelGGL(route_topk_kernel<128>, dim3(n_a * H), dim3(256), shm, stream, means, n_a, H,
                         M, P, k_eff, scale, scores_out, idx_out);
      break;
  }
  return check_launch("route_topk");
}

}  // namespace cast
