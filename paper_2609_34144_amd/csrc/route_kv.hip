// Pooled chunk scores and TopK routing on gfx950 (Sec. 4.4 eq:pooled, eq:topk).
//
// route_means  HBM scan: one 8-wave block per (128-channel group, segment), where a
//              segment is an anchor frame of Q or a history chunk of K; fp32 sums of
//              16-byte coalesced bf16 loads, reduced in a fixed order to the pooled
//              means q_bar, k_bar.
// route_topk   one block per (anchor, head): scores s = scale * q_bar . k_bar for
//              all M chunks, then the k_eff best under (score descending, chunk index
//              ascending), written in ascending chunk order: by counting larger keys
//              for up to kRankMaxM chunks, by bitonic sorts in LDS above.
// No atomics anywhere: results are bit-identical across runs.
#include "cast_common.h"

namespace cast {

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// One block per (channel group of kMeansCh channels, segment); segment s < n_a is
// anchor frame s of q (S tokens), the others are the history chunks of k (Bv
// tokens).  Wave w sums tokens [w T / 8, (w + 1) T / 8) of the segment: its lane
// (row r = lane / 16, column = lane % 16) adds 8 consecutive bf16 channels of the
// tokens t = r mod 4, so one load instruction reads 4 tokens x 256 contiguous
// bytes, eight of them in flight.  The 4 rows are summed by two lane exchanges,
// the 8 waves through LDS in wave order: a fixed order, so runs are bit-identical.
__global__ __launch_bounds__(kMeansWaves * 64) void route_means_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, int n_a, int S, int Bv,
    int D, float* __restrict__ means) {
  __shared__ float red[kMeansWaves][kMeansCh];
  const int grp = blockIdx.x, seg = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int col = lane & 15, row = lane >> 4;
  const int c = grp * kMeansCh + col * 8;
  const uint16_t* base;
  int T;
  if (seg < n_a) {
    base = q + (long long)seg * S * D;
    T = S;
  } else {
    base = k + (long long)(seg - n_a) * Bv * D;
    T = Bv;
  }
  const int t0 = (int)((long long)T * wave / kMeansWaves);
  const int t1 = (int)((long long)T * (wave + 1) / kMeansWaves);
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0f;
  auto add = [&](const u32x4& v) {
    acc[0] += bf16lo(v.x); acc[1] += bf16hi(v.x);
    acc[2] += bf16lo(v.y); acc[3] += bf16hi(v.y);
    acc[4] += bf16lo(v.z); acc[5] += bf16hi(v.z);
    acc[6] += bf16lo(v.w); acc[7] += bf16hi(v.w);
  };
  if (c < D) {
    const long long step = (long long)D / 2;        // 4 tokens, in u32x4 units
    const u32x4* p = reinterpret_cast<const u32x4*>(base + (long long)(t0 + row) * D + c);
    int t = t0 + row;
    for (; t + 28 < t1; t += 32) {
      u32x4 v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p + u * step);
#pragma unroll
      for (int u = 0; u < 8; ++u) add(v[u]);
      p += 8 * step;
    }
    for (; t < t1; t += 4) {
      add(__builtin_nontemporal_load(p));
      p += step;
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    acc[e] += __shfl_xor(acc[e], 16);
    acc[e] += __shfl_xor(acc[e], 32);
  }
  if (row == 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red[wave][col * 8 + e] = acc[e];
  }
  __syncthreads();
  if (threadIdx.x < kMeansCh) {
    const int ch = grp * kMeansCh + threadIdx.x;
    if (ch < D) {
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < kMeansWaves; ++w) s += red[w][threadIdx.x];
      means[(long long)seg * D + ch] = s / (float)T;
    }
  }
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

// Score key of chunk m: ordered float bits (monotone in s), then the inverted chunk
// index, so a larger key is a better chunk and ties go to the lower index.
__device__ __forceinline__ unsigned long long score_key(float s, int m) {
  uint32_t b = __float_as_uint(s);
  if ((b << 1) == 0u) b = 0u;   // -0 and +0 compare equal: give them one key
  const uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);
  return ((unsigned long long)ord << 32) | (uint32_t)(~(uint32_t)m);
}

// One block of 256 threads per (anchor i, head h).  Scores: wave w takes chunks
// m = w, w + 4, ..., four at a time; each lane multiplies its dims of q_bar and
// k_bar_m and the wave sums the products by lane exchanges (fixed order).  With
// M <= kRankMaxM the selection counts, for every chunk, the keys larger than its
// own (no sort): chunk m is kept when fewer than k_eff are larger, and its output
// slot is the number of kept chunks below m (ascending chunk order).  Larger M
// sorts the keys with two bitonic passes in LDS.
template <int DH>
__global__ __launch_bounds__(256) void route_topk_kernel(const float* __restrict__ means, int n_a,
                                                         int H, int M, int P, int k_eff, float scale,
                                                         float* __restrict__ scores_out,
                                                         int32_t* __restrict__ idx_out) {
  extern __shared__ unsigned long long keys[];
  __shared__ unsigned long long kept[kRankMaxM / 64];
  constexpr int PER = DH / 64 > 0 ? DH / 64 : 1;       // dims per lane
  const int i = blockIdx.x / H, h = blockIdx.x - (blockIdx.x / H) * H;
  const int D = H * DH;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float qv[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int d = lane * PER + e;
    qv[e] = d < DH ? means[(long long)i * D + h * DH + d] : 0.0f;
  }
  for (int m0 = wave * 4; m0 < M; m0 += 16) {
    float part[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int m = m0 + u;
      part[u] = 0.0f;
      if (m < M) {
        const float* kr = means + (long long)(n_a + m) * D + h * DH;
#pragma unroll
        for (int e = 0; e < PER; ++e) {
          const int d = lane * PER + e;
          if (d < DH) part[u] = fmaf(qv[e], kr[d], part[u]);
        }
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1)
#pragma unroll
      for (int u = 0; u < 4; ++u) part[u] += __shfl_xor(part[u], o);
    if (lane < 4 && m0 + lane < M) {
      const int m = m0 + lane;
      const float sc = (lane == 0 ? part[0] : lane == 1 ? part[1] : lane == 2 ? part[2] : part[3]) * scale;
      if (scores_out) scores_out[((long long)i * H + h) * M + m] = sc;
      keys[m] = score_key(sc, m);
    }
  }
  int32_t* dst = idx_out + ((long long)i * H + h) * k_eff;
  if (M <= kRankMaxM) {
    __syncthreads();
    for (int m = threadIdx.x; m - (int)(threadIdx.x & 63) < M; m += blockDim.x) {
      bool keep = false;
      if (m < M) {
        const unsigned long long mine = keys[m];
        int rank = 0;
        for (int x = 0; x < M; ++x) rank += keys[x] > mine ? 1 : 0;
        keep = rank < k_eff;
      }
      const unsigned long long mask = __ballot(keep);
      if ((threadIdx.x & 63) == 0) kept[m >> 6] = mask;
    }
    __syncthreads();
    for (int m = threadIdx.x; m < M; m += blockDim.x) {
      const unsigned long long own = kept[m >> 6];
      if ((own >> (m & 63)) & 1ull) {
        int pos = __popcll(own & ((1ull << (m & 63)) - 1ull));
        for (int g = 0; g < (m >> 6); ++g) pos += __popcll(kept[g]);
        dst[pos] = m;
      }
    }
    return;
  }
  for (int m = M + threadIdx.x; m < P; m += blockDim.x) keys[m] = 0ull;
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
  for (int x = threadIdx.x; x < k_eff; x += blockDim.x) {
    uint32_t m = ~(uint32_t)(keys[x] & 0xffffffffull);
    dst[x] = (int32_t)(m < (uint32_t)M ? m : (uint32_t)(M - 1));
  }
}

}  // namespace

RoutePlan plan_route(int n_a, int S, int H, int dh, int M, int Bv) {
  (void)S;
  (void)Bv;
  RoutePlan p{};
  p.D = H * dh;
  p.ngrp = (p.D + kMeansCh - 1) / kMeansCh;
  p.segs = n_a + M;
  p.off_means = 0;
  p.total = align_up((size_t)p.segs * p.D * sizeof(float));
  return p;
}

cast_status_t launch_pool_means(const void* q, const void* k, int n_a, int S, int M, int Bv,
                                const RoutePlan& p, float* means, hipStream_t stream) {
  if (p.segs <= 0) return CAST_OK;
  hipLaunchKernelGGL(route_means_kernel, dim3(p.ngrp, n_a + M), dim3(kMeansWaves * 64), 0, stream,
                     static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), n_a, S, Bv,
                     p.D, means);
  return check_launch("route_means");
}

cast_status_t launch_route(const void* q, const void* k, int n_a, int S, int H, int dh, int M,
                           int Bv, int k_eff, float scale, float* scores_out, int32_t* idx_out,
                           const RoutePlan& p, void* ws, hipStream_t stream) {
  float* means = reinterpret_cast<float*>(static_cast<char*>(ws) + p.off_means);
  cast_status_t st = launch_pool_means(q, k, n_a, S, M, Bv, p, means, stream);
  if (st != CAST_OK) return st;
  int P = 2;
  while (P < M) P <<= 1;
  const size_t shm = (size_t)(P > 64 ? P : 64) * sizeof(unsigned long long);
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
