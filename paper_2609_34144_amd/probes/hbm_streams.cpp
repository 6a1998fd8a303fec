// HBM stream ceilings of one MI355X, and the access pattern of PAR's
// reconstruction pass on its own: the context for PAR's roofline fraction.
//
// Over a 3.36 GB fp32 buffer (64 frames of 64 x 64 tokens x 3072 channels):
//   read     grid-stride 16-byte loads, summed
//   copy     grid-stride 16-byte loads and stores to a second buffer (nontemporal
//            stores)
//   rmw      in-place x += c, grid-stride 16-byte accesses
//   hipMemcpy device to device
//   par      PAR's reconstruction pattern without its arithmetic: one 64-lane
//            wave per (8x8 tile, 64-channel block) takes FPW target frames in
//            turn, loading the tile's 64 tokens (one float per lane and token,
//            256 contiguous bytes per wave and token), adding a constant and
//            storing them back.  FPW = 64 is PAR's own schedule (one wave walks
//            every target of its tile and channel block); FPW = 1 puts one frame
//            per wave.
// Best of five timed runs each; rates count bytes read plus bytes written.
//
//   hipcc -O3 -std=c++17 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       -x hip paper_2609_34144_amd/probes/hbm_streams.cpp -o /tmp/hbm_streams && /tmp/hbm_streams
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

typedef float f32x4 __attribute__((ext_vector_type(4)));

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
      exit(1);                                                                \
    }                                                                         \
  } while (0)

constexpr int kHg = 64, kWg = 64, kD = 3072, kF = 64;
constexpr long long kFrame = (long long)kHg * kWg * kD;
constexpr long long kN = kF * kFrame;   // floats
constexpr int kU = 4;                   // 16-byte accesses in flight per thread

__global__ __launch_bounds__(256) void read_k(const f32x4* a, float* out, long long nv) {
  const long long stride = (long long)gridDim.x * blockDim.x * kU;
  f32x4 s{};
  for (long long i0 = (long long)blockIdx.x * blockDim.x * kU + threadIdx.x; i0 < nv; i0 += stride)
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const long long i = i0 + (long long)u * blockDim.x;
      if (i < nv) s += a[i];
    }
  const float t = s.x + s.y + s.z + s.w;
  if (t == 12345.0f) out[0] = t;   // keeps the loads
}

__global__ __launch_bounds__(256) void copy_k(const f32x4* a, f32x4* b, long long nv) {
  const long long stride = (long long)gridDim.x * blockDim.x * kU;
  for (long long i0 = (long long)blockIdx.x * blockDim.x * kU + threadIdx.x; i0 < nv; i0 += stride) {
    f32x4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const long long i = i0 + (long long)u * blockDim.x;
      if (i < nv) v[u] = a[i];
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const long long i = i0 + (long long)u * blockDim.x;
      if (i < nv) __builtin_nontemporal_store(v[u], &b[i]);
    }
  }
}

__global__ __launch_bounds__(256) void rmw_k(f32x4* a, long long nv, float c) {
  const long long stride = (long long)gridDim.x * blockDim.x * kU;
  for (long long i0 = (long long)blockIdx.x * blockDim.x * kU + threadIdx.x; i0 < nv; i0 += stride) {
    f32x4 v[kU];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const long long i = i0 + (long long)u * blockDim.x;
      if (i < nv) v[u] = a[i];
    }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const long long i = i0 + (long long)u * blockDim.x;
      if (i < nv) a[i] = v[u] + c;
    }
  }
}

// grid (tile, 64-channel block, frame group); FPW frames per wave
template <int FPW>
__global__ __launch_bounds__(64) void par_pattern_k(float* x, float c) {
  const int tile = blockIdx.x, chb = blockIdx.y, f0 = blockIdx.z * FPW;
  const int ty = tile / (kWg / 8), tx = tile % (kWg / 8);
  const int lane = threadIdx.x;
  for (int f = f0; f < f0 + FPW; ++f) {
    float* base = x + (long long)f * kFrame;
    float v[64];
#pragma unroll
    for (int k = 0; k < 64; ++k)
      v[k] = base[((long long)(ty * 8 + k / 8) * kWg + tx * 8 + k % 8) * kD + chb * 64 + lane];
#pragma unroll
    for (int k = 0; k < 64; ++k)
      base[((long long)(ty * 8 + k / 8) * kWg + tx * 8 + k % 8) * kD + chb * 64 + lane] = v[k] + c;
  }
}

template <class G>
float best_ms(G g) {
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  g();   // warm-up
  CHECK(hipDeviceSynchronize());
  float best = 1e30f;
  for (int r = 0; r < 5; ++r) {
    CHECK(hipEventRecord(e0));
    g();
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    float ms = 0.0f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    best = ms < best ? ms : best;
  }
  CHECK(hipEventDestroy(e0));
  CHECK(hipEventDestroy(e1));
  return best;
}

void report(const char* name, float ms, double bytes) {
  printf("| %s | %.3f | %.2f | %.0f%% |\n", name, ms, bytes / (ms * 1e-3) / 1e12, 100.0 * bytes / (ms * 1e-3) / 8e12);
}

int main() {
  float *x = nullptr, *y = nullptr, *o = nullptr;
  CHECK(hipMalloc(&x, kN * sizeof(float)));
  CHECK(hipMalloc(&y, kN * sizeof(float)));
  CHECK(hipMalloc(&o, sizeof(float)));
  CHECK(hipMemset(x, 0, kN * sizeof(float)));
  CHECK(hipMemset(y, 0, kN * sizeof(float)));
  const long long nv = kN / 4;
  const double gb = kN * 4.0;
  const int blocks = 16384;
  printf("buffer %.2f GB\n\n| stream | ms | TB/s | of 8 TB/s |\n|---|---|---|---|\n", gb / 1e9);
  report("read", best_ms([&] { hipLaunchKernelGGL(read_k, dim3(blocks), dim3(256), 0, 0, (const f32x4*)x, o, nv); }), gb);
  report("copy", best_ms([&] { hipLaunchKernelGGL(copy_k, dim3(blocks), dim3(256), 0, 0, (const f32x4*)x, (f32x4*)y, nv); }), 2 * gb);
  report("rmw", best_ms([&] { hipLaunchKernelGGL(rmw_k, dim3(blocks), dim3(256), 0, 0, (f32x4*)x, nv, 1.0f); }), 2 * gb);
  report("hipMemcpy", best_ms([&] { CHECK(hipMemcpyAsync(y, x, kN * sizeof(float), hipMemcpyDeviceToDevice, 0)); }), 2 * gb);
  const dim3 pg(kHg / 8 * (kWg / 8), kD / 64);
  report("par, FPW 64", best_ms([&] { hipLaunchKernelGGL((par_pattern_k<64>), dim3(pg.x, pg.y, kF / 64), dim3(64), 0, 0, x, 1.0f); }), 2 * gb);
  report("par, FPW 16", best_ms([&] { hipLaunchKernelGGL((par_pattern_k<16>), dim3(pg.x, pg.y, kF / 16), dim3(64), 0, 0, x, 1.0f); }), 2 * gb);
  report("par, FPW 1", best_ms([&] { hipLaunchKernelGGL((par_pattern_k<1>), dim3(pg.x, pg.y, kF), dim3(64), 0, 0, x, 1.0f); }), 2 * gb);
  CHECK(hipGetLastError());
  CHECK(hipFree(x));
  CHECK(hipFree(y));
  CHECK(hipFree(o));
  return 0;
}
