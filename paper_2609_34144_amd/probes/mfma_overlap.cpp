// Matrix-core ceiling of one MI355X and the cost of VALU work between a wave's own
// MFMAs: the context for the attention kernel's roofline.
//
// One workgroup of 4 waves per CU (one wave per SIMD, as the earlier single-wave
// attention kernel ran), each wave a loop of 8 independent v_mfma_f32_32x32x16_bf16 chains with K
// independent VALU instructions after every MFMA (K fused multiply-adds, or K
// exponentials each followed by a multiply).  Prints the time per MFMA per wave;
// with no VALU work that is the chip's sustained matrix-core rate:
// 1024 SIMDs x 32768 FLOP / (time per MFMA).  No memory traffic beyond one store
// per thread at the end.
//
//   hipcc -O3 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       -x hip paper_2609_34144_amd/probes/mfma_overlap.cpp -o /tmp/mfma_overlap && /tmp/mfma_overlap
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
      exit(1);                                                                \
    }                                                                         \
  } while (0)

constexpr int kCUs = 256, kThreads = 256, kChains = 8;

template <int K, bool EXP>
__global__ __launch_bounds__(kThreads, 1) void probe(float* out, int iters, float seed) {
  f32x16 acc[kChains];
  for (int m = 0; m < kChains; ++m) acc[m] = f32x16{};
  const unsigned t = threadIdx.x;
  const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{0x3f803f80u ^ t, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
  const bf16x8 b = __builtin_bit_cast(bf16x8, u32x4{0x3f803f80u, 0x3f803f80u ^ t, 0x3f803f80u, 0x3f803f80u});
  float v[8];
  for (int i = 0; i < 8; ++i) v[i] = seed * (float)(t + i) * 1e-3f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int m = 0; m < kChains; ++m) {
      acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[m], 0, 0, 0);
#pragma unroll
      for (int k = 0; k < K; ++k) {
        float& x = v[(m * K + k) % 8];
        if constexpr (EXP) x = __builtin_amdgcn_exp2f(x) * 0.5f;
        else x = fmaf(x, 0.999f, 0.001f);
      }
      __builtin_amdgcn_sched_barrier(0);   // keep the VALU work between the MFMAs
    }
  }
  float s = 0.0f;
  for (int m = 0; m < kChains; ++m)
    for (int e = 0; e < 16; ++e) s += acc[m][e];
  for (int i = 0; i < 8; ++i) s += v[i];
  out[blockIdx.x * kThreads + t] = s;
}

template <int K, bool EXP>
float time_ms(float* d, int iters) {
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  hipLaunchKernelGGL((probe<K, EXP>), dim3(kCUs), dim3(kThreads), 0, 0, d, iters, 1.0f);   // warm-up
  CHECK(hipGetLastError());
  CHECK(hipEventRecord(e0));
  hipLaunchKernelGGL((probe<K, EXP>), dim3(kCUs), dim3(kThreads), 0, 0, d, iters, 1.0f);
  CHECK(hipGetLastError());
  CHECK(hipEventRecord(e1));
  CHECK(hipEventSynchronize(e1));
  float ms = 0.0f;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  CHECK(hipEventDestroy(e0));
  CHECK(hipEventDestroy(e1));
  return ms;
}

template <int K, bool EXP>
void report(float* d, int iters, float base_ms) {
  const float ms = time_ms<K, EXP>(d, iters);
  const double ns = ms * 1e6 / ((double)iters * kChains);
  printf("| %d | %s | %.2f | %.3f |\n", K, EXP ? "exp2 + mul" : "fma", ns, ms / base_ms);
}

int main() {
  float* d = nullptr;
  CHECK(hipMalloc(&d, kCUs * kThreads * sizeof(float)));
  const int iters = 4000;
  const float base = time_ms<0, false>(d, iters);
  const double ns = base * 1e6 / ((double)iters * kChains);
  printf("MFMA only: %.2f ns per 32x32x16 bf16 MFMA per wave -> %.3f PFLOP/s on %d SIMDs\n\n", ns,
         4.0 * kCUs * 32768.0 / ns * 1e-6, 4 * kCUs);
  printf("| VALU per MFMA | kind | ns per MFMA | time / MFMA-only |\n|---|---|---|---|\n");
  report<2, false>(d, iters, base);
  report<4, false>(d, iters, base);
  report<8, false>(d, iters, base);
  report<1, true>(d, iters, base);
  report<2, true>(d, iters, base);
  report<4, true>(d, iters, base);
  CHECK(hipFree(d));
  return 0;
}
