// VALU work of one wave beside the MFMAs of another wave on the same SIMD: the
// context for the routed-attention kernel's two-waves-per-SIMD schedule and for
// its fp32 row sums.
//
// One workgroup of 8 waves per CU.  Waves w and w + 4 share SIMD w % 4: waves 0-3
// issue back-to-back v_mfma_f32_32x32x16_bf16 (six independent chains), waves
// 4-7 run a VALU loop, or idle.  Each wave times its own loop with s_memtime;
// the table gives cycles per loop slot for each group, alone and side by side.
// VALU loops per slot:
//   fma        8 fused multiply-adds
//   exp        2 exponentials
//   sm+dot2    2 x (fma, exp), v_cvt_pk_bf16_f32, v_dot2_f32_bf16 row sum, 2 mul
//   sm+cvt     2 x (fma, exp), v_cvt_pk_bf16_f32, 2 fp32 adds of the packed halves, 2 mul
//   sm fp32    2 x (fma, exp), 2 fp32 adds, 2 mul
//
//   hipcc -O3 -std=c++17 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       -x hip paper_2609_34144_amd/probes/valu_beside_mfma.cpp -o /tmp/valu_beside_mfma && /tmp/valu_beside_mfma
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
      exit(1);                                                                \
    }                                                                         \
  } while (0)

constexpr int kCUs = 256, kSlots = 6;
enum { V_NONE, V_FMA, V_EXP, V_SM_DOT2, V_SM_CVT, V_SM_FP32 };

// MFMA: waves 0-3 issue MFMAs; VK: what waves 4-7 do
template <bool MFMA, int VK>
__global__ __launch_bounds__(512, 1) void probe(float* out, long long* cyc, int iters) {
  const unsigned t = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const bf16x8 a = __builtin_bit_cast(bf16x8, u32x4{0x3f803f80u ^ t, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
  const bf16x8 b = __builtin_bit_cast(bf16x8, u32x4{0x3f803f80u, 0x3f803f80u ^ t, 0x3f803f80u, 0x3f803f80u});
  f32x16 acc[kSlots];
  for (int m = 0; m < kSlots; ++m) acc[m] = f32x16{};
  float v[16];
  for (int i = 0; i < 16; ++i) v[i] = (float)(t + i) * 1e-3f;
  float rs = 0.0f;
  __syncthreads();
  const long long c0 = clock64();
  if (wave < 4) {
    if constexpr (MFMA) {
      for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int m = 0; m < kSlots; ++m) {
          acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[m], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  } else if constexpr (VK != V_NONE) {
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int m = 0; m < kSlots; ++m) {
        if constexpr (VK == V_FMA) {
#pragma unroll
          for (int k = 0; k < 8; ++k) v[(m * 8 + k) % 16] = fmaf(v[(m * 8 + k) % 16], 0.999f, 0.001f);
        } else if constexpr (VK == V_EXP) {
#pragma unroll
          for (int k = 0; k < 2; ++k) v[(m * 2 + k) % 16] = __builtin_amdgcn_exp2f(v[(m * 2 + k) % 16]);
        } else {
          const int i0 = (m * 2) % 16;
          const float p0 = __builtin_amdgcn_exp2f(fmaf(v[i0], 0.5f, -1.0f));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(v[i0 + 1], 0.5f, -1.0f));
          if constexpr (VK == V_SM_FP32) {
            rs += p0;
            rs += p1;
          } else {
            const unsigned w = __builtin_bit_cast(unsigned, __builtin_convertvector(f32x2{p0, p1}, bf16x2));
            if constexpr (VK == V_SM_DOT2) {
              rs = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w),
                                                   bf16x2{(__bf16)1.0f, (__bf16)1.0f}, rs, false);
            } else {
              rs += __uint_as_float(w << 16);
              rs += __uint_as_float(w & 0xffff0000u);
            }
          }
          v[i0] = p0 * 0.25f;
          v[i0 + 1] = p1 * 0.25f;
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  const long long c1 = clock64();
  float s = rs;
  for (int m = 0; m < kSlots; ++m)
    for (int e = 0; e < 16; ++e) s += acc[m][e];
  for (int i = 0; i < 16; ++i) s += v[i];
  out[blockIdx.x * 512 + t] = s;
  if ((t & 63) == 0) cyc[blockIdx.x * 8 + wave] = c1 - c0;
}

template <bool MFMA, int VK>
void run(const char* mfma, const char* valu, float* d, long long* c, int iters) {
  hipLaunchKernelGGL((probe<MFMA, VK>), dim3(kCUs), dim3(512), 0, 0, d, c, iters);   // warm-up
  CHECK(hipGetLastError());
  hipLaunchKernelGGL((probe<MFMA, VK>), dim3(kCUs), dim3(512), 0, 0, d, c, iters);
  CHECK(hipGetLastError());
  CHECK(hipDeviceSynchronize());
  static long long h[kCUs * 8];
  CHECK(hipMemcpy(h, c, sizeof(h), hipMemcpyDeviceToHost));
  double m = 0.0, v = 0.0;
  for (int i = 0; i < kCUs; ++i) {
    for (int w = 0; w < 4; ++w) m += h[i * 8 + w];
    for (int w = 4; w < 8; ++w) v += h[i * 8 + w];
  }
  const double slots = (double)iters * kSlots * kCUs * 4;
  printf("| %s | %s | %.1f | %.1f |\n", mfma, valu, MFMA ? m / slots : 0.0, VK != V_NONE ? v / slots : 0.0);
}

int main() {
  float* d = nullptr;
  long long* c = nullptr;
  CHECK(hipMalloc(&d, kCUs * 512 * sizeof(float)));
  CHECK(hipMalloc(&c, kCUs * 8 * sizeof(long long)));
  const int iters = 3000;
  printf("| waves 0-3 | waves 4-7 | MFMA wave cycles/slot | VALU wave cycles/slot |\n|---|---|---|---|\n");
  run<true, V_NONE>("MFMA", "idle", d, c, iters);
  run<false, V_FMA>("idle", "fma", d, c, iters);
  run<true, V_FMA>("MFMA", "fma", d, c, iters);
  run<false, V_EXP>("idle", "exp", d, c, iters);
  run<true, V_EXP>("MFMA", "exp", d, c, iters);
  run<false, V_SM_DOT2>("idle", "sm+dot2", d, c, iters);
  run<true, V_SM_DOT2>("MFMA", "sm+dot2", d, c, iters);
  run<false, V_SM_CVT>("idle", "sm+cvt", d, c, iters);
  run<true, V_SM_CVT>("MFMA", "sm+cvt", d, c, iters);
  run<false, V_SM_FP32>("idle", "sm fp32", d, c, iters);
  run<true, V_SM_FP32>("MFMA", "sm fp32", d, c, iters);
  CHECK(hipFree(d));
  CHECK(hipFree(c));
  return 0;
}
