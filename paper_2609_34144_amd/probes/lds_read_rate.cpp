// LDS read bandwidth of one MI355X CU: the context for the routed-attention
// kernel, whose MFMA phase reads 1 KB of operands from LDS per 32x32x16 MFMA.
//
// One workgroup of 512 threads (8 waves) per CU; every wave loops over
// ds_read_b128 (16 B per lane) or the transposing ds_read_b64_tr_b16 (8 B per
// lane) at conflict-free addresses of a 64 KB LDS buffer, 8 independent reads in
// flight, and folds the results so that the reads stay.  Prints bytes read per
// CU per shader-clock cycle (the clock taken from s_memtime over the loop, in
// wave 0 of each workgroup) and per nanosecond.
//
//   hipcc -O3 -std=c++17 --offload-arch=gfx950 -Xclang -target-feature -Xclang -packed-fp32-ops \
//       -x hip paper_2609_34144_amd/probes/lds_read_rate.cpp -o /tmp/lds_read_rate && /tmp/lds_read_rate
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

#define CHECK(x)                                                              \
  do {                                                                        \
    hipError_t e_ = (x);                                                      \
    if (e_ != hipSuccess) {                                                   \
      fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
      exit(1);                                                                \
    }                                                                         \
  } while (0)

constexpr int kCUs = 256, kThreads = 512, kWords = 65536 / 16;

template <bool TR>
__global__ __launch_bounds__(kThreads, 1) void probe(unsigned* out, long long* cyc, int iters) {
  __shared__ __attribute__((aligned(16))) u32x4 buf[kWords];
  const int t = threadIdx.x;
  for (int i = t; i < kWords; i += kThreads) buf[i] = u32x4{(unsigned)i, 1u, 2u, 3u};
  __syncthreads();
  const int lane = t & 63, wave = t >> 6;
  unsigned acc = 0;
  const long long c0 = clock64();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      // consecutive lanes read consecutive 16-byte words: conflict-free
      const int w = ((it * 8 + r) * 64 + wave * 512 + lane) & (kWords - 1);
      if constexpr (TR) {
        const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4*)((__attribute__((address_space(3))) char*)buf + (size_t)w * 8));
        acc += (unsigned)v.x + (unsigned)v.w;
      } else {
        const u32x4 v = buf[w];
        acc += v.x + v.w;
      }
    }
  }
  const long long c1 = clock64();
  out[blockIdx.x * kThreads + t] = acc;
  if (t == 0) cyc[blockIdx.x] = c1 - c0;
}

template <bool TR>
void run(const char* name, unsigned* d, long long* c, int iters) {
  hipLaunchKernelGGL((probe<TR>), dim3(kCUs), dim3(kThreads), 0, 0, d, c, iters);   // warm-up
  CHECK(hipGetLastError());
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  CHECK(hipEventRecord(e0));
  hipLaunchKernelGGL((probe<TR>), dim3(kCUs), dim3(kThreads), 0, 0, d, c, iters);
  CHECK(hipGetLastError());
  CHECK(hipEventRecord(e1));
  CHECK(hipEventSynchronize(e1));
  float ms = 0.0f;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  static long long h[kCUs];
  CHECK(hipMemcpy(h, c, sizeof(h), hipMemcpyDeviceToHost));
  double cy = 0.0;
  for (int i = 0; i < kCUs; ++i) cy += (double)h[i];
  cy /= kCUs;
  const double bytes_cu = (double)iters * 8 * kThreads * (TR ? 8 : 16);
  printf("| %s | %.1f | %.1f | %.2f |\n", name, bytes_cu / cy, bytes_cu * kCUs / (ms * 1e-3) / 1e12,
         cy / (ms * 1e6));
  CHECK(hipEventDestroy(e0));
  CHECK(hipEventDestroy(e1));
}

int main() {
  unsigned* d = nullptr;
  long long* c = nullptr;
  CHECK(hipMalloc(&d, kCUs * kThreads * sizeof(unsigned)));
  CHECK(hipMalloc(&c, kCUs * sizeof(long long)));
  const int iters = 20000;
  printf("| read | bytes per CU per cycle | chip TB/s | loop clock GHz (from the kernel time) |\n|---|---|---|---|\n");
  run<false>("ds_read_b128", d, c, iters);
  run<true>("ds_read_b64_tr_b16", d, c, iters);
  CHECK(hipFree(d));
  CHECK(hipFree(c));
  return 0;
}
