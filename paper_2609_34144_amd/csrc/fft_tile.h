// Register-resident DFTs for PAR tiles (edges 1..8), fully unrolled at compile
// time.  Unnormalised: forward X[k] = sum_n x[n] e^{-2 pi i k n / N}, inverse
// uses e^{+...}; the orthonormal 1/sqrt(N) factors are folded into the
// reconstruction coefficients by the caller.
//
// Even lengths use one radix-2 decimation-in-time step (recursively), odd
// lengths a direct DFT.  Twiddles are compile-time constants; the trivial ones
// (1, -1, +-i, and (+-1 +- i)/sqrt2) are applied with their exact short forms.
// Real-input transforms pass literal zero imaginary parts and rely on constant
// folding (the translation unit is built with -fno-signed-zeros so that x + 0
// folds) to prune the dead half of the work.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>
#include <utility>

namespace cast {
namespace fft {

// ---------------------------------------------------------------------------
// compile-time helpers
// ---------------------------------------------------------------------------
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// cos / sin of 2 pi k / n evaluated at compile time (Taylor series after
// reduction to [-pi/4, pi/4] by octant symmetry).
constexpr double kPi = 3.141592653589793238462643383279502884;
constexpr double taylor_sin(double x) {
  double t = x, s = x;
  for (int k = 1; k < 16; ++k) { t *= -x * x / ((2 * k) * (2 * k + 1)); s += t; }
  return s;
}
constexpr double taylor_cos(double x) {
  double t = 1, s = 1;
  for (int k = 1; k < 16; ++k) { t *= -x * x / ((2 * k - 1) * (2 * k)); s += t; }
  return s;
}
constexpr double tw_cos_core(double a) {  // a in [0, pi/2]
  return a > kPi / 4 ? taylor_sin(kPi / 2 - a) : taylor_cos(a);
}
constexpr double tw_cos(int k, int n) {
  // angle = 2 pi k / n, k in [0, n)
  double a = 2.0 * kPi * (double)k / (double)n;
  while (a > kPi) a -= 2.0 * kPi;
  if (a < 0) a = -a;                     // cos even
  if (a > kPi / 2) return -tw_cos_core(kPi - a);
  return tw_cos_core(a);
}
constexpr double tw_sin(int k, int n) {
  double a = 2.0 * kPi * (double)k / (double)n;
  while (a > kPi) a -= 2.0 * kPi;
  double sg = 1.0;
  if (a < 0) { a = -a; sg = -1.0; }      // sin odd
  if (a > kPi / 2) a = kPi - a;          // sin(pi - a) = sin a
  return sg * (a > kPi / 4 ? taylor_cos(kPi / 2 - a) : taylor_sin(a));
}

constexpr float kRsqrt2 = 0.70710678118654752440f;

// y = x * w where w = e^{SIGN 2 pi i K / N}, SIGN = -1 forward, +1 inverse.
template <int N, int K, bool INV>
__device__ __forceinline__ void twiddle(float xr, float xi, float& yr, float& yi) {
  constexpr int k = ((K % N) + N) % N;
  if constexpr (k == 0) {
    yr = xr; yi = xi;
  } else if constexpr (2 * k == N) {
    yr = -xr; yi = -xi;
  } else if constexpr (4 * k == N) {          // w = -i (fwd) / +i (inv)
    if constexpr (!INV) { yr = xi; yi = -xr; } else { yr = -xi; yi = xr; }
  } else if constexpr (4 * k == 3 * N) {      // w = +i (fwd) / -i (inv)
    if constexpr (!INV) { yr = -xi; yi = xr; } else { yr = xi; yi = -xr; }
  } else if constexpr (8 * k == N) {          // w = (1 -+ i)/sqrt2
    if constexpr (!INV) { yr = (xr + xi) * kRsqrt2; yi = (xi - xr) * kRsqrt2; }
    else { yr = (xr - xi) * kRsqrt2; yi = (xi + xr) * kRsqrt2; }
  } else if constexpr (8 * k == 3 * N) {      // w = (-1 -+ i)/sqrt2
    if constexpr (!INV) { yr = (xi - xr) * kRsqrt2; yi = -(xr + xi) * kRsqrt2; }
    else { yr = -(xr + xi) * kRsqrt2; yi = (xr - xi) * kRsqrt2; }
  } else if constexpr (8 * k == 5 * N) {      // w = (-1 +- i)/sqrt2
    if constexpr (!INV) { yr = -(xr + xi) * kRsqrt2; yi = (xr - xi) * kRsqrt2; }
    else { yr = (xi - xr) * kRsqrt2; yi = -(xr + xi) * kRsqrt2; }
  } else if constexpr (8 * k == 7 * N) {      // w = (1 +- i)/sqrt2
    if constexpr (!INV) { yr = (xr - xi) * kRsqrt2; yi = (xi + xr) * kRsqrt2; }
    else { yr = (xr + xi) * kRsqrt2; yi = (xi - xr) * kRsqrt2; }
  } else {
    constexpr float c = (float)tw_cos(k, N);
    constexpr float s = (float)(INV ? tw_sin(k, N) : -tw_sin(k, N));
    yr = xr * c - xi * s;
    yi = xr * s + xi * c;
  }
}

// In-place complex DFT of length N on elements r[O + S*n], i[O + S*n].
template <int N, bool INV, int S = 1, int O = 0, int L>
__device__ __forceinline__ void cdft(float (&r)[L], float (&i)[L]) {
  if constexpr (N == 1) {
    return;
  } else if constexpr (N % 2 == 0) {
    constexpr int H = N / 2;
    // even samples at O + 2S*n, odd at O + S + 2S*n
    cdft<H, INV, 2 * S, O>(r, i);
    cdft<H, INV, 2 * S, O + S>(r, i);
    float er[H], ei[H], orr[H], oi[H];
    static_for<0, H>([&](auto kk) {
      constexpr int k = decltype(kk)::value;
      er[k] = r[O + 2 * S * k];
      ei[k] = i[O + 2 * S * k];
      twiddle<N, k, INV>(r[O + S + 2 * S * k], i[O + S + 2 * S * k], orr[k], oi[k]);
    });
    static_for<0, H>([&](auto kk) {
      constexpr int k = decltype(kk)::value;
      r[O + S * k] = er[k] + orr[k];
      i[O + S * k] = ei[k] + oi[k];
      r[O + S * (k + H)] = er[k] - orr[k];
      i[O + S * (k + H)] = ei[k] - oi[k];
    });
  } else {
    float xr[N], xi[N];
    static_for<0, N>([&](auto nn) {
      constexpr int n = decltype(nn)::value;
      xr[n] = r[O + S * n];
      xi[n] = i[O + S * n];
    });
    static_for<0, N>([&](auto kk) {
      constexpr int k = decltype(kk)::value;
      float ar = xr[0], ai = xi[0];
      static_for<1, N>([&](auto nn) {
        constexpr int n = decltype(nn)::value;
        float tr, ti;
        twiddle<N, (k * n) % N, INV>(xr[n], xi[n], tr, ti);
        ar += tr;
        ai += ti;
      });
      r[O + S * k] = ar;
      i[O + S * k] = ai;
    });
  }
}

// Real-input forward DFT: x[0..N) -> X[0..N/2] (stored half).
template <int N>
__device__ __forceinline__ void rdft(const float (&x)[N], float (&Xr)[N / 2 + 1],
                                     float (&Xi)[N / 2 + 1]) {
  float r[N], i[N];
  static_for<0, N>([&](auto nn) {
    constexpr int n = decltype(nn)::value;
    r[n] = x[n];
    i[n] = 0.0f;
  });
  cdft<N, false>(r, i);
  static_for<0, N / 2 + 1>([&](auto kk) {
    constexpr int k = decltype(kk)::value;
    Xr[k] = r[k];
    Xi[k] = (k == 0 || 2 * k == N) ? 0.0f : i[k];
  });
}

// Inverse of a Hermitian spectrum given by its stored half X[0..N/2]:
// x[n] = Re X[0] + [N even] Re X[N/2] (-1)^n + 2 Re sum_{0<k<N/2} X[k] e^{+2 pi i k n / N}.
template <int N>
__device__ __forceinline__ void c2r(const float (&Xr)[N / 2 + 1], const float (&Xi)[N / 2 + 1],
                                    float (&x)[N]) {
  float r[N], i[N];
  static_for<0, N>([&](auto kk) {
    constexpr int k = decltype(kk)::value;
    if constexpr (k == 0 || 2 * k == N) {
      r[k] = Xr[k];
      i[k] = 0.0f;
    } else if constexpr (2 * k < N) {
      r[k] = Xr[k];
      i[k] = Xi[k];
    } else {
      r[k] = Xr[N - k];
      i[k] = -Xi[N - k];
    }
  });
  cdft<N, true>(r, i);
  static_for<0, N>([&](auto nn) {
    constexpr int n = decltype(nn)::value;
    x[n] = r[n];
  });
}

}  // namespace fft
}  // namespace cast
