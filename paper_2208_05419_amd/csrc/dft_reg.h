// dft_reg.h -- fixed-size complex DFTs held entirely in registers.
//
// DftReg<N, INV>::run(v) replaces v[0..N) by X[k] = sum_n v[n] exp(-+2 pi i n k / N)
// (INV: exp(+...)), unscaled, natural order in and out.  N is a compile-time product
// of 2, 3, 4 and 5.  A composite N = P * M is split in one of two ways:
//  * gcd(P, M) = 1: the prime-factor algorithm (Good; Thomas): with n = (M p + P m) mod N
//    and k = (M a kp + P b km) mod N, a = M^-1 mod P, b = P^-1 mod M, the DFT is an
//    M-point DFT along m followed by a P-point DFT along p with no twiddle factors;
//  * otherwise one decimation-in-time step (Cooley and Tukey): the P interleaved
//    subsequences v[r + P m] get M-point DFTs U_r, U_r[k] is multiplied by
//    exp(-+2 pi i r k / N), and for each k a P-point DFT over r gives X[k + M q].
// All indices are compile-time constants after unrolling, so the values stay in VGPRs.
//
// The twiddle constants are evaluated at compile time from Taylor series of sin and
// cos on the first quadrant (terms to x^29, far below double rounding there), with
// the quadrant reduction done exactly in integers.
#pragma once
#include <hip/hip_runtime.h>

namespace afno {
namespace ct {

constexpr double kTwoPi = 6.28318530717958647692528676655900577;

constexpr double taylor_sin(double x) {
  double t = x, s = x;
  for (int n = 1; n < 15; ++n) {
    t *= -x * x / ((2.0 * n) * (2.0 * n + 1.0));
    s += t;
  }
  return s;
}
constexpr double taylor_cos(double x) {
  double t = 1.0, s = 1.0;
  for (int n = 1; n < 15; ++n) {
    t *= -x * x / ((2.0 * n - 1.0) * (2.0 * n));
    s += t;
  }
  return s;
}
// cos and sin of 2 pi m / n
constexpr double cos2pi(long m, long n) {
  m %= n;
  if (m < 0) m += n;
  const long q = (4 * m) / n;                 // quadrant
  const double th = kTwoPi * (double)(4 * m - q * n) / (double)(4 * n);  // in [0, pi/2)
  return q == 0 ? taylor_cos(th) : q == 1 ? -taylor_sin(th) : q == 2 ? -taylor_cos(th) : taylor_sin(th);
}
constexpr double sin2pi(long m, long n) {
  m %= n;
  if (m < 0) m += n;
  const long q = (4 * m) / n;
  const double th = kTwoPi * (double)(4 * m - q * n) / (double)(4 * n);
  return q == 0 ? taylor_sin(th) : q == 1 ? taylor_cos(th) : q == 2 ? -taylor_sin(th) : -taylor_cos(th);
}

// table of exp(-2 pi i m / N), m in [0, N), as floats
template <int N>
struct Roots {
  float re[N], im[N];
  constexpr Roots() : re(), im() {
    for (int m = 0; m < N; ++m) {
      re[m] = (float)cos2pi(m, N);
      im[m] = (float)(-sin2pi(m, N));
    }
  }
};

constexpr int first_factor(int n) {
  return (n % 4 == 0 && n != 4) ? 4 : (n % 2 == 0 ? 2 : (n % 3 == 0 ? 3 : 5));
}

constexpr int gcd(int a, int b) { return b == 0 ? a : gcd(b, a % b); }

// the full power of the smallest prime dividing n (n itself when n is a prime power)
constexpr int prime_power(int n) {
  const int p = n % 2 == 0 ? 2 : (n % 3 == 0 ? 3 : 5);
  int q = 1;
  while (n % (q * p) == 0) q *= p;
  return q;
}

// x^-1 mod m for gcd(x, m) = 1
constexpr int inv_mod(int x, int m) {
  for (int y = 1; y < m; ++y)
    if ((x * y) % m == 1) return y;
  return m == 1 ? 0 : -1;
}

}  // namespace ct

__host__ __device__ __forceinline__ float2 c_add(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__host__ __device__ __forceinline__ float2 c_sub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__host__ __device__ __forceinline__ float2 c_mul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
// * (-i) forward, * (+i) inverse
template <bool INV>
__host__ __device__ __forceinline__ float2 c_rot(float2 a) {
  return INV ? make_float2(-a.y, a.x) : make_float2(a.y, -a.x);
}

template <int P, bool INV>
__host__ __device__ __forceinline__ void butterfly(float2* v) {
  if constexpr (P == 1) {
  } else if constexpr (P == 2) {
    const float2 a = v[0], b = v[1];
    v[0] = c_add(a, b);
    v[1] = c_sub(a, b);
  } else if constexpr (P == 3) {
    const float s3 = 0.866025403784438647f;
    const float2 a = v[0], t1 = c_add(v[1], v[2]);
    const float2 t2 = make_float2(a.x - 0.5f * t1.x, a.y - 0.5f * t1.y);
    const float2 d = c_sub(v[1], v[2]);
    const float2 t3 = c_rot<INV>(make_float2(s3 * d.x, s3 * d.y));
    v[0] = c_add(a, t1);
    v[1] = c_add(t2, t3);
    v[2] = c_sub(t2, t3);
  } else if constexpr (P == 4) {
    const float2 s02 = c_add(v[0], v[2]), d02 = c_sub(v[0], v[2]);
    const float2 s13 = c_add(v[1], v[3]), d13 = c_rot<INV>(c_sub(v[1], v[3]));
    v[0] = c_add(s02, s13);
    v[2] = c_sub(s02, s13);
    v[1] = c_add(d02, d13);
    v[3] = c_sub(d02, d13);
  } else {
    static_assert(P == 5, "radix must be 2, 3, 4 or 5");
    const float c1 = 0.309016994374947424f, c2 = -0.809016994374947424f;
    const float s1 = 0.951056516295153572f, s2 = 0.587785252292473129f;
    const float2 a0 = v[0];
    const float2 b1 = c_add(v[1], v[4]), d1 = c_sub(v[1], v[4]);
    const float2 b2 = c_add(v[2], v[3]), d2 = c_sub(v[2], v[3]);
    const float2 r1 = make_float2(a0.x + c1 * b1.x + c2 * b2.x, a0.y + c1 * b1.y + c2 * b2.y);
    const float2 r2 = make_float2(a0.x + c2 * b1.x + c1 * b2.x, a0.y + c2 * b1.y + c1 * b2.y);
    const float2 i1 = c_rot<INV>(make_float2(s1 * d1.x + s2 * d2.x, s1 * d1.y + s2 * d2.y));
    const float2 i2 = c_rot<INV>(make_float2(s2 * d1.x - s1 * d2.x, s2 * d1.y - s1 * d2.y));
    v[0] = c_add(a0, c_add(b1, b2));
    v[1] = c_add(r1, i1);
    v[4] = c_sub(r1, i1);
    v[2] = c_add(r2, i2);
    v[3] = c_sub(r2, i2);
  }
}

// exp(-+2 pi i m / N) with m a compile-time constant after unrolling
template <int N, bool INV>
__host__ __device__ __forceinline__ float2 root(int m) {
  constexpr ct::Roots<N> R{};
  return make_float2(R.re[m % N], INV ? -R.im[m % N] : R.im[m % N]);
}

template <int N, bool INV>
struct DftReg {
  // coprime split where N has two distinct primes, else a radix-4/2/3/5 step
  static constexpr bool kPfa = N > 5 && ct::prime_power(N) != N;
  static constexpr int P = (N <= 5) ? N : (kPfa ? ct::prime_power(N) : ct::first_factor(N));
  static constexpr int M = N / P;
  __host__ __device__ __forceinline__ static void run(float2* v) {
    if constexpr (M == 1) {
      butterfly<P, INV>(v);
    } else if constexpr (kPfa) {
      constexpr int A = ct::inv_mod(M % P, P), Bm = ct::inv_mod(P % M, M);
      float2 u[P][M];
#pragma unroll
      for (int p = 0; p < P; ++p)
#pragma unroll
        for (int m = 0; m < M; ++m) u[p][m] = v[(M * p + P * m) % N];
#pragma unroll
      for (int p = 0; p < P; ++p) DftReg<M, INV>::run(u[p]);
#pragma unroll
      for (int km = 0; km < M; ++km) {
        float2 w[P];
#pragma unroll
        for (int p = 0; p < P; ++p) w[p] = u[p][km];
        DftReg<P, INV>::run(w);
#pragma unroll
        for (int kp = 0; kp < P; ++kp) v[(M * A * kp + P * Bm * km) % N] = w[kp];
      }
    } else {
      float2 u[P][M];
#pragma unroll
      for (int r = 0; r < P; ++r)
#pragma unroll
        for (int m = 0; m < M; ++m) u[r][m] = v[r + P * m];
#pragma unroll
      for (int r = 0; r < P; ++r) DftReg<M, INV>::run(u[r]);
#pragma unroll
      for (int r = 1; r < P; ++r)
#pragma unroll
        for (int k = 1; k < M; ++k) u[r][k] = c_mul(u[r][k], root<N, INV>(r * k));
#pragma unroll
      for (int k = 0; k < M; ++k) {
        float2 w[P];
#pragma unroll
        for (int r = 0; r < P; ++r) w[r] = u[r][k];
        butterfly<P, INV>(w);
#pragma unroll
        for (int q = 0; q < P; ++q) v[k + M * q] = w[q];
      }
    }
  }
};

}  // namespace afno
