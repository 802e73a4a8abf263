// fft_lds.h -- batched mixed-radix (2, 3, 4, 5) complex FFTs over LDS for gfx950.
//
// A workgroup transforms NSIG signals of length N that sit in LDS as
// buf[n * ld + s] (float2, signal s fastest, so the 64 lanes of a wave touch
// consecutive 8-byte words).  Thread t owns signal s = t % NSIG and butterfly slot
// t / NSIG of NSUB = blockDim / NSIG slots.
//
// Each pass is one radix-R Stockham step (Govindaraju et al., "High performance
// discrete Fourier transforms on graphics processors", SC'08): with L the product of
// the radices already applied, butterfly j (0 <= j < N/R, k = j mod L) reads
// v_t = buf[j + t N/R], multiplies v_t by exp(-+2 pi i t k / (L R)), takes an R-point
// DFT and writes result t to position (j - k) R + k + t L.  After the last pass the
// spectrum is in natural order.  The pass is done in place: every thread reads all of
// its inputs, the workgroup synchronises, then every thread writes.  A thread holds
// at most EMAX complex values; the host checks that ceil((N/R) / NSUB) <= ceil(EMAX / R)
// for every radix of the plan.
//
// Forward (INV = false) uses exp(-i ...), inverse exp(+i ...); neither scales.
#pragma once
#include <hip/hip_runtime.h>

namespace afno {

constexpr int kMaxPasses = 16;

struct Radices {
  int n;                 // transform length
  int count;             // number of passes
  int r[kMaxPasses];     // radix of each pass, product = n
};

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
  return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cscale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }
// multiply by -i (forward) or +i (inverse)
template <bool INV>
__device__ __forceinline__ float2 mul_mi(float2 a) {
  return INV ? make_float2(-a.y, a.x) : make_float2(a.y, -a.x);
}

// R-point DFT in registers, X_m = sum_t v_t exp(-+2 pi i t m / R).
template <int R, bool INV>
__device__ __forceinline__ void dft_small(float2 (&v)[R]);

template <>
__device__ __forceinline__ void dft_small<2, false>(float2 (&v)[2]) {
  float2 a = v[0], b = v[1];
  v[0] = cadd(a, b); v[1] = csub(a, b);
}
template <>
__device__ __forceinline__ void dft_small<2, true>(float2 (&v)[2]) {
  float2 a = v[0], b = v[1];
  v[0] = cadd(a, b); v[1] = csub(a, b);
}

template <int R, bool INV>
__device__ __forceinline__ void dft3(float2 (&v)[R]) {
  // X1 = a - (b + c)/2 -+ i (sqrt3/2)(b - c),  X2 = a - (b + c)/2 +- i (sqrt3/2)(b - c)
  const float s3 = 0.866025403784438647f;
  float2 a = v[0], b = v[1], c = v[2];
  float2 t1 = cadd(b, c);
  float2 t2 = make_float2(a.x - 0.5f * t1.x, a.y - 0.5f * t1.y);
  float2 t3 = mul_mi<INV>(cscale(csub(b, c), s3));
  v[0] = cadd(a, t1);
  v[1] = cadd(t2, t3);
  v[2] = csub(t2, t3);
}
template <> __device__ __forceinline__ void dft_small<3, false>(float2 (&v)[3]) { dft3<3, false>(v); }
template <> __device__ __forceinline__ void dft_small<3, true>(float2 (&v)[3]) { dft3<3, true>(v); }

template <int R, bool INV>
__device__ __forceinline__ void dft4(float2 (&v)[R]) {
  float2 s02 = cadd(v[0], v[2]), d02 = csub(v[0], v[2]);
  float2 s13 = cadd(v[1], v[3]), d13 = mul_mi<INV>(csub(v[1], v[3]));
  v[0] = cadd(s02, s13);
  v[2] = csub(s02, s13);
  v[1] = cadd(d02, d13);
  v[3] = csub(d02, d13);
}
template <> __device__ __forceinline__ void dft_small<4, false>(float2 (&v)[4]) { dft4<4, false>(v); }
template <> __device__ __forceinline__ void dft_small<4, true>(float2 (&v)[4]) { dft4<4, true>(v); }

template <int R, bool INV>
__device__ __forceinline__ void dft5(float2 (&v)[R]) {
  // cos and sin of 2 pi / 5 and 4 pi / 5
  const float c1 = 0.309016994374947424f, c2 = -0.809016994374947424f;
  const float s1 = 0.951056516295153572f, s2 = 0.587785252292473129f;
  float2 a0 = v[0];
  float2 b1 = cadd(v[1], v[4]), d1 = csub(v[1], v[4]);
  float2 b2 = cadd(v[2], v[3]), d2 = csub(v[2], v[3]);
  float2 r1 = make_float2(a0.x + c1 * b1.x + c2 * b2.x, a0.y + c1 * b1.y + c2 * b2.y);
  float2 r2 = make_float2(a0.x + c2 * b1.x + c1 * b2.x, a0.y + c2 * b1.y + c1 * b2.y);
  float2 i1 = mul_mi<INV>(make_float2(s1 * d1.x + s2 * d2.x, s1 * d1.y + s2 * d2.y));
  float2 i2 = mul_mi<INV>(make_float2(s2 * d1.x - s1 * d2.x, s2 * d1.y - s1 * d2.y));
  v[0] = cadd(a0, cadd(b1, b2));
  v[1] = cadd(r1, i1);
  v[4] = csub(r1, i1);
  v[2] = cadd(r2, i2);
  v[3] = csub(r2, i2);
}
template <> __device__ __forceinline__ void dft_small<5, false>(float2 (&v)[5]) { dft5<5, false>(v); }
template <> __device__ __forceinline__ void dft_small<5, true>(float2 (&v)[5]) { dft5<5, true>(v); }

// One in-place Stockham pass of radix R.  tw[m] = exp(-2 pi i m / N), m in [0, N).
template <int R, int EMAX, bool INV>
__device__ __forceinline__ void fft_pass(float2* buf, int ld, int N, int L, int sig, int sub,
                                         int nsub, const float2* tw) {
  constexpr int BMAX = (EMAX + R - 1) / R;
  const int nbf = N / R;
  const int twstep = N / (L * R);
  float2 v[BMAX][R];
#pragma unroll
  for (int q = 0; q < BMAX; ++q) {
    const int j = sub + q * nsub;
    if (j < nbf) {
#pragma unroll
      for (int t = 0; t < R; ++t) v[q][t] = buf[(j + t * nbf) * ld + sig];
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < BMAX; ++q) {
    const int j = sub + q * nsub;
    if (j < nbf) {
      const int k = j % L;
#pragma unroll
      for (int t = 1; t < R; ++t) {
        float2 w = tw[t * k * twstep];
        if (INV) w.y = -w.y;
        v[q][t] = cmul(v[q][t], w);
      }
      dft_small<R, INV>(v[q]);
      const int base = (j - k) * R + k;
#pragma unroll
      for (int t = 0; t < R; ++t) buf[(base + t * L) * ld + sig] = v[q][t];
    }
  }
  __syncthreads();
}

// Full transform: all passes of `rd` on the NSIG signals of buf.  Must be called by
// every thread of the workgroup (it synchronises).
template <int EMAX, bool INV>
__device__ void fft_lds(float2* buf, int ld, const Radices& rd, int sig, int sub, int nsub,
                        const float2* tw) {
  int L = 1;
  for (int p = 0; p < rd.count; ++p) {
    const int R = rd.r[p];
    switch (R) {
      case 2: fft_pass<2, EMAX, INV>(buf, ld, rd.n, L, sig, sub, nsub, tw); break;
      case 3: fft_pass<3, EMAX, INV>(buf, ld, rd.n, L, sig, sub, nsub, tw); break;
      case 4: fft_pass<4, EMAX, INV>(buf, ld, rd.n, L, sig, sub, nsub, tw); break;
      default: fft_pass<5, EMAX, INV>(buf, ld, rd.n, L, sig, sub, nsub, tw); break;
    }
    L *= R;
  }
}

// tw[m] = exp(-2 pi i m / N) for m in [0, N), from double-precision sincospi, rounded
// once to float.  Synchronises the workgroup.
__device__ __forceinline__ void make_twiddles(float2* tw, int N) {
  for (int m = threadIdx.x; m < N; m += blockDim.x) {
    double s, c;
    sincospi(2.0 * (double)m / (double)N, &s, &c);
    tw[m] = make_float2((float)c, (float)(-s));
  }
  __syncthreads();
}

}  // namespace afno
