// kernel_common.h -- storage types, MFMA operand helpers and the cutoff test shared by
// the generic and the size-specialised kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace afno {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Store;
template <> struct Store<float> {
  static constexpr int kVec = 4;  // elements per 16-byte vector
  __device__ static float to(float v) { return v; }
};
template <> struct Store<bf16> {
  static constexpr int kVec = 8;
  __device__ static bf16 to(float v) { return (bf16)v; }  // round to nearest even
};
__device__ __forceinline__ float ld_f(const float* p) { return *p; }
__device__ __forceinline__ float ld_f(const bf16* p) { return (float)*p; }

// 16-byte vector of T viewed as floats / bf16
union V16 {
  uint4 u;
  float f[4];
  bf16 h[8];
};

// One complex value (re, im) in storage type T.
__device__ __forceinline__ float2 ld_c(const float* p) { return *reinterpret_cast<const float2*>(p); }
__device__ __forceinline__ float2 ld_c(const bf16* p) {
  union { uint32_t u; bf16 h[2]; } w;
  w.u = *reinterpret_cast<const uint32_t*>(p);
  return make_float2((float)w.h[0], (float)w.h[1]);
}
__device__ __forceinline__ void st_c(float* p, float2 v) { *reinterpret_cast<float2*>(p) = v; }
__device__ __forceinline__ void st_c(bf16* p, float2 v) {
  union { uint32_t u; bf16 h[2]; } w;
  w.h[0] = (bf16)v.x;
  w.h[1] = (bf16)v.y;
  *reinterpret_cast<uint32_t*>(p) = w.u;
}
// Two complex values (4 T) in one access.
__device__ __forceinline__ float4 ld_c2(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ float4 ld_c2(const bf16* p) {
  union { uint2 u; bf16 h[4]; } w;
  w.u = *reinterpret_cast<const uint2*>(p);
  return make_float4((float)w.h[0], (float)w.h[1], (float)w.h[2], (float)w.h[3]);
}
__device__ __forceinline__ void st_c2(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void st_c2(bf16* p, float4 v) {
  union { uint2 u; bf16 h[4]; } w;
  w.h[0] = (bf16)v.x; w.h[1] = (bf16)v.y; w.h[2] = (bf16)v.z; w.h[3] = (bf16)v.w;
  *reinterpret_cast<uint2*>(p) = w.u;
}

// MFMA operand types per storage dtype.
template <typename T> struct Mma;

// bf16: v_mfma_f32_16x16x32_bf16.  Lane l: A row l%16, k 8(l/16)..+7; B column l%16,
// k 8(l/16)..+7; D column l%16, rows 4(l/16)..+3.
template <> struct Mma<bf16> {
  static constexpr int kK = 32;
  typedef bf16x8 Frag;
  // A fragment: 8 consecutive bf16 of an LDS row.
  __device__ static Frag load_a(const bf16* row, int kbase, int lane) {
    return *reinterpret_cast<const bf16x8*>(row + kbase + 8 * (lane >> 4));
  }
  // B fragment of the real-ified complex weight at output column nu = 2j + sg:
  //   Wexp[2i + rho][2j + sg] = (Wr, -Wi ; Wi, Wr)[rho][sg]
  // w points at the block's [n_in][n_out][2] complex weights.  Each dword holds one
  // complex weight (lo = re, hi = im); sg = 0 needs (re, -im), sg = 1 needs (im, re):
  // a byte permutation and a sign flip with per-lane constants, so no lane diverges
  // and all four loads are in flight before the first use.
  __device__ static Frag load_b(const bf16* w, int n_out, int kbase, int j, int sg, int lane) {
    const int i0 = (kbase >> 1) + 4 * (lane >> 4);
    const uint32_t* wp = reinterpret_cast<const uint32_t*>(w) + (int64_t)i0 * n_out + j;
    uint32_t v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = wp[(int64_t)q * n_out];
    const uint32_t sel = sg ? 0x01000302u : 0x03020100u;
    const uint32_t flip = sg ? 0u : 0x80000000u;
    union { uint32_t u[4]; Frag f; } r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r.u[q] = __builtin_amdgcn_perm(v[q], v[q], sel) ^ flip;
    return r.f;
  }
  __device__ static f32x4 mma(Frag a, Frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

// fp32: v_mfma_f32_16x16x4_f32.  Lane l: A row l%16, k l/16; B column l%16, k l/16.
template <> struct Mma<float> {
  static constexpr int kK = 4;
  typedef float Frag;
  __device__ static Frag load_a(const float* row, int kbase, int lane) {
    return row[kbase + (lane >> 4)];
  }
  // Wexp[2i + rho][2j + sg]: component rho ^ sg of w[i][j], negated for rho = 1, sg = 0
  // (per-lane constants, no divergence).
  __device__ static Frag load_b(const float* w, int n_out, int kbase, int j, int sg, int lane) {
    const int kap = kbase + (lane >> 4);
    const int i = kap >> 1, rho = kap & 1;
    const float v = w[((int64_t)i * n_out + j) * 2 + (rho ^ sg)];
    const uint32_t flip = (uint32_t)(rho & (sg ^ 1)) << 31;
    return __uint_as_float(__float_as_uint(v) ^ flip);
  }
  __device__ static f32x4 mma(Frag a, Frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
};

// One lane's B fragment of the real-ified weight in storage form: four dwords (eight bf16)
// for the bf16 MFMA, one float for the fp32 MFMA.
template <typename T> struct FragWord;
template <> struct FragWord<bf16> {
  typedef uint4 type;
  __device__ static type make(const bf16* w, int n_out, int kbase, int j, int sg, int lane) {
    union { Mma<bf16>::Frag f; uint4 u; } r;
    r.f = Mma<bf16>::load_b(w, n_out, kbase, j, sg, lane);
    return r.u;
  }
};
template <> struct FragWord<float> {
  typedef uint32_t type;
  __device__ static type make(const float* w, int n_out, int kbase, int j, int sg, int lane) {
    return __float_as_uint(Mma<float>::load_b(w, n_out, kbase, j, sg, lane));
  }
};

// Fragment-ordered weights of one block: index ((layer * KSTEPS + s) * NT16 + t) * 64 + lane,
// k-step s of Mma<T>::kK real inputs, n-tile t of 16 real output columns.
template <typename T>
__host__ __device__ constexpr int64_t frag_words_per_block(int bs) {
  return (int64_t)2 * (2 * bs / (sizeof(T) == 2 ? 32 : 4)) * (2 * bs / 16) * 64;
}

// hard mode cutoff along H: row kh kept when |signed kh| < kept_h
__device__ __forceinline__ bool row_kept(int r, int H, int kept_h) {
  if (r >= H) return false;
  int s = (r <= H / 2) ? r : r - H;
  s = s < 0 ? -s : s;
  return s < kept_h;
}

// the rows the cutoff keeps, compacted (2 kept_h - 1 of them, kept_h <= H / 2): kept row k'
// -> spectral row (0, 1, .., kept_h - 1, then H - kept_h + 1, .., H - 1), and back (-1: a row
// the cutoff drops)
__host__ __device__ __forceinline__ int kept_row(int kp, int H, int kept_h) {
  return kp < kept_h ? kp : H - (2 * kept_h - 1 - kp);
}
__host__ __device__ __forceinline__ int kept_index(int h, int H, int kept_h) {
  if (h < kept_h) return h;
  if (h > H - kept_h) return h - (H - (2 * kept_h - 1));
  return -1;
}

// S(v) = v - lam (v > lam), v + lam (v < -lam), else 0, written as v - clamp(v, -lam, lam)
// (exactly 0 inside the band, exact shifts outside it)
__device__ __forceinline__ float softshrink(float v, float lam) {
  return v - __builtin_amdgcn_fmed3f(v, -lam, lam);
}

// cache-policy operand of the buffer intrinsics on gfx950: the non-temporal (streaming) hint
constexpr int kNonTemporal = 2;

// Raw buffer access: a per-workgroup base in a scalar resource descriptor, a 32-bit
// per-lane byte offset and a wave-uniform byte offset, so addressing costs no 64-bit
// vector arithmetic.  Accesses beyond `bytes` read 0 and do not write.
struct Buf {
  __amdgpu_buffer_rsrc_t r;
  __device__ __forceinline__ Buf(const void* base, uint32_t bytes)
      : r(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                            0x00020000)) {}
  template <int AUX = 0>
  __device__ __forceinline__ uint32_t ld32(uint32_t voff, uint32_t soff) const {
    return __builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, AUX);
  }
  __device__ __forceinline__ void st32(uint32_t v, uint32_t voff, uint32_t soff) const {
    __builtin_amdgcn_raw_buffer_store_b32(v, r, voff, soff, 0);
  }
  __device__ __forceinline__ uint2 ld64(uint32_t voff, uint32_t soff) const {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    return make_uint2(v[0], v[1]);
  }
  __device__ __forceinline__ void st64(uint2 v, uint32_t voff, uint32_t soff) const {
    typedef uint32_t u2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(u2{v.x, v.y}, r, voff, soff, 0);
  }
  template <int AUX = 0>
  __device__ __forceinline__ void st128(uint4 v, uint32_t voff, uint32_t soff) const {
    typedef uint32_t u4 __attribute__((ext_vector_type(4)));
    __builtin_amdgcn_raw_buffer_store_b128(u4{v.x, v.y, v.z, v.w}, r, voff, soff, AUX);
  }
};
__device__ __forceinline__ uint32_t buf_bytes(uint64_t n) {
  return n >= 0xffffffffull ? 0xffffffffu : (uint32_t)n;
}
// one complex value from / to 32 bits of storage
__device__ __forceinline__ float2 unpack_c(uint32_t v, const bf16*) {
  return make_float2(__uint_as_float(v << 16), __uint_as_float(v & 0xffff0000u));
}
__device__ __forceinline__ uint32_t pack_c(float2 z, const bf16*) {
  union { uint32_t u; bf16 h[2]; } w;
  w.h[0] = (bf16)z.x;
  w.h[1] = (bf16)z.y;
  return w.u;
}

}  // namespace afno
