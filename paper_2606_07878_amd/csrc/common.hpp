// common.hpp - element types, conversions and the CDNA4 MFMA step used by
// every kernel of the compactor library (gfx950 only).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace still {

typedef _Float16 f16;
typedef f16 half8 __attribute__((ext_vector_type(8)));
typedef f16 half4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// bfloat16 held as raw bits (I/O type of the bf16 mode).
struct bf16 {
  uint16_t x;
};

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(f16 v) { return (float)v; }
__device__ __forceinline__ float to_f32(bf16 v) { return __uint_as_float((uint32_t)v.x << 16); }

// float -> bfloat16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ bf16 f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  bf16 r;
  if ((u & 0x7fffffffu) > 0x7f800000u) {
    r.x = (uint16_t)((u >> 16) | 0x40u);
  } else {
    u += 0x7fffu + ((u >> 16) & 1u);
    r.x = (uint16_t)(u >> 16);
  }
  return r;
}

template <class T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ f16 from_f32<f16>(float v) { return (f16)v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return f32_to_bf16(v); }

// ---------------------------------------------------------------------------
// MFMA step on 32x32 output tiles.  A "fragment" is the 16 bytes one lane
// contributes per step: lanes 0-31 hold k in [0,E), lanes 32-63 k in [E,2E)
// of a 2E-wide k chunk, for row (A) or column (B) lane%32.
//  * f16: one v_mfma_f32_32x32x16_f16 (E = 8, k chunk 16).
//  * f32: four v_mfma_f32_32x32x2_f32, component s of both operands forming
//    the k pair (s, E+s); any fixed pairing sums every k exactly once.
// Output layout (both): lane l, register j -> row 8*(j/4) + 4*(l/32) + j%4,
// column l%32.
// ---------------------------------------------------------------------------
template <class CT> struct Mma;

template <> struct Mma<f16> {
  typedef half8 frag;
  static constexpr int E = 8;
  static __device__ __forceinline__ void mma(f32x16& c, const frag& a, const frag& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mma<float> {
  typedef f32x4 frag;
  static constexpr int E = 4;
  static __device__ __forceinline__ void mma(f32x16& c, const frag& a, const frag& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0], b[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1], b[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[2], b[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[3], b[3], c, 0, 0, 0);
  }
};

// Load E consecutive elements of type T (16-byte aligned run) as a CT fragment.
template <class CT, class T> struct VecLoad;

template <> struct VecLoad<f16, f16> {
  static __device__ __forceinline__ half8 load(const f16* p) { return *(const half8*)p; }
};
template <> struct VecLoad<f16, bf16> {
  static __device__ __forceinline__ half8 load(const bf16* p) {
    uint4 u = *(const uint4*)p;
    half8 r;
    uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r[2 * i] = (f16)__uint_as_float(w[i] << 16);
      r[2 * i + 1] = (f16)__uint_as_float(w[i] & 0xffff0000u);
    }
    return r;
  }
};
template <> struct VecLoad<f16, float> {
  static __device__ __forceinline__ half8 load(const float* p) {
    f32x4 a = *(const f32x4*)p;
    f32x4 b = *(const f32x4*)(p + 4);
    half8 r;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      r[i] = (f16)a[i];
      r[4 + i] = (f16)b[i];
    }
    return r;
  }
};
template <> struct VecLoad<float, float> {
  static __device__ __forceinline__ f32x4 load(const float* p) { return *(const f32x4*)p; }
};

// ---------------------------------------------------------------------------
// Fragment-tiled layouts of the fp16 cross-attention operands.  One MFMA
// operand fragment (64 lanes x 8 halfs: 32 rows x 16 contraction indices) is
// 1 KB of contiguous memory, so each fragment load of a wave is one fully
// coalesced 1 KB read.  Lane l of a fragment holds row l % 32 and contraction
// indices 8 * (l / 32) + [0, 8) of the fragment's 16.
//   k (projected keys) of KV head h, cross head c (hc = h * nc + c), key n,
//   storage position x (npad keys per head, a multiple of 256):
//     [hc][n / 32][x / 16][lane = n % 32 + 32 * ((x / 8) % 2)][x % 8]
//   Position x of a width step of 16 need not hold width x: the key
//   projection stores its accumulator registers in place, so the query and
//   the key side agree on one permutation of the 16 widths of each step (the
//   contraction over the step does not depend on the order).
//   X^T of KV head h, feature f, key n:
//     [h][f / 32][n / 16][lane = f % 32 + 32 * ((n / 8) % 2)][n % 8]
// ---------------------------------------------------------------------------
__host__ __device__ __forceinline__ long ktile_off(long hc, long n, long x, long npad, long dc) {
  return ((((hc * (npad >> 5) + (n >> 5)) * (dc >> 4) + (x >> 4)) << 9) + (((n & 31) + (((x >> 3) & 1) << 5)) << 3) +
          (x & 7));
}
__host__ __device__ __forceinline__ long xtile_off(long h, long f, long n, long npad, long d2) {
  return ((((h * (d2 >> 5) + (f >> 5)) * (npad >> 4) + (n >> 4)) << 9) + (((f & 31) + (((n >> 3) & 1) << 5)) << 3) +
          (n & 7));
}

// Keys whose fp16-path logit lies within this many log2 units of their row's
// maximum are candidates for the exact-logit refinement of cross-attention.
constexpr float REFINE_MARGIN = 10.f;

template <class CT> __device__ __forceinline__ typename Mma<CT>::frag zero_frag() {
  typename Mma<CT>::frag z;
#pragma unroll
  for (int i = 0; i < Mma<CT>::E; ++i) z[i] = (CT)0;
  return z;
}

// (cos, sin) of the RoPE angle pos * inv.  The angle is formed in fp64 and
// reduced there to x = angle - q pi/2 with |x| <= pi/4 (pi/2 in two parts);
// sin x and cos x come from their Taylor series in fp32 (the first omitted
// terms are below 3e-8 on |x| <= pi/4), then the quadrant q mod 4 picks the
// signs and the order.
__device__ __forceinline__ float2 rope_cs(double pos, double inv) {
  const double ang = pos * inv;
  const double q = rint(ang * 0.63661977236758134);
  double r = fma(-q, 1.5707963267948966, ang);
  r = fma(-q, 6.123233995736766e-17, r);
  const float x = (float)r, x2 = x * x;
  const float s = fmaf(x * x2, -1.f / 6 + x2 * (1.f / 120 + x2 * (-1.f / 5040 + x2 * (1.f / 362880))), x);
  const float c = fmaf(x2, -0.5f + x2 * (1.f / 24 + x2 * (-1.f / 720 + x2 * (1.f / 40320))), 1.f);
  // quadrant k = q mod 4 (exact in fp64); branch-free: odd k swaps the two
  // values, k in {1, 2} negates the cosine, k in {2, 3} the sine
  const int k = (int)(q - 4.0 * floor(q * 0.25));
  const bool swap = k & 1;
  const uint32_t nc = (uint32_t)((k + 1) & 2) << 30, ns = (uint32_t)(k & 2) << 30;
  return make_float2(__uint_as_float(__float_as_uint(swap ? s : c) ^ nc),
                     __uint_as_float(__float_as_uint(swap ? c : s) ^ ns));
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// Swizzle of the 16-byte unit index within an LDS row of U units.  Rows are
// read 16 at a time at one unit (MFMA fragments) and written U units at a
// time per row (staging); the mask is a bijection on the row bits that decide
// the bank group under both 128-byte and 256-byte LDS access phases.
template <int U> __device__ __forceinline__ int lds_swz(int r);
template <> __device__ __forceinline__ int lds_swz<4>(int r) { return (((r >> 1) ^ (r >> 3)) & 1) | ((r >> 1) & 2); }
template <> __device__ __forceinline__ int lds_swz<8>(int r) { return ((r ^ (r >> 3)) & 1) | (r & 6); }

}  // namespace still
