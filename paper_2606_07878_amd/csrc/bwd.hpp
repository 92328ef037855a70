// bwd.hpp - kernels of the compactor's backward pass (fp32): a strided
// batched MFMA GEMM that takes either operand layout, and the row-wise
// forward/backward steps (RMSNorm, QK-norm with RoPE, softmax, SwiGLU/GELU,
// bias column sums, RoPE-fix staging).
//
// The backward pass keeps every intermediate of the forward pass it needs
// (the attention probabilities included), so each step of the chain rule is
// a GEMM or a row-wise kernel over saved tensors.
#pragma once
#include "common.hpp"

namespace still {

// ---------------------------------------------------------------------------
// Strided batched GEMM on v_mfma_f32_32x32x2_f32:
//   C[b](m, n) = alpha * sum_k A[b](m, k) B[b](n, k)   (+ C[b](m, n) if accumulate)
// with A[b](m, k) = A[b1 * sa1 + b2 * sa2 + m * am + k * ak], one of am, ak
// equal to 1 (likewise B), b = b1 * nb2 + b2 the batch index, C row-major
// with leading dimension ldc.  64 x 64 tiles, k stages of 32 (the next
// stage loaded into registers during the current one's MFMAs), four waves
// each owning one 32 x 32 MFMA tile; operands staged in LDS as [row][k].
// ---------------------------------------------------------------------------
struct SgemmArgs {
  const float* A;
  const float* B;
  float* C;
  long am, ak, sa1, sa2;
  long bn, bk, sb1, sb2;
  long ldc, sc1, sc2;
  int M, N, K, nb2;
  float alpha;
  int accumulate;
  const float* bias;   // per output column n, added to alpha * acc (NULL = none)
  // split-K (one batch only): ksplit > 0 makes grid row z sum k in
  // [z ksplit, (z + 1) ksplit) and store its raw sums (no alpha, bias or
  // accumulate) into part[z][m][n] (float for the fp32 kernel, double for the
  // fp64 one); ksplit_reduce_kernel then forms C in a fixed order
  int ksplit;
  void* part;
};

// Load this thread's part of a 64 x 16 tile (rows r0.., k k0..) of a
// strided operand (k < K, rows < R; zeros outside) into registers, and store
// it into LDS [64][LK].  K-contiguous sources: 4 consecutive k per thread;
// row-contiguous sources: 4 consecutive rows; edges fall back to scalar loads.
template <bool KCONT>
__device__ __forceinline__ void sgemm_load(const float* __restrict__ X, long xr, long xk, int R, int K, int r0,
                                           int k0, float (&v)[4]) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) v[i] = 0.f;
  if (KCONT) {
    const int r = tid >> 2, k = (tid & 3) * 4;
    const int gr = r0 + r, gk = k0 + k;
    if (gr < R) {
      const float* p = X + gr * xr + gk;
      if (gk + 3 < K && ((uintptr_t)p & 15u) == 0) {
        const f32x4 q = *(const f32x4*)p;
        v[0] = q[0];
        v[1] = q[1];
        v[2] = q[2];
        v[3] = q[3];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (gk + i < K) v[i] = p[i];
      }
    }
  } else {
    const int k = tid >> 4, r = (tid & 15) * 4;
    const int gr = r0 + r, gk = k0 + k;
    if (gk < K) {
      const float* p = X + gk * xk + gr;
      if (gr + 3 < R && ((uintptr_t)p & 15u) == 0) {
        const f32x4 q = *(const f32x4*)p;
        v[0] = q[0];
        v[1] = q[1];
        v[2] = q[2];
        v[3] = q[3];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (gr + i < R) v[i] = p[i];
      }
    }
  }
}
template <bool KCONT>
__device__ __forceinline__ void sgemm_store(const float (&v)[4], float* __restrict__ S, int LK) {
  const int tid = threadIdx.x;
  if (KCONT) {
    const int r = tid >> 2, k = (tid & 3) * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) S[r * LK + k + i] = v[i];
  } else {
    const int k = tid >> 4, r = (tid & 15) * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) S[(r + i) * LK + k] = v[i];
  }
}

template <bool AK, bool BK>
__global__ __launch_bounds__(256) void sgemm_kernel(SgemmArgs g) {
  constexpr int T = 64, KS = 32, LK = KS + 4;   // k stage = two 16-wide halves
  __shared__ __attribute__((aligned(16))) float As[T * LK];
  __shared__ __attribute__((aligned(16))) float Bs[T * LK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1, l32 = lane & 31, lg = lane >> 5;
  const int m0 = blockIdx.y * T, n0 = blockIdx.x * T;
  const int kz = g.ksplit ? (int)blockIdx.z : 0;
  const int b = g.ksplit ? 0 : (int)blockIdx.z, b1 = b / g.nb2, b2 = b - b1 * g.nb2;
  const int kbeg = kz * g.ksplit, kend = g.ksplit ? min(g.K, kbeg + g.ksplit) : g.K;
  const float* A = g.A + b1 * g.sa1 + b2 * g.sa2;
  const float* B = g.B + b1 * g.sb1 + b2 * g.sb2;
  f32x16 acc = zero16();
  // the next k stage is loaded into registers while the current one's MFMAs run
  float ra[2][4], rb[2][4];
  auto load = [&](int k0) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      sgemm_load<AK>(A, g.am, g.ak, g.M, kend, m0, k0 + 16 * h, ra[h]);
      sgemm_load<BK>(B, g.bn, g.bk, g.N, kend, n0, k0 + 16 * h, rb[h]);
    }
  };
  load(kbeg);
  for (int k0 = kbeg; k0 < kend; k0 += KS) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      sgemm_store<AK>(ra[h], As + 16 * h, LK);
      sgemm_store<BK>(rb[h], Bs + 16 * h, LK);
    }
    __syncthreads();
    if (k0 + KS < kend) load(k0 + KS);
#pragma unroll
    for (int kc = 0; kc < KS; kc += 8) {
      const f32x4 af = *(const f32x4*)&As[(wm * 32 + l32) * LK + kc + 4 * lg];
      const f32x4 bf = *(const f32x4*)&Bs[(wn * 32 + l32) * LK + kc + 4 * lg];
      Mma<float>::mma(acc, af, bf);
    }
    __syncthreads();
  }
  if (g.ksplit) {
    float* P = (float*)g.part + (long)kz * g.M * g.N;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int m = m0 + wm * 32 + 8 * (j >> 2) + 4 * lg + (j & 3);
      const int n = n0 + wn * 32 + l32;
      if (m < g.M && n < g.N) P[(long)m * g.N + n] = acc[j];
    }
    return;
  }
  float* C = g.C + b1 * g.sc1 + b2 * g.sc2;
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    const int m = m0 + wm * 32 + 8 * (j >> 2) + 4 * lg + (j & 3);
    const int n = n0 + wn * 32 + l32;
    if (m < g.M && n < g.N) {
      float* c = C + (long)m * g.ldc + n;
      const float v = g.alpha * acc[j] + (g.bias ? g.bias[n] : 0.f);
      *c = g.accumulate ? *c + v : v;
    }
  }
}

// The same product in fp64 (fp64 MFMA, v_mfma_f64_16x16x4_f64), for the
// steps whose rounding the d_l logit scale amplifies: the cross-attention
// logit path and its adjoint.  Operands and result may be float or double.
// 64 x 64 tiles staged through LDS in k chunks of 32; wave (wm, wn) owns the
// 32 x 32 quadrant (wm, wn) as 2 x 2 MFMA tiles of 16 x 16.  Operand layout
// of the MFMA: lane l supplies A[l % 16][l / 16] and B[l / 16][l % 16] of
// the 16 x 4 and 4 x 16 step; the result is C[l / 16 + 4 v][l % 16] in
// register pair v of lane l (checked with a probe on the hardware).
typedef double f64x4 __attribute__((ext_vector_type(4)));

template <bool AK, bool BK, class TA, class TB, class TC>
__global__ __launch_bounds__(256) void dgemm_kernel(SgemmArgs g, const TA* __restrict__ A0, const TB* __restrict__ B0,
                                                    TC* __restrict__ C0) {
  constexpr int T = 64, KS = 32, PER = T * KS / 256;
  __shared__ double As[KS][T + 1];
  __shared__ double Bs[KS][T + 1];
  const int tid = threadIdx.x;
  const int m0 = blockIdx.y * T, n0 = blockIdx.x * T;
  const int kz = g.ksplit ? (int)blockIdx.z : 0;
  const int b = g.ksplit ? 0 : (int)blockIdx.z, b1 = b / g.nb2, b2 = b - b1 * g.nb2;
  const int kbeg = kz * g.ksplit, kend = g.ksplit ? min(g.K, kbeg + g.ksplit) : g.K;
  const TA* A = A0 + b1 * g.sa1 + b2 * g.sa2;
  const TB* B = B0 + b1 * g.sb1 + b2 * g.sb2;
  const int lane = tid & 63, wave = tid >> 6, wm = wave >> 1, wn = wave & 1;
  const int li = lane & 15, lk = lane >> 4;
  f64x4 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f64x4{0.0, 0.0, 0.0, 0.0};
  // the next k chunk's operands are loaded into registers while the current
  // chunk's MFMAs run (consecutive threads walk each operand's contiguous
  // dimension); they stay in their own type until the LDS store, so that a
  // conversion does not wait for the loads in front of the MFMAs
  TA ra[PER];
  TB rb[PER];
  auto load = [&](int k0) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = tid + 256 * u;
      const int r = AK ? e / KS : e % T, k = AK ? e % KS : e / T;
      const int gr = m0 + r, gk = k0 + k;
      ra[u] = (gr < g.M && gk < kend) ? A[gr * g.am + gk * g.ak] : (TA)0;
    }
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = tid + 256 * u;
      const int r = BK ? e / KS : e % T, k = BK ? e % KS : e / T;
      const int gr = n0 + r, gk = k0 + k;
      rb[u] = (gr < g.N && gk < kend) ? B[gr * g.bn + gk * g.bk] : (TB)0;
    }
  };
  load(kbeg);
  for (int k0 = kbeg; k0 < kend; k0 += KS) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int e = tid + 256 * u;
      As[AK ? e % KS : e / T][AK ? e / KS : e % T] = (double)ra[u];
      Bs[BK ? e % KS : e / T][BK ? e / KS : e % T] = (double)rb[u];
    }
    __syncthreads();
    if (k0 + KS < kend) load(k0 + KS);
#pragma unroll
    for (int k = 0; k < KS; k += 4) {
      double av[2], bv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) av[i] = As[k + lk][32 * wm + 16 * i + li];
#pragma unroll
      for (int j = 0; j < 2; ++j) bv[j] = Bs[k + lk][32 * wn + 16 * j + li];
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f64_16x16x4f64(av[i], bv[j], acc[i][j], 0, 0, 0);
    }
    __syncthreads();
  }
  if (g.ksplit) {
    double* P = (double*)g.part + (long)kz * g.M * g.N;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int m = m0 + 32 * wm + 16 * i + lk + 4 * v, n = n0 + 32 * wn + 16 * j + li;
          if (m < g.M && n < g.N) P[(long)m * g.N + n] = acc[i][j][v];
        }
    return;
  }
  TC* C = C0 + b1 * g.sc1 + b2 * g.sc2;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int m = m0 + 32 * wm + 16 * i + lk + 4 * v, n = n0 + 32 * wn + 16 * j + li;
        if (m >= g.M || n >= g.N) continue;
        TC* c = C + (long)m * g.ldc + n;
        const double val = (double)g.alpha * acc[i][j][v] + (g.bias ? (double)g.bias[n] : 0.0);
        *c = (TC)(g.accumulate ? (double)*c + val : val);
      }
}

// Split-K epilogue: C(m, n) = alpha * sum_z part[z][m][n] (+ bias[n])
// (+ C(m, n) if accumulate), the splits summed in order (deterministic).
template <class TP, class TC>
__global__ void ksplit_reduce_kernel(const TP* __restrict__ part, int splits, int M, int N, TC* __restrict__ C,
                                     long ldc, double alpha, const float* __restrict__ bias, int accumulate) {
  const long total = (long)M * N;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    double s = 0.0;
    for (int z = 0; z < splits; ++z) s += (double)part[z * total + i];
    const long m = i / N, n = i - m * N;
    double v = alpha * s + (bias ? (double)bias[n] : 0.0);
    TC* c = C + m * ldc + n;
    if (accumulate) v += (double)*c;
    *c = (TC)v;
  }
}

// ---------------------------------------------------------------------------
// Row-wise steps (one wave per row unless stated)
// ---------------------------------------------------------------------------

// Y = X r, r = 1 / sqrt(mean(X^2) + eps) (saved per row)
static __global__ __launch_bounds__(256) void b_rms_fwd_kernel(const float* __restrict__ X, float* __restrict__ Y,
                                                               float* __restrict__ r, long rows, int D, float eps) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* x = X + row * D;
  double ss = 0.0;
  for (int j = lane; j < D; j += 64) ss += (double)x[j] * x[j];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  const float rr = (float)(1.0 / sqrt(ss / D + (double)eps));
  for (int j = lane; j < D; j += 64) Y[row * D + j] = x[j] * rr;
  if (lane == 0) r[row] = rr;
}

// dX += r dY - (r^3 / D) X (X . dY)
static __global__ __launch_bounds__(256) void b_rms_bwd_kernel(const float* __restrict__ X, const float* __restrict__ dY,
                                                               const float* __restrict__ r, float* __restrict__ dX,
                                                               long rows, int D) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* x = X + row * D;
  const float* dy = dY + row * D;
  double dot = 0.0;
  for (int j = lane; j < D; j += 64) dot += (double)x[j] * dy[j];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) dot += __shfl_xor(dot, o);
  const float rr = r[row];
  const float c = (float)((double)rr * rr * rr / D * dot);
  for (int j = lane; j < D; j += 64) dX[row * D + j] += rr * dy[j] - c * x[j];
}

// Per (row, head) slice of width w: y = RoPE(x / max(||x||, eps), p) with
// the slice's norm saved (norm = 1 and no division when NORM is off; no
// rotation when pos is NULL).  The row's position is pos[row % pmod], the
// pair (j, j + w/2) angle pos * invf[j] (fp64).  One wave per slice.
template <bool NORM, class T = float>
__global__ __launch_bounds__(256) void b_nrope_fwd_kernel(const T* __restrict__ X, T* __restrict__ Y,
                                                          T* __restrict__ nrm, long rows, int nh, int w,
                                                          const double* __restrict__ pos, long pmod,
                                                          const double* __restrict__ invf, float eps) {
  const long s = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (s >= rows * nh) return;
  const long row = s / nh;
  const int c = (int)(s - row * nh);
  const T* x = X + row * ((long)nh * w) + (long)c * w;
  T* y = Y + row * ((long)nh * w) + (long)c * w;
  double inv = 1.0;
  if (NORM) {
    double ss = 0.0;
    for (int j = lane; j < w; j += 64) ss += (double)x[j] * x[j];
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    const double n = sqrt(ss);
    inv = 1.0 / fmax(n, (double)eps);
    if (lane == 0) nrm[s] = (T)n;
  }
  const int hw = w / 2;
  const double p = pos ? pos[row % pmod] : 0.0;
  for (int j = lane; j < hw; j += 64) {
    const double a = (double)x[j] * inv, b = (double)x[j + hw] * inv;
    if (pos) {
      double sn, cs;
      sincos(p * invf[j], &sn, &cs);
      y[j] = (T)(a * cs - b * sn);
      y[j + hw] = (T)(b * cs + a * sn);
    } else {
      y[j] = (T)a;
      y[j + hw] = (T)b;
    }
  }
}

// Adjoint of b_nrope_fwd: dX = l2n'(X)[R(-p) dY] (in place over dY allowed).
// With NORM: dx = (g - y (y . g)) / n, g the un-rotated gradient, y = x / n.
template <bool NORM, class T = float>
__global__ __launch_bounds__(256) void b_nrope_bwd_kernel(const T* __restrict__ X, const T* __restrict__ nrm,
                                                          const T* dY, T* dX, long rows, int nh, int w,
                                                          const double* __restrict__ pos, long pmod,
                                                          const double* __restrict__ invf, float eps) {
  const long s = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (s >= rows * nh) return;
  const long row = s / nh;
  const int c = (int)(s - row * nh);
  const long off = row * ((long)nh * w) + (long)c * w;
  const int hw = w / 2;
  const double p = pos ? pos[row % pmod] : 0.0;
  // un-rotate into dX, and the dot product y . g
  double yg = 0.0;
  const double n = NORM ? (double)nrm[s] : 1.0;
  const double inv = NORM ? 1.0 / fmax(n, (double)eps) : 1.0;
  for (int j = lane; j < hw; j += 64) {
    double g0 = dY[off + j], g1 = dY[off + j + hw];
    if (pos) {
      double sn, cs;
      sincos(p * invf[j], &sn, &cs);
      const double a = g0, b = g1;
      g0 = a * cs + b * sn;
      g1 = b * cs - a * sn;
    }
    dX[off + j] = (T)g0;
    dX[off + j + hw] = (T)g1;
    if (NORM) yg += (double)X[off + j] * inv * g0 + (double)X[off + j + hw] * inv * g1;
  }
  if (!NORM) return;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) yg += __shfl_xor(yg, o);
  const bool above = n > (double)eps;
  for (int j = lane; j < hw; j += 64) {   // the elements this lane wrote above
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const long o = off + j + e * hw;
      const double g = dX[o];
      dX[o] = (T)(above ? (g - (double)X[o] * inv * yg) * inv : g * inv);
    }
  }
}

// P = softmax(scale * S) over rows of length n (S of type TS, P float; P may
// overwrite S when both are float).  Exponents and sums in fp64.
template <class TS>
__global__ __launch_bounds__(256) void b_softmax_fwd_kernel(const TS* S, float* P, long rows, int n, float scale) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const TS* s = S + row * n;
  float* pr = P + row * n;
  double m = -INFINITY;
  for (int j = lane; j < n; j += 64) m = fmax(m, (double)scale * s[j]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o));
  double sum = 0.0;
  for (int j = lane; j < n; j += 64) sum += exp((double)scale * s[j] - m);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  const double inv = 1.0 / sum;
  for (int j = lane; j < n; j += 64) pr[j] = (float)(exp((double)scale * s[j] - m) * inv);
}

// dS = scale * P * (dP - rowsum(P * dP)) (in place over dP, of type TD).
template <class TD>
__global__ __launch_bounds__(256) void b_softmax_bwd_kernel(const float* __restrict__ P, TD* __restrict__ dP, long rows,
                                                            int n, float scale) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* p = P + row * n;
  TD* d = dP + row * n;
  double dot = 0.0;
  for (int j = lane; j < n; j += 64) dot += (double)p[j] * d[j];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) dot += __shfl_xor(dot, o);
  for (int j = lane; j < n; j += 64) d[j] = (TD)((double)scale * p[j] * ((double)d[j] - dot));
}

__device__ __forceinline__ float b_silu(float x) { return x / (1.f + expf(-x)); }
__device__ __forceinline__ float b_gelu(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }

// FFN activation, elementwise over n values: SwiGLU a = SiLU(g) * u, or
// GELU a = gelu(u) (g unused).
static __global__ void b_act_fwd_kernel(const float* __restrict__ g, const float* __restrict__ u, float* __restrict__ a,
                                        long n, int swiglu) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    a[i] = swiglu ? b_silu(g[i]) * u[i] : b_gelu(u[i]);
}

// Adjoint: dg = da * u * SiLU'(g), du = da * SiLU(g) (SwiGLU), or
// du = da * gelu'(u) (GELU).  dg / du may overwrite da.
static __global__ void b_act_bwd_kernel(const float* __restrict__ g, const float* __restrict__ u, const float* da,
                                        float* dg, float* du, long n, int swiglu) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) {
    const float d = da[i];
    if (swiglu) {
      const float x = g[i], sg = 1.f / (1.f + expf(-x));
      dg[i] = d * u[i] * sg * (1.f + x * (1.f - sg));
      du[i] = d * x * sg;
    } else {
      const float x = u[i];
      du[i] = d * (0.5f * (1.f + erff(x * 0.70710678118654752f)) + x * expf(-0.5f * x * x) * 0.3989422804014327f);
    }
  }
}

// db[j] = sum over rows of dX[row][j], j < w (ld = row stride), in fp64 and
// in a fixed order (deterministic): chunk c of gridDim.y sums rows
// [c R, c R + R) per column into part[c][j] (one thread per column), then the
// chunks are added in order.
constexpr int COLSUM_CHUNKS = 64;
template <class T>
__global__ __launch_bounds__(256) void b_colsum_part_kernel(const T* __restrict__ dX, long rows, long ld, int w,
                                                            double* __restrict__ part) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= w) return;
  const long R = (rows + gridDim.y - 1) / gridDim.y;
  const long r0 = blockIdx.y * R, r1 = r0 + R < rows ? r0 + R : rows;
  double s = 0.0;
  for (long r = r0; r < r1; ++r) s += dX[r * ld + j];
  part[(long)blockIdx.y * w + j] = s;
}
static __global__ void b_colsum_fin_kernel(const double* __restrict__ part, int chunks, int w, float* __restrict__ db) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= w) return;
  double s = 0.0;
  for (int c = 0; c < chunks; ++c) s += part[(long)c * w + j];
  db[j] = (float)s;
}

static __global__ void b_fill_kernel(float* __restrict__ x, long n, float v) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) x[i] = v;
}

static __global__ void b_copy_kernel(const float* __restrict__ x, float* __restrict__ y, long n) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x) y[i] = x[i];
}

// X[h*N + n] = [R(-p_n) K[h][n] ; V[h][n]] (fp64 angles), one thread per pair.
static __global__ void b_stage_x_kernel(const float* __restrict__ K, const float* __restrict__ V,
                                        const double* __restrict__ pos, const double* __restrict__ invf, long HN, long N,
                                        int d, float* __restrict__ X) {
  const int hd = d / 2;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < HN * hd; i += (long)gridDim.x * blockDim.x) {
    const long row = i / hd;
    const int j = (int)(i - row * hd);
    const float* k = K + row * d;
    double sn, cs;
    sincos(pos[row % N] * invf[j], &sn, &cs);
    const double a = k[j], b = k[j + hd];
    float* x = X + row * 2 * d;
    x[j] = (float)(a * cs + b * sn);
    x[j + hd] = (float)(b * cs - a * sn);
    x[d + j] = V[row * d + j];
    x[d + j + hd] = V[row * d + j + hd];
  }
}

}  // namespace still
