// misc.hpp - the bandwidth-bound steps around the MFMA products:
// position bookkeeping and rotation tables, RoPE-fix staging of X = [K; V],
// latent init, RMSNorm, QK-norm finalisation, the self-attention row softmax,
// the split-N merge and padding fills.
#pragma once
#include "common.hpp"

namespace still {

// ---------------------------------------------------------------------------
// Latent / output positions: p_i = p_min + i (p_max - p_min)/(t-1) over the
// supplied key positions (p_0 = p_min when t = 1).  One workgroup.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void positions_kernel(const double* __restrict__ p, long N, int t,
                                                        double* __restrict__ pq, double* __restrict__ out) {
  __shared__ double smin[256], smax[256];
  double lo = INFINITY, hi = -INFINITY;
  for (long i = threadIdx.x; i < N; i += 256) {
    const double v = p[i];
    lo = fmin(lo, v);
    hi = fmax(hi, v);
  }
  smin[threadIdx.x] = lo;
  smax[threadIdx.x] = hi;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (threadIdx.x < s) {
      smin[threadIdx.x] = fmin(smin[threadIdx.x], smin[threadIdx.x + s]);
      smax[threadIdx.x] = fmax(smax[threadIdx.x], smax[threadIdx.x + s]);
    }
    __syncthreads();
  }
  lo = smin[0];
  hi = smax[0];
  const double step = t > 1 ? (hi - lo) / (double)(t - 1) : 0.0;
  for (int i = threadIdx.x; i < t; i += 256) {
    const double v = lo + (double)i * step;
    pq[i] = v;
    if (out) out[i] = v;
  }
}

// ---------------------------------------------------------------------------
// Rotation table: tab[r][j] = (cos, sin)(p_r * base^(-2j/w)), j < w/2.
// Angles are formed and reduced in float64 (positions up to ~1e5 times
// frequencies near 1 need more than float32's 24 bits), then rounded.
// ---------------------------------------------------------------------------
__global__ void rope_table_kernel(const double* __restrict__ pos, long R, int w, double base,
                                  float2* __restrict__ tab) {
  const int hh = w / 2;
  const long total = R * hh;
  for (long idx = blockIdx.x * (long)blockDim.x + threadIdx.x; idx < total; idx += (long)gridDim.x * blockDim.x) {
    const long r = idx / hh;
    const int j = (int)(idx - r * hh);
    const double inv = pow(base, -2.0 * (double)j / (double)w);
    const double ang = pos[r] * inv;
    double sn, cs;
    sincos(ang, &sn, &cs);
    tab[idx] = make_float2((float)cs, (float)sn);
  }
}

// ---------------------------------------------------------------------------
// RoPE-fix staging: X[h*N + n] = [R(-p_n) k_n ; v_n] (row-major, 2d wide) and
// its transpose X^T[h][f][n] (key-contiguous, zero for n in [N, ldxt)).
// One workgroup per (RW keys, head); the transpose goes through LDS.
// ---------------------------------------------------------------------------
template <class IT, class CT>
__global__ __launch_bounds__(256) void stage_x_kernel(const IT* __restrict__ K, const IT* __restrict__ V,
                                                      const float2* __restrict__ tab, long N, int d,
                                                      CT* __restrict__ X, CT* __restrict__ XT, long ldxt,
                                                      int RW) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  CT* tile = (CT*)smem_raw;              // [RW][2d + 1]
  const int h = blockIdx.y;
  const long n0 = (long)blockIdx.x * RW;
  const int d2 = 2 * d, hh = d / 2, ld = d2 + 1;
  const IT* Kh = K + (long)h * N * d;
  const IT* Vh = V + (long)h * N * d;
  for (int e = threadIdx.x; e < RW * d2; e += 256) {
    const int r = e / d2, f = e - r * d2;
    const long n = n0 + r;
    float val = 0.f;
    if (n < N) {
      if (f < d) {
        const int j = f < hh ? f : f - hh;
        const float2 cs = tab[n * hh + j];
        const float a = to_f32(Kh[n * d + j]), b = to_f32(Kh[n * d + j + hh]);
        // inverse rotation: (a, b) -> (a cos + b sin, b cos - a sin)
        val = f < hh ? a * cs.x + b * cs.y : b * cs.x - a * cs.y;
      } else {
        val = to_f32(Vh[n * d + (f - d)]);
      }
      X[((long)h * N + n) * d2 + f] = from_f32<CT>(val);
    }
    tile[r * ld + f] = from_f32<CT>(val);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < RW * d2; e += 256) {
    const int f = e / RW, r = e - f * RW;
    const long n = n0 + r;
    if (n < ldxt) XT[((long)h * d2 + f) * ldxt + n] = tile[r * ld + f];
  }
}

// Z = latents (fp32 residual stream).
template <class IT>
__global__ void init_z_kernel(const IT* __restrict__ lat, float* __restrict__ Z, long n) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n; i += (long)gridDim.x * blockDim.x)
    Z[i] = to_f32(lat[i]);
}

// Y = RMSNorm(Z) per row (non-parametric), one wave per row.
template <class OT>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* __restrict__ Z, OT* __restrict__ Y, long rows,
                                                      int D, float eps) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* z = Z + row * D;
  float s = 0.f;
  for (int i = lane; i < D; i += 64) s += z[i] * z[i];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  const float r = 1.f / sqrtf(s / (float)D + eps);
  for (int i = lane; i < D; i += 64) Y[row * D + i] = from_f32<OT>(z[i] * r);
}

// rn[r][c] = 1 / max(sqrt(sum_p part[r][c][p]), eps)   (QK-norm factors)
__global__ void finalize_norm_kernel(const float* __restrict__ part, long rows, int nh, int np,
                                     float eps, float* __restrict__ rn) {
  const long total = rows * nh;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const float* p = part + i * np;
    float s = 0.f;
    for (int k = 0; k < np; ++k) s += p[k];
    rn[i] = 1.f / fmaxf(sqrtf(s), eps);
  }
}

// Row softmax of the self-attention logits: S [rows][ld] fp32 (first t
// columns valid) -> P (columns >= t set to zero).  One wave per row.
template <class CT>
__global__ __launch_bounds__(256) void softmax_rows_kernel(const float* __restrict__ S, CT* __restrict__ P,
                                                           long rows, int t, int ld) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* s = S + row * ld;
  float m = -INFINITY;
  for (int i = lane; i < t; i += 64) m = fmaxf(m, s[i]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  float sum = 0.f;
  for (int i = lane; i < t; i += 64) sum += expf(s[i] - m);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  const float inv = 1.f / sum;
  for (int i = lane; i < ld; i += 64) P[row * ld + i] = from_f32<CT>(i < t ? expf(s[i] - m) * inv : 0.f);
}

// Merge split-N partials: O[h*t + i][c*2d + f] = sum_s 2^(m_s - M) O_s / sum_s 2^(m_s - M) l_s.
template <class CT>
__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ opart, const float* __restrict__ mpart,
                                                    const float* __restrict__ lpart, int S, int H, int nc, int t,
                                                    int d2, CT* __restrict__ O) {
  const long row = blockIdx.x;     // (h*nc + c)*t + i
  const long HCT = (long)H * nc * t;
  const int hc = (int)(row / t), i = (int)(row - (long)hc * t);
  const int h = hc / nc, c = hc - h * nc;
  float M = -INFINITY;
  for (int s = 0; s < S; ++s) M = fmaxf(M, mpart[s * HCT + row]);
  float L = 0.f;
  for (int s = 0; s < S; ++s) {
    const float ms = mpart[s * HCT + row];
    if (ms != -INFINITY) L += exp2f(ms - M) * lpart[s * HCT + row];
  }
  const float invL = 1.f / L;
  CT* dst = O + ((long)h * t + i) * ((long)nc * d2) + (long)c * d2;
  for (int f = threadIdx.x; f < d2; f += 256) {
    float acc = 0.f;
    for (int s = 0; s < S; ++s) {
      const float ms = mpart[s * HCT + row];
      if (ms != -INFINITY) acc += exp2f(ms - M) * opart[(s * HCT + row) * d2 + f];
    }
    dst[f] = from_f32<CT>(acc * invL);
  }
}

// Fill columns [c0, c1) of a [rows][ld] matrix with zeros.
template <class T>
__global__ void zero_cols_kernel(T* __restrict__ A, long rows, int ld, int c0, int c1) {
  const int w = c1 - c0;
  const long total = rows * w;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const long r = i / w;
    A[r * ld + c0 + (i - r * w)] = from_f32<T>(0.f);
  }
}

}  // namespace still
