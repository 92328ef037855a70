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
static __global__ __launch_bounds__(256) void positions_kernel(const double* __restrict__ p, long N, int t,
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
static __global__ void rope_table_kernel(const double* __restrict__ pos, long R, int w, double base,
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
// One workgroup per (RW keys, head).  Rows are read and written in runs of 8
// elements (16-byte bf16 / fp16 accesses); the transpose goes through LDS and
// is written in runs of 8 keys.  RW is a multiple of 8 dividing 256.
// ---------------------------------------------------------------------------
template <class T> __device__ __forceinline__ void load8(const T* p, float (&o)[8]);
template <> __device__ __forceinline__ void load8<bf16>(const bf16* p, float (&o)[8]) {
  const uint4 u = *(const uint4*)p;
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[2 * i] = __uint_as_float(w[i] << 16);
    o[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
template <> __device__ __forceinline__ void load8<float>(const float* p, float (&o)[8]) {
  const f32x4 a = *(const f32x4*)p, b = *(const f32x4*)(p + 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    o[i] = a[i];
    o[4 + i] = b[i];
  }
}
template <class T> __device__ __forceinline__ void store8(T* p, const float (&v)[8]) {
  T t[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) t[i] = from_f32<T>(v[i]);
  if constexpr (sizeof(T) == 2) {
    *(uint4*)p = *(const uint4*)t;
  } else {
    *(f32x4*)p = *(const f32x4*)t;
    *(f32x4*)(p + 4) = *(const f32x4*)(t + 4);
  }
}

// ---------------------------------------------------------------------------
// fp16 range of the staged cache.  The fp16 operands hold magnitudes up to
// 65504 while bf16 inputs reach 3.4e38, so each KV head's X = [R(-p) K; V]
// is staged times a power of two 2^-e_h, e_h >= 0 the smallest exponent that
// brings max(|K|, |V|) of the head to at most 2^14 (the rotation keeps the
// norm of each pair).  The scaling is exact, leaves the keys' directions
// (hence the QK-normed logits) unchanged when the key bias is scaled with
// them, and is undone on the value path by the output projection; for caches
// within 2^14 it is 1 and changes nothing.
// ---------------------------------------------------------------------------
// scale[h] = 2^-e_h and scale[H + h] = 2^e_h from the per-workgroup maxima
// of |K|, |V| that the staging pass wrote for head h.  One workgroup per head.
static __global__ __launch_bounds__(256) void kv_scale_kernel(const float* __restrict__ part, int nblk, int H,
                                                       float* __restrict__ scale) {
  __shared__ float red[4];
  const int h = blockIdx.x;
  float m = 0.f;
  for (int b = threadIdx.x; b < nblk; b += 256) m = fmaxf(m, part[(long)h * nblk + b]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    float s = 1.f, inv = 1.f;
    while (m * s > 16384.f) {   // at most ~113 halvings (m < 2^128; NaN stops at once)
      s *= 0.5f;
      inv *= 2.f;
    }
    scale[h] = s;
    scale[H + h] = inv;
  }
}

// Staging passes: pass 0 stages every head unscaled and, with `part`,
// writes each workgroup's max(|K|, |V|) (part[h][blockIdx.x]); pass 1
// re-stages, times hscale[h], only the heads whose scale is not 1 (the
// workgroups of the other heads exit at once).
template <class IT, class CT>
__global__ __launch_bounds__(256) void stage_x_kernel(const IT* __restrict__ K, const IT* __restrict__ V,
                                                      const double* __restrict__ pos, const double* __restrict__ invf,
                                                      long N, int d,
                                                      CT* __restrict__ X, CT* __restrict__ XT, long ldxt,
                                                      int RW, float* __restrict__ part, const float* __restrict__ hscale,
                                                      int pass) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem_raw[];
  CT* tile = (CT*)smem_raw;              // [RW][2d + 8]
  const int h = blockIdx.y;
  const float sc = pass ? hscale[h] : 1.f;   // fp16 range scale of this head (exact power of two)
  if (sc == 1.f && pass) return;             // uniform
  float amax = 0.f;
  const long n0 = (long)blockIdx.x * RW;
  const int d2 = 2 * d, hh = d / 2, ld = d2 + 8;
  const IT* Kh = K + (long)h * N * d;
  const IT* Vh = V + (long)h * N * d;
  // phase 1: per row, hh/8 key runs (each giving both rotation halves) and d/8 value runs
  const int kit = hh / 8, per_row = kit + d / 8;
  for (int e = threadIdx.x; e < RW * per_row; e += 256) {
    const int r = e / per_row, q = e - r * per_row;
    const long n = n0 + r;
    CT* xr = X + ((long)h * N + n) * d2;
    if (q < kit) {
      const int j = 8 * q;
      float y0[8], y1[8];
      if (n < N) {
        float a[8], b[8];
        load8(Kh + n * d + j, a);
        load8(Kh + n * d + j + hh, b);
#pragma unroll
        for (int u = 0; u < 8; ++u) amax = fmaxf(amax, fmaxf(fabsf(a[u]), fabsf(b[u])));
        const double pn = pos[n];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float2 cs = rope_cs(pn, invf[j + u]);   // base RoPE of pair j + u at position n
          // inverse rotation: (a, b) -> (a cos + b sin, b cos - a sin)
          y0[u] = a[u] * cs.x + b[u] * cs.y;
          y1[u] = b[u] * cs.x - a[u] * cs.y;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          y0[u] *= sc;
          y1[u] *= sc;
        }
        store8(xr + j, y0);
        store8(xr + j + hh, y1);
      } else {
#pragma unroll
        for (int u = 0; u < 8; ++u) y0[u] = y1[u] = 0.f;
      }
      store8(tile + r * ld + j, y0);
      store8(tile + r * ld + j + hh, y1);
    } else {
      const int f = 8 * (q - kit);
      float v[8];
      if (n < N) {
        load8(Vh + n * d + f, v);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          amax = fmaxf(amax, fabsf(v[u]));
          v[u] *= sc;
        }
        store8(xr + d + f, v);
      } else {
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = 0.f;
      }
      store8(tile + r * ld + d + f, v);
    }
  }
  if (part) {   // this workgroup's max |K|, |V| (reduced through the LDS tile's tail before phase 2 reuses nothing)
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) amax = fmaxf(amax, __shfl_xor(amax, o));
    __shared__ float red[4];
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = amax;
    __syncthreads();
    if (threadIdx.x == 0) part[(long)h * gridDim.x + blockIdx.x] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  }
  __syncthreads();
  // phase 2: X^T, 8 keys per store: the fragment-tiled layout of the fp16
  // cross-attention (xtile_off, ldxt keys per head), or row-major [h][f][ldxt]
  const int runs = RW / 8;
  for (int e = threadIdx.x; e < d2 * runs; e += 256) {
    const int f = e / runs, c8 = e - f * runs;
    const long n = n0 + 8 * c8;
    if (n >= ldxt) continue;
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = to_f32(tile[(8 * c8 + u) * ld + f]);
    if constexpr (sizeof(CT) == 2) store8(XT + xtile_off(h, f, n, ldxt, d2), v);
    else store8(XT + ((long)h * d2 + f) * ldxt + n, v);
  }
}

// Z = latents (fp32 residual stream).
template <class IT>
__global__ void init_z_kernel(const IT* __restrict__ lat, float* __restrict__ Z, long n) {
  const long stride = (long)gridDim.x * blockDim.x, i0 = blockIdx.x * (long)blockDim.x + threadIdx.x;
  if ((n & 7) == 0 && (((uintptr_t)lat | (uintptr_t)Z) & 15) == 0) {   // 8 values per thread and step
    for (long i = i0; i < n / 8; i += stride) {
      float v[8];
      if constexpr (sizeof(IT) == 2) {
        const uint4 u = *(const uint4*)(lat + 8 * i);
        const uint32_t wd[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          v[2 * k] = to_f32(__builtin_bit_cast(IT, (uint16_t)(wd[k] & 0xffffu)));
          v[2 * k + 1] = to_f32(__builtin_bit_cast(IT, (uint16_t)(wd[k] >> 16)));
        }
      } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = to_f32(lat[8 * i + k]);
      }
      *(f32x4*)(Z + 8 * i) = f32x4{v[0], v[1], v[2], v[3]};
      *(f32x4*)(Z + 8 * i + 4) = f32x4{v[4], v[5], v[6], v[7]};
    }
  } else {
    for (long i = i0; i < n; i += stride) Z[i] = to_f32(lat[i]);
  }
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

// Y = RMSNorm(Z) split into a high and a low fp16 part (Y ~= hi + lo to
// about 22 bits) for products whose result must be more accurate than one
// fp16 rounding of Y allows.
static __global__ __launch_bounds__(256) void rmsnorm_split_kernel(const float* __restrict__ Z, f16* __restrict__ Yhi,
                                                            f16* __restrict__ Ylo, long rows, int D, float eps) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* z = Z + row * D;
  float s = 0.f;
  for (int i = lane; i < D; i += 64) s += z[i] * z[i];
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
  const float r = 1.f / sqrtf(s / (float)D + eps);
  for (int i = lane; i < D; i += 64) {
    const float y = z[i] * r;
    const f16 hi = (f16)y;
    Yhi[row * D + i] = hi;
    Ylo[row * D + i] = (f16)(y - (float)hi);
  }
}


// rn[r][c] = 1 / max(sqrt(sum_p part[c*np + p][r]), eps)   (QK-norm factors)
static __global__ void finalize_norm_kernel(const float* __restrict__ part, long rows, int nh, int np,
                                     float eps, float* __restrict__ rn) {
  const long total = rows * nh;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const long r = i / nh;
    const int c = (int)(i - r * nh);
    const float* p = part + (long)c * np * rows + r;   // partials [c*np + k][rows]
    float s = 0.f;
    for (int k = 0; k < np; ++k) s += p[(long)k * rows];
    rn[i] = 1.f / fmaxf(sqrtf(s), eps);
  }
}

// Row softmax of the self-attention logits: S [rows][ld] fp32 (first t
// columns valid) -> P (columns >= t set to zero).  One wave per row.
// With `ref` (fp32 mode), the row's 4 largest logits are first recomputed from
// the fp32 q and k rows with a tree-reduced dot product: the MFMA product
// accumulates the head width sequentially, and the d_l logit scale amplifies
// that rounding for exactly the keys that carry the row's mass.
struct SoftmaxRefine {
  const float* q;     // [H*t][Es]  un-normalised self-attention queries (fp32)
  const float* k;     // [H*t][Es]  keys
  const float* rq;    // [H*t][ns]  1 / ||q~||
  const float* rk;    // [H*t][ns]
  int Es, ds, ns, t;
  float scale;
};

template <class CT>
__global__ __launch_bounds__(256) void softmax_rows_kernel(const float* __restrict__ S, CT* __restrict__ P,
                                                           long rows, int t, int ld, SoftmaxRefine ref) {
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* s = S + row * ld;
  if (!ref.q && ld <= 1024) {
    // the whole row in registers: element 256u + 4*lane + e of the row
    float v[16];
    float m = -INFINITY;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i0 = 256 * u + 4 * lane;
      f32x4 x = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      if (i0 < ld) x = *(const f32x4*)(s + i0);   // ld is a multiple of 4
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[4 * u + e] = (i0 + e < t) ? x[e] : -INFINITY;
        m = fmaxf(m, v[4 * u + e]);
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      v[k] = expf(v[k] - m);   // masked entries give 0
      sum += v[k];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    const float inv = 1.f / sum;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int i0 = 256 * u + 4 * lane;
      if (i0 >= ld) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) P[row * ld + i0 + e] = from_f32<CT>(v[4 * u + e] * inv);
    }
    return;
  }
  float m = -INFINITY;
  for (int i = lane; i < t; i += 64) m = fmaxf(m, s[i]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  int fix_j[4];
  float fix_v[4];
  int nfix = 0;
  if (ref.q) {
    // pick the row's 4 largest logits one at a time (ties: lowest column)
    float last = INFINITY;
    int lastj = -1;
    for (int r = 0; r < 4; ++r) {
      float bv = -INFINITY;
      int bj = 0x7fffffff;
      for (int i = lane; i < t; i += 64) {
        const float v = s[i];
        const bool after = v < last || (v == last && i > lastj);
        if (after && (v > bv || (v == bv && i < bj))) {
          bv = v;
          bj = i;
        }
      }
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) {
        const float ov = __shfl_xor(bv, o);
        const int oj = __shfl_xor(bj, o);
        if (ov > bv || (ov == bv && oj < bj)) {
          bv = ov;
          bj = oj;
        }
      }
      if (bj >= t) break;
      last = bv;
      lastj = bj;
      const long hc = row / t;
      const int i = (int)(row - hc * t);
      const int h = (int)(hc / ref.ns), c = (int)(hc - (long)h * ref.ns);
      const float* qr = ref.q + ((long)h * ref.t + i) * ref.Es + (long)c * ref.ds;
      const float* kr = ref.k + ((long)h * ref.t + bj) * ref.Es + (long)c * ref.ds;
      float dot = 0.f;
      for (int e = lane; e < ref.ds; e += 64) dot += qr[e] * kr[e];
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) dot += __shfl_xor(dot, o);
      fix_j[nfix] = bj;
      fix_v[nfix] = dot * ref.scale * ref.rq[((long)h * ref.t + i) * ref.ns + c] *
                    ref.rk[((long)h * ref.t + bj) * ref.ns + c];
      ++nfix;
    }
    for (int r = 0; r < nfix; ++r) m = fmaxf(m, fix_v[r]);
  }
  auto val = [&](int i) {
    float v = s[i];
    for (int r = 0; r < nfix; ++r) v = (i == fix_j[r]) ? fix_v[r] : v;
    return v;
  };
  float sum = 0.f;
  for (int i = lane; i < t; i += 64) sum += expf(val(i) - m);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
  const float inv = 1.f / sum;
  for (int i = lane; i < ld; i += 64) P[row * ld + i] = from_f32<CT>(i < t ? expf(val(i) - m) * inv : 0.f);
}

// ---------------------------------------------------------------------------
// Exact-logit refinement of the heaviest keys.  The flash pass computes
// logits from fp16-rounded q and k; for the few keys that carry almost all of
// a latent's attention mass those roundings (amplified by the d_l logit
// scale) matter, so their logits are recomputed accurately and the softmax
// weights corrected.  P X is linear in P, so replacing the weights of the
// selected keys is exact for them; every other key keeps a weight below
// 2^-REFINE_MARGIN of the row maximum.
// ---------------------------------------------------------------------------

// Pick, per latent row, every candidate of the flash pass's per-split lists
// whose logit lies within REFINE_MARGIN of the row maximum, largest first, up
// to R of them: slots [0, rcnt[row]) of the row hold them.  Exact ties (duplicated
// cache rows) are taken together up to that cap, so their weights stay
// consistent.  More than CAP in-margin entries in a row: the first CAP read
// are ranked.  A split's
// list of C entries holds CB fixed entries, then (with ocnt) ocnt[split][row]
// overflow entries.
//
// One wave per row: the lists are read with coalesced loads, the in-margin
// candidates (usually two or three) are compacted into LDS, and each takes
// its rank among them, equal logits ordered by key index, so the selection
// does not depend on the order in which the flash pass appended overflow
// entries.
template <int R>
__global__ __launch_bounds__(256) void refine_select_kernel(const float* __restrict__ cval,
                                                            const int* __restrict__ cidx,
                                                            const int* __restrict__ ocnt,
                                                            const float* __restrict__ mpart, int S, long HCT, int C,
                                                            int CB, int* __restrict__ ridx, float* __restrict__ rval,
                                                            int* __restrict__ rcnt) {
  constexpr int CAP = 512;   // in-margin candidates kept per row
  __shared__ float sv[4][CAP];
  __shared__ int si[4][CAP];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const long row = blockIdx.x * 4L + wv;
  const bool active = row < HCT;
  float M = -INFINITY;
  if (active)
    for (int s = lane; s < S; s += 64) M = fmaxf(M, mpart[s * HCT + row]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  const float cut = M - REFINE_MARGIN;
  int n = 0;
  if (active) {
    for (int s = 0; s < S; ++s) {
      const long base = (s * HCT + row) * C;
      const int cnt = CB + (ocnt ? ocnt[s * HCT + row] : 0);
      for (int k0 = 0; k0 < cnt; k0 += 64) {
        const int k = k0 + lane;
        float v = -INFINITY;
        int id = -1;
        if (k < cnt) {
          v = cval[base + k];
          id = cidx[base + k];
        }
        const bool keep = id >= 0 && v >= cut;
        const unsigned long long mask = __ballot(keep);
        const int pos = n + __popcll(mask & ((1ull << lane) - 1ull));
        if (keep && pos < CAP) {
          sv[wv][pos] = v;
          si[wv][pos] = id;
        }
        n += __popcll(mask);
      }
    }
  }
  n = min(n, CAP);
  __syncthreads();
  if (!active) return;
  for (int j = lane; j < n; j += 64) {
    const float v = sv[wv][j];
    const int id = si[wv][j];
    int rank = 0;
    for (int q = 0; q < n; ++q) {
      const float vq = sv[wv][q];
      const int iq = si[wv][q];
      rank += (vq > v || (vq == v && iq < id)) ? 1 : 0;
    }
    if (rank < R) {
      ridx[row * R + rank] = id;
      rval[row * R + rank] = v;
    }
  }
  if (lane == 0) rcnt[row] = min(n, R);
}

// Pack the refinement slots of each (KV head, cross head) list b: crow[b][j],
// j < count[b], lists the slots (latent i, rank q < rcnt[b][i]) as i * R + q,
// in slot order.  One workgroup per list.
static __global__ __launch_bounds__(256) void refine_compact_kernel(const int* __restrict__ rcnt, int t, int R,
                                                             int* __restrict__ crow, int* __restrict__ count) {
  __shared__ int ssum[256];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int per = (t + 255) / 256;
  const int lo = min(t, tid * per), hi = min(t, lo + per);
  const int* rc = rcnt + (long)b * t;
  int n = 0;
  for (int i = lo; i < hi; ++i) n += rc[i];
  ssum[tid] = n;
  __syncthreads();
  for (int o = 1; o < 256; o <<= 1) {   // inclusive scan
    const int v = tid >= o ? ssum[tid - o] : 0;
    __syncthreads();
    ssum[tid] += v;
    __syncthreads();
  }
  int pos = ssum[tid] - n;
  int* cb = crow + (long)b * t * R;
  for (int i = lo; i < hi; ++i) {
    const int ni = rc[i];
    for (int q = 0; q < ni; ++q) cb[pos++] = i * R + q;
  }
  if (tid == 255) count[b] = ssum[255];
}

// Merge split-N partials into O[h*t + i][c*2d + f]:
//   O = (sum_s 2^(m_s - M) O_s + sum_r D_r X_r) / (sum_s 2^(m_s - M) l_s + sum_r D_r)
// where, for each refined key r, D_r = 2^(S_exact - M) - 2^(S_flash - M) swaps
// the weight the flash pass gave it for the accurate one (R = 0: plain merge).
// Slots [0, rcnt[row]) of a row hold its refined keys.
constexpr int REFINE_RMAX = 256;  // refined keys per latent the merge handles (64 per pass of a wave)
struct RefineArgs {
  int R, NP;
  const int* ridx;          // [H*nc*t][R]
  const int* rcnt;          // [H*nc*t]      refined keys of each row
  const float* rval;        // [H*nc*t][R]   logits used by the flash pass (log2 units)
  // NP > 0: [H*nc*t*R][NP] (dot, sum of squares) partials of the exact keys,
  //         combined here with rq into the exact logit;
  // NP = 0: [H*nc*t*R] with .x = exact logit - flash logit (fp64 refinement)
  const float2* rpart;
  const float* rq;          // [H*t][nc]     1 / ||q~||
  const void* X;            // [H*N][2d]     the rows the flash pass multiplied by P
  long N;
  float scale_log2, l2_eps;
};

// One wave per output row (h, c, i); lane l owns features [l*VPL, (l+1)*VPL).
// All loads that do not depend on one another are issued before any result
// is used: the first split's partial row, every split's (m, l), and the
// first 64 refined keys' indices, flash logits and exact-logit data (one key
// per lane); the rows of X of the refined keys follow, four at a time, once
// their indices are known.  Rows with more refined keys take them 64 at a
// time afterwards.
template <class CT, int VPL>
__global__ __launch_bounds__(256) void merge_kernel(const float* __restrict__ opart, const float* __restrict__ mpart,
                                                    const float* __restrict__ lpart, int S, int H, int nc, int t,
                                                    CT* __restrict__ O, RefineArgs ra) {
  constexpr int d2 = 64 * VPL;
  const int lane = threadIdx.x & 63;
  const long row = blockIdx.x * 4L + (threadIdx.x >> 6);   // (h*nc + c)*t + i
  const long HCT = (long)H * nc * t;
  if (row >= HCT) return;   // whole wave
  const int hc = (int)(row / t), i = (int)(row - (long)hc * t);
  const int h = hc / nc, c = hc - h * nc;
  const int f0 = lane * VPL;
  // split 0's partial row (every split holds a partial for every row)
  float v0[VPL];
  {
    const float* op = opart + row * d2 + f0;
#pragma unroll
    for (int u = 0; u < VPL; u += 2) {
      const float2 v = *(const float2*)(op + u);
      v0[u] = v.x;
      v0[u + 1] = v.y;
    }
  }
  float ms_l = -INFINITY, ls_l = 0.f;   // this lane's split (lane < S; more splits loop below)
  if (lane < S) {
    ms_l = mpart[lane * HCT + row];
    ls_l = lpart[lane * HCT + row];
  }
  int key = -1;
  float rv = 0.f, dot = 0.f, ss = 0.f;
  const int nref = ra.R > 0 ? ra.rcnt[row] : 0;
  const int n0 = min(nref, 64);
  auto ref_load = [&](int r, int& key, float& rv, float& dot, float& ss) {
    dot = 0.f;
    ss = 0.f;
    key = ra.ridx[row * ra.R + r];
    rv = ra.rval[row * ra.R + r];
    if (ra.NP == 0) {
      dot = ra.rpart[row * ra.R + r].x;
    } else {
      const float2* p = ra.rpart + (row * ra.R + r) * ra.NP;
      float d1 = 0.f, s1 = 0.f;
      int k = 0;
      for (; k + 1 < ra.NP; k += 2) {
        const float2 a = p[k], b = p[k + 1];
        dot += a.x;
        ss += a.y;
        d1 += b.x;
        s1 += b.y;
      }
      if (k < ra.NP) {
        dot += p[k].x;
        ss += p[k].y;
      }
      dot += d1;
      ss += s1;
    }
  };
  if (lane < n0) ref_load(lane, key, rv, dot, ss);
  const float rqv = ra.R > 0 && ra.NP > 0 ? ra.rq[((long)h * t + i) * nc + c] : 0.f;
  // maximum and normaliser over the splits
  float M = ms_l;
  for (int s = lane + 64; s < S; s += 64) M = fmaxf(M, mpart[s * HCT + row]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  float L = ms_l != -INFINITY ? exp2f(ms_l - M) * ls_l : 0.f;
  for (int s = lane + 64; s < S; s += 64) {
    const float ms = mpart[s * HCT + row];
    if (ms != -INFINITY) L += exp2f(ms - M) * lpart[s * HCT + row];
  }
  // weight change of each refined key: 2^(exact - M) - 2^(flash - M)
  auto delta = [&](float rv, float dot, float ss) -> float {
    if (ra.NP == 0) return exp2f(rv - M) * expm1f(dot * 0.69314718055994531f);
    const float sx = ra.scale_log2 * rqv * dot / fmaxf(sqrtf(ss), ra.l2_eps);
    return exp2f(sx - M) - exp2f(rv - M);
  };
  float dl = lane < n0 ? delta(rv, dot, ss) : 0.f;
  L += dl;
  const float w0 = __shfl(ms_l, 0);
  float acc[VPL];
  const float ws0 = w0 != -INFINITY ? exp2f(w0 - M) : 0.f;
#pragma unroll
  for (int u = 0; u < VPL; ++u) acc[u] = ws0 * v0[u];
  // refined keys' rows of X, four at a time; keys cb .. cb + nk - 1 held by
  // lanes 0 .. nk - 1 (key index, weight change)
  auto add_rows = [&](int nk) {
    for (int r0 = 0; r0 < nk; r0 += 4) {
      float xr[4][VPL];
      float dr[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = __shfl(key, r0 + q);
        dr[q] = __shfl(dl, r0 + q);
        const bool use = r0 + q < nk;
        const CT* x = (const CT*)ra.X + ((long)h * ra.N + (use ? n : 0)) * d2 + f0;
#pragma unroll
        for (int u = 0; u < VPL; ++u) xr[q][u] = to_f32(x[u]);
        if (!use) dr[q] = 0.f;
      }
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int u = 0; u < VPL; ++u) acc[u] += dr[q] * xr[q][u];
    }
  };
  add_rows(n0);
  for (int cb = 64; cb < nref; cb += 64) {   // rows with more than 64 refined keys
    const int nk = min(nref - cb, 64);
    key = -1;
    dl = 0.f;
    if (lane < nk) {
      ref_load(cb + lane, key, rv, dot, ss);
      dl = delta(rv, dot, ss);
    }
    L += dl;
    add_rows(nk);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) L += __shfl_xor(L, o);
  for (int s = 1; s < S; ++s) {
    const float ms = mpart[s * HCT + row];
    if (ms == -INFINITY) continue;
    const float ws = exp2f(ms - M);
    const float* op = opart + (s * HCT + row) * d2 + f0;
#pragma unroll
    for (int u = 0; u < VPL; u += 2) {
      const float2 v = *(const float2*)(op + u);
      acc[u] += ws * v.x;
      acc[u + 1] += ws * v.y;
    }
  }
  const float invL = 1.f / L;
  CT* dst = O + ((long)h * t + i) * ((long)nc * d2) + (long)c * d2 + f0;
#pragma unroll
  for (int u = 0; u < VPL; ++u) dst[u] = from_f32<CT>(acc[u] * invL);
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

// Zero keys [t, npad) of rows feature-major values in the tiled layout
// (xtile_off): rows = (KV heads) x (features per head), npad keys per row.
static __global__ void zero_xtile_tail_kernel(f16* __restrict__ A, long rows, int t, long npad) {
  const long w = npad - t;
  const long total = rows * w;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const long r = i / w;
    A[xtile_off(0, r, t + (i - r * w), npad, 32)] = (f16)0.f;
  }
}

// Zero keys [n0, npad) of the fragment-tiled key layout (ktile_off) of
// `heads` heads of width dc, one 16-byte unit per thread and step: the
// cross-attention masks those keys additively, which needs finite logits.
static __global__ void zero_ktile_tail_kernel(f16* __restrict__ k, long heads, int n0, long npad, int dc) {
  const long w = npad - n0, units_per_key = dc / 8;
  const long total = heads * w * units_per_key;
  const uint4 z = {0u, 0u, 0u, 0u};
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < total; i += (long)gridDim.x * blockDim.x) {
    const long hc = i / (w * units_per_key), r = i - hc * (w * units_per_key);
    const long n = n0 + r / units_per_key, x = (r % units_per_key) * 8;
    *(uint4*)(k + ktile_off(hc, n, x, npad, dc)) = z;
  }
}

// Element-type conversion of up to CONV_SEGS weight matrices per launch
// (bf16 -> fp16 for the MFMA operands), one segment per grid row, 8 elements
// per thread and step; segment lengths are multiples of 8 and 16-byte aligned.
constexpr int CONV_SEGS = 16;
struct ConvSegs {
  const void* src[CONV_SEGS];
  void* dst[CONV_SEGS];
  long n8[CONV_SEGS];   // length / 8
};

template <class IT, class CT>
__global__ void convert_kernel(ConvSegs segs) {
  const int s = blockIdx.y;
  const IT* src = (const IT*)segs.src[s];
  CT* dst = (CT*)segs.dst[s];
  const long n8 = segs.n8[s];
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n8; i += (long)gridDim.x * blockDim.x)
    *(typename Mma<CT>::frag*)(dst + 8 * i) = VecLoad<CT, IT>::load(src + 8 * i);
}

}  // namespace still
