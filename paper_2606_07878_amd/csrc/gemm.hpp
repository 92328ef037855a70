// gemm.hpp - tiled MFMA GEMM C = A * B^T for the latent-side and projection
// products of the compactor, with the epilogues those products need fused in.
//
//   A [M][K] row-major (K contiguous), B [N][K] row-major (the [out][in] weight
//   layout), both converted to the compute type CT on their way into LDS.
//   256 threads = 4 waves in a 2x2 grid; each wave owns a (BM/2) x (BN/2) block
//   of 32x32 MFMA tiles; two LDS stages, one barrier per k step.
//
// Paired epilogues (PAIR, SWIGLU) need two columns of the result in the same
// lane: the tile's BN columns are two halves of BN/2, half 0 holding the first
// member of each pair and half 1 the second, and every wave owns the same
// sub-range in both halves.
//   PAIR:   pair P -> columns (c*hd + j, c*hd + j + hd/2), c = P / (hd/2),
//           j = P % (hd/2): rotate-half RoPE partners (optional rotation by a
//           cos/sin table, optional bias, optional per-row sum of squares of
//           the un-rotated biased values for the later L2 QK-norm).
//   SWIGLU: pair P -> row P of W_g (half 0) and of W_u (half 1);
//           out[:, P] = SiLU(g) * u.
#pragma once
#include "common.hpp"

namespace still {

enum EpiKind { EPI_STORE = 0, EPI_RESID = 1, EPI_PAIR = 2, EPI_SWIGLU = 3, EPI_SCALE = 4, EPI_GELU = 5, EPI_REFINE = 6 };

struct GemmArgs {
  int M, N, K;   // N = output columns, or column pairs for PAIR / SWIGLU
  int nb2;       // batch index z -> (z / nb2, z % nb2), strides s*1, s*2 (elements)
  const void* A;
  const void* A2;      // optional low part of a split A operand: C = (A + A2) B^T, same layout as A
  long lda, sA1, sA2;
  const void* B;
  const void* B2;  // SWIGLU: W_u
  long ldb, sB1, sB2;
  int bwrap;           // B column k >= bwrap reads column k - bwrap (0 = off)
  void* C;
  long ldc, sC1, sC2;
  const void* bias;    // per output column, NULL = none
  long sBias2;         // bias offset per unit of the inner batch index
  int hd;              // PAIR: head width
  const float2* tab;   // PAIR: rotation table, row (r % tab_mod), entry [row*hd/2 + j]; NULL = none
  int tab_mod;
  float* part;         // PAIR: per-row sum-of-squares partials, NULL = none
  long ldpart;
  float* C2;           // PAIR: optional fp32 copy of the (rotated) outputs, ldc as C
  // REFINE: row r of batch (b1, b2) is candidate slot r of latent i = r / R;
  // its key index is ridx[r] (< 0: empty).  The epilogue rotates by tab[key],
  // dots with qex row i and writes (dot, sum of squares) partials.
  const int* ridx;
  long sI1, sI2;
  int R;
  const float* qex;
  long ldqex, sE1, sE2;
  float2* rpart;
  long sR1, sR2;
  float scale;         // SCALE: C = acc * scale * rq[r] * rk[col]
  const float* rq;
  long ldrq, sQ1, sQ2;
  const float* rk;
  long ldrk, sK1, sK2;
};

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + expf(-x)); }
__device__ __forceinline__ float gelu_f(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }

template <class CT, class TA, class TB, class TC, class TBias, int EPI, int BM, int BN, int BK>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
  typedef Mma<CT> MM;
  typedef typename MM::frag frag;
  constexpr int E = MM::E;
  constexpr int PAD = 16 / sizeof(CT);
  constexpr int LR = BK + PAD;                 // LDS row stride (elements)
  constexpr int TM = BM / 64, TN = BN / 64;    // 32x32 tiles per wave
  constexpr int KV = BK / E;                   // 16-byte vectors per tile row
  constexpr int AV = BM * KV / 256, BV = BN * KV / 256;
  constexpr bool PAIRED = (EPI == EPI_PAIR || EPI == EPI_SWIGLU || EPI == EPI_REFINE);
  static_assert(AV >= 1 && BV >= 1 && BM * KV % 256 == 0 && BN * KV % 256 == 0, "tile/threads");
  static_assert(TN % 2 == 0, "BN must allow two column halves per wave");

  __shared__ __attribute__((aligned(16))) CT As[2][BM * LR];
  __shared__ __attribute__((aligned(16))) CT Bs[2][BN * LR];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, lg = lane >> 5;

  // XCD-aware tile order: consecutive tiles of the N dimension (which share
  // the A row block) stay on one XCD when the grid size allows it.
  const int gx = gridDim.x, gy = gridDim.y;
  int lin = blockIdx.x + gx * blockIdx.y;
  const int T = gx * gy;
  if ((T & 7) == 0) lin = (lin & 7) * (T >> 3) + (lin >> 3);
  const int nt = lin % gx, mt = lin / gx;

  const int bz = blockIdx.z, b1 = bz / g.nb2, b2 = bz - b1 * g.nb2;
  const TA* A = (const TA*)g.A + b1 * g.sA1 + b2 * g.sA2;
  const TB* B = (const TB*)g.B + b1 * g.sB1 + b2 * g.sB2;
  const TB* B2 = PAIRED && g.B2 ? (const TB*)g.B2 + b1 * g.sB1 + b2 * g.sB2 : nullptr;
  const int M = g.M, N = g.N, K = g.K;
  const int m0 = mt * BM;
  const int hh = g.hd >> 1;

  // global -> register staging
  frag ra[AV], rb[BV];
  const TB* brow_ptr[BV];
  bool bvalid[BV];
#pragma unroll
  for (int i = 0; i < BV; ++i) {
    const int v = tid + i * 256, lc = v / KV;
    if (PAIRED) {
      const int half = lc / (BN / 2);
      const int P = nt * (BN / 2) + (lc % (BN / 2));
      bvalid[i] = P < N;
      if (EPI == EPI_PAIR || EPI == EPI_REFINE) {
        const int c = P / hh, j = P - c * hh;
        brow_ptr[i] = B + (long)(c * g.hd + j + half * hh) * g.ldb;
      } else {
        brow_ptr[i] = (half ? B2 : B) + (long)P * g.ldb;
      }
    } else {
      const int n = nt * BN + lc;
      bvalid[i] = n < N;
      brow_ptr[i] = B + (long)n * g.ldb;
    }
  }

  const TA* Alo = g.A2 ? (const TA*)g.A2 + b1 * g.sA1 + b2 * g.sA2 : nullptr;
  auto load_stage = [&](int k0, const TA* Ap) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int v = tid + i * 256, r = v / KV, kk = (v % KV) * E;
      const int gr = m0 + r, gk = k0 + kk;
      ra[i] = (gr < M && gk < K) ? VecLoad<CT, TA>::load(Ap + (long)gr * g.lda + gk) : zero_frag<CT>();
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      const int v = tid + i * 256, kk = (v % KV) * E;
      const int gk = k0 + kk;
      const int gkb = (g.bwrap && gk >= g.bwrap) ? gk - g.bwrap : gk;
      rb[i] = (bvalid[i] && gk < K) ? VecLoad<CT, TB>::load(brow_ptr[i] + gkb) : zero_frag<CT>();
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
      const int v = tid + i * 256, r = v / KV, kk = (v % KV) * E;
      *(frag*)&As[buf][r * LR + kk] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BV; ++i) {
      const int v = tid + i * 256, r = v / KV, kk = (v % KV) * E;
      *(frag*)&Bs[buf][r * LR + kk] = rb[i];
    }
  };

  // local LDS column of the wave's tile tn (two halves, same sub-range in each)
  auto col_base = [&](int tn) {
    const int half = tn / (TN / 2), i = tn % (TN / 2);
    return half * (BN / 2) + wn * (BN / 4) + i * 32;
  };

  f32x16 acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) acc[a][b] = zero16();

  const int nk1 = (K + BK - 1) / BK;
  const int nk = Alo ? 2 * nk1 : nk1;      // split A: second pass over K with the low part
  load_stage(0, A);
  store_stage(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      const int kn = kt + 1;
      if (kn < nk1) load_stage(kn * BK, A);
      else load_stage((kn - nk1) * BK, Alo);
    }
#pragma unroll
    for (int ks = 0; ks < BK / (2 * E); ++ks) {
      frag af[TM], bfr[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a)
        af[a] = *(const frag*)&As[cur][(wm * (BM / 2) + a * 32 + l32) * LR + ks * 2 * E + lg * E];
#pragma unroll
      for (int b = 0; b < TN; ++b)
        bfr[b] = *(const frag*)&Bs[cur][(col_base(b) + l32) * LR + ks * 2 * E + lg * E];
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) MM::mma(acc[a][b], af[a], bfr[b]);
    }
    if (kt + 1 < nk) store_stage(cur ^ 1);
    __syncthreads();
  }

  // ------------------------------------------------------------------ epilogue
  TC* C = (TC*)g.C + b1 * g.sC1 + b2 * g.sC2;
  const TBias* bias = g.bias ? (const TBias*)g.bias + b2 * g.sBias2 : nullptr;
  if constexpr (!PAIRED) {
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int col = nt * BN + col_base(b) + l32;
        if (col >= N) continue;
        const float bv = bias ? to_f32(bias[col]) : 0.f;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int r = m0 + wm * (BM / 2) + a * 32 + 8 * (j >> 2) + 4 * lg + (j & 3);
          if (r >= M) continue;
          float v = acc[a][b][j];
          TC* dst = C + (long)r * g.ldc + col;
          if constexpr (EPI == EPI_RESID) {
            *dst = from_f32<TC>(to_f32(*dst) + v);
          } else if constexpr (EPI == EPI_SCALE) {
            const float* rq = g.rq + b1 * g.sQ1 + b2 * g.sQ2;
            const float* rk = g.rk + b1 * g.sK1 + b2 * g.sK2;
            *dst = from_f32<TC>(v * g.scale * rq[(long)r * g.ldrq] * rk[(long)col * g.ldrk]);
          } else if constexpr (EPI == EPI_GELU) {
            *dst = from_f32<TC>(gelu_f(v + bv));
          } else {
            *dst = from_f32<TC>(v + bv);
          }
        }
      }
  } else {
    float ss[TM][16], dd[TM][16];
#pragma unroll
    for (int a = 0; a < TM; ++a)
#pragma unroll
      for (int j = 0; j < 16; ++j) ss[a][j] = dd[a][j] = 0.f;
#pragma unroll
    for (int b = 0; b < TN / 2; ++b) {
      const int P = nt * (BN / 2) + wn * (BN / 4) + b * 32 + l32;
      if (P >= N) continue;
      if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
        for (int a = 0; a < TM; ++a)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int r = m0 + wm * (BM / 2) + a * 32 + 8 * (j >> 2) + 4 * lg + (j & 3);
            if (r >= M) continue;
            C[(long)r * g.ldc + P] = from_f32<TC>(silu_f(acc[a][b][j]) * acc[a][b + TN / 2][j]);
          }
      } else {
        const int c = P / hh, jp = P - c * hh;
        const int col0 = c * g.hd + jp, col1 = col0 + hh;
        const int* ridx = (EPI == EPI_REFINE) ? g.ridx + b1 * g.sI1 + b2 * g.sI2 : nullptr;
        const float bv0 = bias ? to_f32(bias[col0]) : 0.f;
        const float bv1 = bias ? to_f32(bias[col1]) : 0.f;
#pragma unroll
        for (int a = 0; a < TM; ++a)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int r = m0 + wm * (BM / 2) + a * 32 + 8 * (j >> 2) + 4 * lg + (j & 3);
            if (r >= M) continue;
            const float v0 = acc[a][b][j] + bv0, v1 = acc[a][b + TN / 2][j] + bv1;
            ss[a][j] += v0 * v0 + v1 * v1;
            float y0 = v0, y1 = v1;
            if (g.tab) {
              long trow;
              if constexpr (EPI == EPI_REFINE) {
                const int key = ridx[r];
                trow = key < 0 ? 0 : key;
              } else {
                trow = r % g.tab_mod;
              }
              const float2 cs = g.tab[trow * hh + jp];
              y0 = v0 * cs.x - v1 * cs.y;
              y1 = v1 * cs.x + v0 * cs.y;
            }
            if constexpr (EPI == EPI_REFINE) {
              const int i = r / g.R;
              const float* qe = g.qex + b1 * g.sE1 + b2 * g.sE2 + (long)i * g.ldqex;
              dd[a][j] += y0 * qe[col0] + y1 * qe[col1];
            } else {
              C[(long)r * g.ldc + col0] = from_f32<TC>(y0);
              C[(long)r * g.ldc + col1] = from_f32<TC>(y1);
              if (g.C2) {
                g.C2[(long)r * g.ldc + col0] = y0;
                g.C2[(long)r * g.ldc + col1] = y1;
              }
            }
          }
      }
    }
    if constexpr (EPI == EPI_REFINE) {
      const int P0 = nt * (BN / 2);
      const int nparts = (hh / (BN / 2)) * 2;
      const int pidx = (P0 / (BN / 2)) * 2 + wn;
      float2* rp = g.rpart + b1 * g.sR1 + b2 * g.sR2;
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          float s = ss[a][j], q = dd[a][j];
#pragma unroll
          for (int o = 1; o < 32; o <<= 1) {
            s += __shfl_xor(s, o);
            q += __shfl_xor(q, o);
          }
          const int r = m0 + wm * (BM / 2) + a * 32 + 8 * (j >> 2) + 4 * lg + (j & 3);
          if (l32 == 0 && r < M) rp[(long)r * nparts + pidx] = make_float2(q, s);
        }
    }
    if constexpr (EPI == EPI_PAIR) {
      if (g.part) {
        // the tile's pairs lie inside one head c (hd/2 is a multiple of BN/2)
        const int P0 = nt * (BN / 2);
        const int c = P0 / hh;
        const int nparts = (hh / (BN / 2)) * 2;
        const int pidx = ((P0 - c * hh) / (BN / 2)) * 2 + wn;
#pragma unroll
        for (int a = 0; a < TM; ++a)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            float s = ss[a][j];
            s += __shfl_xor(s, 1);
            s += __shfl_xor(s, 2);
            s += __shfl_xor(s, 4);
            s += __shfl_xor(s, 8);
            s += __shfl_xor(s, 16);
            const int r = m0 + wm * (BM / 2) + a * 32 + 8 * (j >> 2) + 4 * lg + (j & 3);
            if (l32 == 0 && r < M) g.part[(long)r * g.ldpart + c * nparts + pidx] = s;
          }
      }
    }
  }
}

template <class CT, class TA, class TB, class TC, class TBias, int EPI, int BM, int BN, int BK>
hipError_t launch_gemm(const GemmArgs& g, int batch, hipStream_t st) {
  constexpr bool PAIRED = (EPI == EPI_PAIR || EPI == EPI_SWIGLU || EPI == EPI_REFINE);
  const int ntn = PAIRED ? (g.N + BN / 2 - 1) / (BN / 2) : (g.N + BN - 1) / BN;
  const int ntm = (g.M + BM - 1) / BM;
  if (ntn <= 0 || ntm <= 0 || batch <= 0) return hipSuccess;
  dim3 grid(ntn, ntm, batch);
  hipLaunchKernelGGL((gemm_kernel<CT, TA, TB, TC, TBias, EPI, BM, BN, BK>), grid, dim3(256), 0, st, g);
  return hipGetLastError();
}

}  // namespace still
