// refine64.hpp - fp32 validation mode: the refined keys' cross-attention
// logits in fp64.
//
// With QK-norm the logits are d_l * cos(q, k) (App. A, cross-attention), so a
// relative rounding of 1e-7 in q~ or k~ moves the heaviest keys' weights by
// about d_l * 1e-7 ~ 1e-4, the size of the fp32 mode's whole error budget.
// The flash pass therefore keeps its fp32 logits for the bulk of the keys,
// and for the refined keys (those carrying nearly all of a latent's mass)
// the logit is recomputed from the fp32 inputs with every step in fp64:
//   q = RoPE_c(l2n(RMSNorm(Z) W_Q^T + b_Q), p_q)      q64_gemm + q64_finalize
//   k = RoPE_c(l2n(X_n W_K^T + b_K), p_n),  X_n = [R(-p_n) K_n ; V_n]
//   logit = s * log2(e) * q . k                          refine64
// The result is handed to the merge as the difference to the logit the flash
// pass used, so the weight swap 2^(fp32 logit - M) -> 2^(exact - M) keeps
// full precision (the logits themselves are ~1e3 in log2 units).
#pragma once
#include "common.hpp"

namespace still {

// inv_freq[j] = base^(-2j / w), j < w/2 (the RoPE frequencies of width w)
static __global__ void inv_freq64_kernel(double base, int w, double* __restrict__ out) {
  const int j = blockIdx.x * blockDim.x + threadIdx.x;
  if (j < w / 2) out[j] = pow(base, -2.0 * (double)j / (double)w);
}

struct Q64Args {
  const float* Z;      // [rows][D] latent state (fp32)
  const float* W;      // [E][D]    W_Q ([out][in])
  const float* bias;   // [E] or NULL
  double* Q;           // [rows][E] q~ (fp64)
  long rows;
  int D, E;
  float rms_eps;
};

// Q = RMSNorm(Z) W^T + b in fp64.  Tile 128 rows x 128 columns, k chunks of
// 8; thread (tr, tc) of a 16 x 16 grid owns rows tr + 16 i and columns
// tc + 16 j (i, j < 8).  The RMS factor of each row is formed in fp64 first.
static __global__ __launch_bounds__(256) void q64_gemm_kernel(Q64Args a) {
  constexpr int BM = 128, BN = 128, BK = 8;
  __shared__ double As[BK][BM];
  __shared__ double Bs[BK][BN];
  __shared__ double rs[BM];
  const int tid = threadIdx.x;
  const long r0 = (long)blockIdx.y * BM;
  const int c0 = blockIdx.x * BN;
  {  // 2 threads per row
    const int r = tid >> 1, part = tid & 1;
    const long row = r0 + r;
    double ss = 0.0;
    if (row < a.rows) {
      const float* z = a.Z + row * a.D;
      for (int k = part; k < a.D; k += 2) {
        const double v = z[k];
        ss = fma(v, v, ss);
      }
    }
    ss += __shfl_xor(ss, 1);
    if (part == 0) rs[r] = 1.0 / sqrt(ss / (double)a.D + (double)a.rms_eps);
  }
  __syncthreads();
  const int tr = tid >> 4, tc = tid & 15;
  double acc[8][8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.0;
  for (int k0 = 0; k0 < a.D; k0 += BK) {
    for (int e = tid; e < BM * BK; e += 256) {
      const int r = e / BK, k = e % BK;
      const long row = r0 + r;
      double v = 0.0;
      if (row < a.rows && k0 + k < a.D) v = (double)a.Z[row * a.D + k0 + k] * rs[r];
      As[k][r] = v;
    }
    for (int e = tid; e < BN * BK; e += 256) {
      const int c = e / BK, k = e % BK;
      double v = 0.0;
      if (c0 + c < a.E && k0 + k < a.D) v = (double)a.W[(long)(c0 + c) * a.D + k0 + k];
      Bs[k][c] = v;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      double av[8], bv[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) av[i] = As[k][tr + 16 * i];
#pragma unroll
      for (int j = 0; j < 8; ++j) bv[j] = Bs[k][tc + 16 * j];
#pragma unroll
      for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] = fma(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const long row = r0 + tr + 16 * i;
    if (row >= a.rows) continue;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int col = c0 + tc + 16 * j;
      if (col >= a.E) continue;
      a.Q[row * a.E + col] = acc[i][j] + (a.bias ? (double)a.bias[col] : 0.0);
    }
  }
}

// In place: each (row, head c) slice of width dc of Q becomes
// RoPE_c(q~ / max(||q~||, eps)) at the row's latent position.  One wave per
// slice.
static __global__ __launch_bounds__(256) void q64_finalize_kernel(double* __restrict__ Q, long rows, int nc, int dc, int t,
                                                           const double* __restrict__ pq,
                                                           const double* __restrict__ invf, double l2_eps) {
  const long s = blockIdx.x * 4L + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (s >= rows * nc) return;
  const long row = s / nc;
  const int c = (int)(s - row * nc);
  double* q = Q + row * ((long)nc * dc) + (long)c * dc;
  double ss = 0.0;
  for (int j = lane; j < dc; j += 64) ss = fma(q[j], q[j], ss);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  const double inv = 1.0 / fmax(sqrt(ss), l2_eps);
  const double p = pq[row % t];
  const int hh = dc / 2;
  for (int j = lane; j < hh; j += 64) {
    double sn, cs;
    sincos(p * invf[j], &sn, &cs);
    const double a = q[j] * inv, b = q[j + hh] * inv;
    q[j] = a * cs - b * sn;
    q[j + hh] = b * cs + a * sn;
  }
}

struct Refine64Args {
  const float* K;        // [H][N][d] RoPE'd keys
  const float* V;        // [H][N][d] values
  const double* pos;     // [N] key positions
  const double* invf_b;  // [d/2] base-model RoPE frequencies
  const double* invf_c;  // [dc/2] compactor RoPE frequencies
  const float* W;        // [nc*dc][2d] W_K
  const float* bias;     // [nc*dc] b_K or NULL
  const double* Q;       // [H*t][nc*dc] normalised, rotated q (q64_finalize)
  const int* ridx;       // [H*nc][t*R] key of each slot
  const float* rval;     // [H*nc][t*R] fp32 logit of the flash pass (log2 units)
  const int* crow;       // [H*nc][t*R] compacted list: row -> slot
  const int* count;      // [H*nc]
  float2* rpart;         // [H*nc][t*R]: .x = exact logit - fp32 logit
  long N;
  int H, t, R, nc, dc, d;
  double scale_log2, l2_eps;
  int ntile;             // row tiles of BM per list in the grid (workgroups loop past it)
};

// Workgroup = BM = 16 candidate rows of one (h, c) list.  Their X rows are
// built in fp64 in LDS (base RoPE un-rotation with fp64 angles); the key
// projection runs over chunks of 32 RoPE pairs (64 widths), W_K chunks
// staged in LDS as fp64, thread (r, g) owning row r and pairs 2g, 2g + 1 of
// the chunk; its epilogue adds the bias, accumulates the sum of squares and
// the dot product of the rotated key with q.
template <int D>
__global__ __launch_bounds__(256) void refine64_kernel(Refine64Args a) {
  constexpr int BM = 16, PC = 32, KC = 32;   // rows, pairs per chunk, k per W stage
  constexpr int D2 = 2 * D;
  __shared__ double Xs[BM][D2 + 1];
  __shared__ double Ws[2 * PC][KC + 1];
  __shared__ int2 rinfo[BM];   // (key, latent)
  __shared__ int rslot[BM];
  const int tid = threadIdx.x;
  const int nb = a.H * a.nc;
  const int b = blockIdx.x % nb, rt0 = blockIdx.x / nb;
  const int h = b / a.nc, c = b - h * a.nc;
  const int cnt = a.count[b];
  const int TR = a.t * a.R;
  const int hh = a.dc / 2, hd = D / 2;
  const long Ec = (long)a.nc * a.dc;
  const int r = tid >> 4, g = tid & 15;
  for (int rt = rt0; rt * BM < cnt; rt += a.ntile) {
    const int r0 = rt * BM;
    __syncthreads();   // previous tile's LDS reads done
    if (tid < BM) {
      int key = 0, lat = 0, slot = -1;
      if (r0 + tid < cnt) {
        slot = a.crow[(long)b * TR + r0 + tid];
        key = max(a.ridx[(long)b * TR + slot], 0);
        lat = slot / a.R;
      }
      rinfo[tid] = make_int2(key, lat);
      rslot[tid] = slot;
    }
    __syncthreads();
    // X rows: [R(-p) K ; V] in fp64
    for (int e = tid; e < BM * hd; e += 256) {
      const int rr = e / hd, j = e - rr * hd;
      const long n = rinfo[rr].x;
      const float* kr = a.K + ((long)h * a.N + n) * D;
      const float* vr = a.V + ((long)h * a.N + n) * D;
      double sn, cs;
      sincos(a.pos[n] * a.invf_b[j], &sn, &cs);
      const double k0 = kr[j], k1 = kr[j + hd];
      Xs[rr][j] = k0 * cs + k1 * sn;
      Xs[rr][j + hd] = k1 * cs - k0 * sn;
      Xs[rr][D + j] = vr[j];
      Xs[rr][D + j + hd] = vr[j + hd];
    }
    double dot = 0.0, ss = 0.0;
    const long key = rinfo[r].x;
    const double pk = a.pos[key];
    const double* qrow = a.Q + ((long)h * a.t + rinfo[r].y) * Ec + (long)c * a.dc;
    for (int p0 = 0; p0 < hh; p0 += PC) {
      double acc[2][2] = {{0.0, 0.0}, {0.0, 0.0}};   // [pair][member]
      for (int k0 = 0; k0 < D2; k0 += KC) {
        __syncthreads();
        // W_K rows of the chunk: local row q < PC -> width p0 + q, q >= PC -> width p0 + q - PC + dc/2
        for (int e = tid; e < 2 * PC * KC; e += 256) {
          const int q = e / KC, k = e - q * KC;
          const int width = q < PC ? p0 + q : p0 + (q - PC) + hh;
          double v = 0.0;
          if (p0 + (q % PC) < hh) v = a.W[((long)c * a.dc + width) * D2 + k0 + k];
          Ws[q][k] = v;
        }
        __syncthreads();
#pragma unroll 8
        for (int k = 0; k < KC; ++k) {
          const double x = Xs[r][k0 + k];
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            acc[u][0] = fma(x, Ws[2 * g + u][k], acc[u][0]);
            acc[u][1] = fma(x, Ws[PC + 2 * g + u][k], acc[u][1]);
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int j = p0 + 2 * g + u;
        if (j >= hh) continue;
        const double v0 = acc[u][0] + (a.bias ? (double)a.bias[(long)c * a.dc + j] : 0.0);
        const double v1 = acc[u][1] + (a.bias ? (double)a.bias[(long)c * a.dc + j + hh] : 0.0);
        ss = fma(v0, v0, fma(v1, v1, ss));
        double sn, cs;
        sincos(pk * a.invf_c[j], &sn, &cs);
        dot += (v0 * cs - v1 * sn) * qrow[j] + (v1 * cs + v0 * sn) * qrow[j + hh];
      }
    }
    // the 16 threads of a row are 16 consecutive lanes
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) {
      dot += __shfl_xor(dot, o);
      ss += __shfl_xor(ss, o);
    }
    if (g == 0 && rslot[r] >= 0) {
      const long sl = (long)b * TR + rslot[r];
      const double logit = a.scale_log2 * dot / fmax(sqrt(ss), a.l2_eps);
      a.rpart[sl] = make_float2((float)(logit - (double)a.rval[sl]), 0.f);
    }
  }
}

}  // namespace still
