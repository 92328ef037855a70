// attn.hpp - flash-style latent -> cache cross-attention (one KV head h, one
// cross head c per grid row), split over the key axis.
//
// For a tile of TT latents and a key range, stream key blocks of NB keys:
//   S^T = K_blk Q^T              (contraction over the head width, MFMA)
//   logits = S^T * rk[key] * rq[lat] * s * log2(e)   (QK-norm folded in)
//   online softmax over keys (running max m, running sum l per latent)
//   O^T += X_blk^T P^T           (contraction over the block's keys, MFMA)
// and write the un-normalised partial (O, m, l) of the key range.  The value
// projection W_V is applied afterwards to the merged O = P X (exact
// re-association of P (X W_V)).
//
// Orientation: keys are MFMA rows and latents MFMA columns in the first
// product, so every lane owns one latent and the softmax statistics stay in
// the lane; the S^T accumulator is then already a valid B operand of the
// second product once the block's keys are read from X^T in the matching
// (permuted) order.
#pragma once
#include "common.hpp"

namespace still {

struct AttnArgs {
  const void* q;     // [H*t][nc*dc]  rotated, un-normalised queries (CT)
  long ldq;
  const float* rq;   // [H*t][nc]     1 / max(||q~||, eps)
  const void* k;     // [H*N][nc*dc]  rotated, un-normalised keys (CT)
  long ldk;
  const float* rk;   // [H*N][nc]
  const void* xt;    // [H][2d][ldxt] X^T (CT), zero beyond N up to ldxt
  long ldxt;
  float* opart;      // [S][H*nc][t][2d]
  float* mpart;      // [S][H*nc][t]
  float* lpart;      // [S][H*nc][t]
  int H, N, t, nc, dc, d2;
  float scale_log2;  // logit scale * log2(e)
  int keys_per_split;
  float* cval;       // TOPK > 0: [S][H*nc][t][2*TOPK] largest logits seen (log2 units) ...
  int* cidx;         // ... and their key indices (-1 = none), per half-lane
};

template <class CT, int TT, int NB, int DK, int D2, int TOPK>
__global__ __launch_bounds__(256) void cross_attn_kernel(AttnArgs a) {
  typedef Mma<CT> MM;
  typedef typename MM::frag frag;
  constexpr int E = MM::E;
  constexpr int PAD = 16 / sizeof(CT);
  constexpr int LQ = DK + PAD;           // Q/K stage row stride
  constexpr int LX = NB + PAD;           // X^T block row stride
  constexpr int KT = NB / 32;            // key tiles per block
  constexpr int FT = D2 / 32;            // feature tiles
  constexpr int QV = TT * DK / E / 256;  // stage vectors per thread
  constexpr int KVv = NB * DK / E / 256;
  constexpr int XV = D2 * NB / E / 256;
  static_assert(TT == 128, "4 waves x 32 latents");
  static_assert(QV >= 1 && KVv >= 1 && XV >= 1, "tile sizes");

  __shared__ __attribute__((aligned(16))) CT Qs[2][TT * LQ];
  __shared__ __attribute__((aligned(16))) CT Ks[2][NB * LQ];
  __shared__ __attribute__((aligned(16))) CT Xs[D2 * LX];
  __shared__ float rks[NB];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, lg = lane >> 5;
  const int hc = blockIdx.y, h = hc / a.nc, c = hc - h * a.nc;
  const int t0 = blockIdx.x * TT;
  const int split = blockIdx.z;
  const int nbeg = split * a.keys_per_split;
  const int nend = min(a.N, nbeg + a.keys_per_split);

  const CT* qbase = (const CT*)a.q + (long)h * a.t * a.ldq + (long)c * a.dc;
  const CT* kbase = (const CT*)a.k + (long)h * a.N * a.ldk + (long)c * a.dc;
  const CT* xtb = (const CT*)a.xt + (long)h * a.d2 * a.ldxt;
  const float* rkb = a.rk + (long)h * a.N * a.nc + c;

  const int my_lat = t0 + wave * 32 + l32;
  const float rq = my_lat < a.t ? a.rq[((long)h * a.t + my_lat) * a.nc + c] : 0.f;
  const float qscale = rq * a.scale_log2;

  f32x16 o[FT];
#pragma unroll
  for (int f = 0; f < FT; ++f) o[f] = zero16();
  float m_run = -INFINITY, l_run = 0.f;
  // top-TOPK keys of this lane's half of the key range, by logit (descending)
  float tv[TOPK > 0 ? TOPK : 1];
  int ti[TOPK > 0 ? TOPK : 1];
#pragma unroll
  for (int q = 0; q < (TOPK > 0 ? TOPK : 1); ++q) {
    tv[q] = -INFINITY;
    ti[q] = -1;
  }

  frag rq_[QV], rk_[KVv], rx[XV];
  auto load_qk = [&](int n0, int d0) {
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int v = tid + i * 256, r = v / (DK / E), kk = (v % (DK / E)) * E;
      const int lat = t0 + r;
      rq_[i] = lat < a.t ? *(const frag*)(qbase + (long)lat * a.ldq + d0 + kk) : zero_frag<CT>();
    }
#pragma unroll
    for (int i = 0; i < KVv; ++i) {
      const int v = tid + i * 256, r = v / (DK / E), kk = (v % (DK / E)) * E;
      const int n = n0 + r;
      rk_[i] = n < nend ? *(const frag*)(kbase + (long)n * a.ldk + d0 + kk) : zero_frag<CT>();
    }
  };
  auto store_qk = [&](int buf) {
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int v = tid + i * 256, r = v / (DK / E), kk = (v % (DK / E)) * E;
      *(frag*)&Qs[buf][r * LQ + kk] = rq_[i];
    }
#pragma unroll
    for (int i = 0; i < KVv; ++i) {
      const int v = tid + i * 256, r = v / (DK / E), kk = (v % (DK / E)) * E;
      *(frag*)&Ks[buf][r * LQ + kk] = rk_[i];
    }
  };
  auto load_x = [&](int n0) {
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = tid + i * 256, f = v / (NB / E), kk = (v % (NB / E)) * E;
      rx[i] = *(const frag*)(xtb + (long)f * a.ldxt + n0 + kk);   // padded: always in bounds
    }
  };

  const int nd = a.dc / DK;
  for (int n0 = nbeg; n0 < nend; n0 += NB) {
    // ---- S^T = K_blk Q^T over the head width
    f32x16 s[KT];
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) s[kt] = zero16();
    load_x(n0);
    load_qk(n0, 0);
    store_qk(0);
    __syncthreads();
    for (int di = 0; di < nd; ++di) {
      const int cur = di & 1;
      if (di + 1 < nd) load_qk(n0, (di + 1) * DK);
#pragma unroll
      for (int ks = 0; ks < DK / (2 * E); ++ks) {
        const frag bq = *(const frag*)&Qs[cur][(wave * 32 + l32) * LQ + ks * 2 * E + lg * E];
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) {
          const frag ak = *(const frag*)&Ks[cur][(kt * 32 + l32) * LQ + ks * 2 * E + lg * E];
          MM::mma(s[kt], ak, bq);
        }
      }
      if (di + 1 < nd) store_qk(cur ^ 1);
      __syncthreads();
    }
    // ---- stage X^T block and the key norms
#pragma unroll
    for (int i = 0; i < XV; ++i) {
      const int v = tid + i * 256, f = v / (NB / E), kk = (v % (NB / E)) * E;
      *(frag*)&Xs[f * LX + kk] = rx[i];
    }
    if (tid < NB) {
      const int n = n0 + tid;
      rks[tid] = n < nend ? rkb[(long)n * a.nc] : 0.f;
    }
    __syncthreads();

    // ---- online softmax (lane owns latent my_lat; keys in registers)
    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int kl = kt * 32 + 8 * (j >> 2) + 4 * lg + (j & 3);
        float x = s[kt][j] * rks[kl] * qscale;
        x = (n0 + kl < nend) ? x : -INFINITY;
        s[kt][j] = x;
        mx = fmaxf(mx, x);
        if constexpr (TOPK > 0) {
          if (x > tv[TOPK - 1]) {
            float v = x;
            int id = n0 + kl;
#pragma unroll
            for (int q = 0; q < TOPK; ++q) {
              const bool gt = v > tv[q];
              const float tvq = tv[q];
              const int tiq = ti[q];
              tv[q] = gt ? v : tvq;
              ti[q] = gt ? id : tiq;
              v = gt ? tvq : v;
              id = gt ? tiq : id;
            }
          }
        }
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = (m_new == -INFINITY) ? 1.f : exp2f(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = (m_new == -INFINITY) ? 0.f : exp2f(s[kt][j] - m_new);
        s[kt][j] = p;
        psum += p;
      }
    psum += __shfl_xor(psum, 32);
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int f = 0; f < FT; ++f)
#pragma unroll
      for (int j = 0; j < 16; ++j) o[f][j] *= alpha;

    // ---- O^T += X^T P^T
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      if constexpr (E == 8) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          half8 bp;
#pragma unroll
          for (int e = 0; e < 8; ++e) bp[e] = (f16)s[kt][8 * hf + e];
          const int key0 = kt * 32 + 16 * hf + 4 * lg;   // keys key0..+3 and key0+8..+11
#pragma unroll
          for (int f = 0; f < FT; ++f) {
            const CT* xr = &Xs[(f * 32 + l32) * LX];
            const half4 lo = *(const half4*)(xr + key0);
            const half4 hi = *(const half4*)(xr + key0 + 8);
            half8 ax;
            ax[0] = lo[0]; ax[1] = lo[1]; ax[2] = lo[2]; ax[3] = lo[3];
            ax[4] = hi[0]; ax[5] = hi[1]; ax[6] = hi[2]; ax[7] = hi[3];
            MM::mma(o[f], *(const frag*)&ax, *(const frag*)&bp);
          }
        }
      } else {
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) {
          frag bp;
#pragma unroll
          for (int e = 0; e < 4; ++e) bp[e] = s[kt][4 * qd + e];
          const int key0 = kt * 32 + 8 * qd + 4 * lg;     // keys key0..+3
#pragma unroll
          for (int f = 0; f < FT; ++f) {
            const frag ax = *(const frag*)&Xs[(f * 32 + l32) * LX + key0];
            MM::mma(o[f], ax, bp);
          }
        }
      }
    }
  }

  // ---- write the partial (O un-normalised, m, l) of this key range
  if (my_lat < a.t) {
    const long row = ((long)split * a.H * a.nc + hc) * a.t + my_lat;
    float* op = a.opart + row * a.d2;
#pragma unroll
    for (int f = 0; f < FT; ++f)
#pragma unroll
      for (int j = 0; j < 16; ++j) op[f * 32 + 8 * (j >> 2) + 4 * lg + (j & 3)] = o[f][j];
    if (lg == 0) {
      a.mpart[row] = m_run;
      a.lpart[row] = l_run;
    }
    if constexpr (TOPK > 0) {
#pragma unroll
      for (int q = 0; q < TOPK; ++q) {
        a.cval[row * (2 * TOPK) + lg * TOPK + q] = tv[q];
        a.cidx[row * (2 * TOPK) + lg * TOPK + q] = ti[q];
      }
    }
  }
}

}  // namespace still

namespace still {

// ---------------------------------------------------------------------------
// fp16 cross-attention, workgroup = TT latents x one key range, 4 waves.
// Key blocks of 256: wave w owns keys [64w, 64w+64) of the block in the QK
// product and output features [w*D2/4, (w+1)*D2/4) in the P.X product.
//   QK:  S^T[key][lat] over the head width in chunks of DK.  K fragments are
//        loaded from global memory straight into registers (each key row is
//        read once per workgroup); Q chunks are staged through LDS and shared
//        by the 4 waves.  Within a chunk, lane half g holds the contiguous run
//        [g*DK/2, (g+1)*DK/2) of the head width, so MFMA step s pairs element
//        e of both operands with width index g*DK/2 + 8s + e (any fixed
//        pairing contracts every index once).
//   softmax: per-latent block maxima combined across the waves through LDS;
//        P (fp16) written to LDS as [latent][key].
//   P.X: O^T[feat][lat] += X^T[feat][key] P^T[key][lat]; X^T fragments from
//        global memory (64-byte runs of keys per lane half), P from LDS.
// 1-D grid ordered so that the t tiles of one (KV head, cross head, split)
// are consecutive workgroups of one XCD: they read the same keys through
// that XCD's L2.
// ---------------------------------------------------------------------------
template <int TT, int DK, int D2, int TOPK>
__global__ __launch_bounds__(256) void xattn_f16_kernel(AttnArgs a) {
  constexpr int LT = TT / 32;            // latent tiles
  constexpr int KB = 256;                // keys per block
  constexpr int FW = D2 / 4;             // output features per wave
  constexpr int FT = FW / 32;            // feature tiles per wave
  constexpr int NS = DK / 16;            // MFMA steps per chunk
  constexpr int LQ = DK + 8;             // Q stage row stride (halfs)
  constexpr int LP = KB + 8;             // P row stride (halfs)
  constexpr int QV = TT * DK / 8 / 256;  // Q stage vectors per thread
  static_assert(FT >= 1 && QV >= 1 && NS >= 1, "tile sizes");

  __shared__ __attribute__((aligned(16))) f16 Qs[2][TT * LQ];
  __shared__ __attribute__((aligned(16))) f16 Ps[TT * LP];
  __shared__ float red_m[4][TT], red_l[4][TT];
  __shared__ float rks[KB];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, lg = lane >> 5;

  const int ntt = (a.t + TT - 1) / TT, HC = a.H * a.nc;
  const int total = gridDim.x;
  int L = blockIdx.x;
  if ((total & 7) == 0) L = (L & 7) * (total >> 3) + (L >> 3);
  const int tt = L % ntt, rest = L / ntt;
  const int hc = rest % HC, split = rest / HC;
  const int h = hc / a.nc, c = hc - h * a.nc;
  const int t0 = tt * TT;
  const int nbeg = split * a.keys_per_split;
  const int nend = min(a.N, nbeg + a.keys_per_split);

  const f16* qb = (const f16*)a.q + (long)h * a.t * a.ldq + (long)c * a.dc;
  const f16* kb = (const f16*)a.k + (long)h * a.N * a.ldk + (long)c * a.dc;
  const f16* xtb = (const f16*)a.xt + (long)h * a.d2 * a.ldxt;
  const float* rkb = a.rk + (long)h * a.N * a.nc + c;

  // q arrives pre-scaled by 1/||q~|| * scale * log2(e) (qprescale_kernel), so a
  // logit in log2 units is S^T * rk[key]
  float m_run[LT], l_run[LT];
#pragma unroll
  for (int lt = 0; lt < LT; ++lt) {
    m_run[lt] = -INFINITY;
    l_run[lt] = 0.f;
  }
  f32x16 o[FT][LT];
#pragma unroll
  for (int f = 0; f < FT; ++f)
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) o[f][lt] = zero16();
  float tv[LT][TOPK > 0 ? TOPK : 1];
  int ti[LT][TOPK > 0 ? TOPK : 1];
#pragma unroll
  for (int lt = 0; lt < LT; ++lt)
#pragma unroll
    for (int q = 0; q < (TOPK > 0 ? TOPK : 1); ++q) {
      tv[lt][q] = -INFINITY;
      ti[lt][q] = -1;
    }

  half8 qreg[QV];
  auto load_q = [&](int d0) {
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int v = tid + i * 256, r = v / (DK / 8), kk = (v % (DK / 8)) * 8;
      const int lat = t0 + r;
      qreg[i] = lat < a.t ? *(const half8*)(qb + (long)lat * a.ldq + d0 + kk) : zero_frag<f16>();
    }
  };
  auto store_q = [&](int buf) {
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int v = tid + i * 256, r = v / (DK / 8), kk = (v % (DK / 8)) * 8;
      *(half8*)&Qs[buf][r * LQ + kk] = qreg[i];
    }
  };
  // K fragments of this wave's 64 keys for one chunk: [key tile][step]
  auto load_k = [&](half8 (&kr)[2][NS], int n0, int d0) {
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      const int n = n0 + 64 * w + 32 * kt + l32;
      const f16* src = kb + (long)n * a.ldk + d0 + (DK / 2) * lg;
#pragma unroll
      for (int s = 0; s < NS; ++s) kr[kt][s] = n < nend ? *(const half8*)(src + 8 * s) : zero_frag<f16>();
    }
  };
  // X^T fragments for P.X step group s4: [feature tile][step]
  auto load_x = [&](half8 (&xr)[FT][4], int n0, int s4) {
#pragma unroll
    for (int f = 0; f < FT; ++f) {
      const int fr = FW * w + 32 * f + l32;
      const f16* src = xtb + (long)fr * a.ldxt + n0 + 64 * s4 + 32 * lg;
#pragma unroll
      for (int s = 0; s < 4; ++s) xr[f][s] = *(const half8*)(src + 8 * s);   // X^T padded to the block size
    }
  };

  const int nd = a.dc / DK;   // even (checked on the host)
  half8 kA[2][NS], kB[2][NS];
  half8 xA[FT][4], xB[FT][4];
  for (int n0 = nbeg; n0 < nend; n0 += KB) {
    f32x16 s[LT][2];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) s[lt][0] = s[lt][1] = zero16();
    load_q(0);
    load_k(kA, n0, 0);
    store_q(0);
    {
      const int n = n0 + tid;
      rks[tid] = n < nend ? rkb[(long)n * a.nc] : 0.f;
    }
    __syncthreads();
    auto chunk = [&](int ci, half8 (&kc)[2][NS], half8 (&kn)[2][NS]) {
      const int cur = ci & 1;
      const bool more = ci + 1 < nd;
      if (more) {
        load_q((ci + 1) * DK);
        load_k(kn, n0, (ci + 1) * DK);
      } else {
        load_x(xA, n0, 0);
      }
#pragma unroll
      for (int st = 0; st < NS; ++st) {
#pragma unroll
        for (int lt = 0; lt < LT; ++lt) {
          const half8 bq = *(const half8*)&Qs[cur][(32 * lt + l32) * LQ + (DK / 2) * lg + 8 * st];
#pragma unroll
          for (int kt = 0; kt < 2; ++kt)
            s[lt][kt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kc[kt][st], bq, s[lt][kt], 0, 0, 0);
        }
      }
      if (more) store_q(cur ^ 1);
      __syncthreads();
    };
    for (int ci = 0; ci < nd; ci += 2) {
      chunk(ci, kA, kB);
      chunk(ci + 1, kB, kA);
    }

    // ---- softmax statistics for the block
    float rkv[2][16];
    const bool tail = n0 + KB > nend;    // keys past the range only in a split's last block
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int kl = 64 * w + 32 * kt + 8 * (j >> 2) + 4 * lg + (j & 3);
        rkv[kt][j] = (tail && n0 + kl >= nend) ? -INFINITY : rks[kl];
      }
    float mx[LT];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) {
      mx[lt] = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int kl = 64 * w + 32 * kt + 8 * (j >> 2) + 4 * lg + (j & 3);
          float x = s[lt][kt][j] * rkv[kt][j];   // masked keys carry rk = -inf (S may be 0)
          x = (rkv[kt][j] == -INFINITY) ? -INFINITY : x;
          s[lt][kt][j] = x;
          mx[lt] = fmaxf(mx[lt], x);
          if constexpr (TOPK > 0) {
            if (x > tv[lt][TOPK - 1]) {
              float v = x;
              int id = n0 + kl;
#pragma unroll
              for (int q = 0; q < TOPK; ++q) {
                const bool gt = v > tv[lt][q];
                const float tq = tv[lt][q];
                const int iq = ti[lt][q];
                tv[lt][q] = gt ? v : tq;
                ti[lt][q] = gt ? id : iq;
                v = gt ? tq : v;
                id = gt ? iq : id;
              }
            }
          }
        }
      mx[lt] = fmaxf(mx[lt], __shfl_xor(mx[lt], 32));
      if (lg == 0) red_m[w][32 * lt + l32] = mx[lt];
    }
    __syncthreads();
    float alpha[LT];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) {
      const int li = 32 * lt + l32;
      const float mb = fmaxf(fmaxf(red_m[0][li], red_m[1][li]), fmaxf(red_m[2][li], red_m[3][li]));
      const float m_new = fmaxf(m_run[lt], mb);
      alpha[lt] = (m_new == -INFINITY) ? 1.f : exp2f(m_run[lt] - m_new);
      float ps = 0.f;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int jq = 0; jq < 4; ++jq) {
          half4 pv;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float p = (m_new == -INFINITY) ? 0.f : exp2f(s[lt][kt][4 * jq + u] - m_new);
            ps += p;
            pv[u] = (f16)p;
          }
          *(half4*)&Ps[li * LP + 64 * w + 32 * kt + 8 * jq + 4 * lg] = pv;
        }
      ps += __shfl_xor(ps, 32);
      if (lg == 0) red_l[w][li] = ps;
      m_run[lt] = m_new;
      // rescale only when some latent of the tile saw a new maximum
      if (__any(alpha[lt] != 1.f)) {
#pragma unroll
        for (int f = 0; f < FT; ++f)
#pragma unroll
          for (int j = 0; j < 16; ++j) o[f][lt][j] *= alpha[lt];
      }
    }
    __syncthreads();
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) {
      const int li = 32 * lt + l32;
      l_run[lt] = l_run[lt] * alpha[lt] + (red_l[0][li] + red_l[1][li]) + (red_l[2][li] + red_l[3][li]);
    }

    // ---- O^T += X^T P^T over the block's 256 keys
    auto xstep = [&](int s4, half8 (&xc)[FT][4], half8 (&xn)[FT][4]) {
      if (s4 + 1 < 4) load_x(xn, n0, s4 + 1);
#pragma unroll
      for (int st = 0; st < 4; ++st) {
#pragma unroll
        for (int lt = 0; lt < LT; ++lt) {
          const half8 bp = *(const half8*)&Ps[(32 * lt + l32) * LP + 64 * s4 + 32 * lg + 8 * st];
#pragma unroll
          for (int f = 0; f < FT; ++f)
            o[f][lt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(xc[f][st], bp, o[f][lt], 0, 0, 0);
        }
      }
    };
    xstep(0, xA, xB);
    xstep(1, xB, xA);
    xstep(2, xA, xB);
    xstep(3, xB, xA);
  }

  // ---- partial (O un-normalised, m, l) and the top keys of this key range
#pragma unroll
  for (int lt = 0; lt < LT; ++lt) {
    const int lat = t0 + 32 * lt + l32;
    if (lat >= a.t) continue;
    const long row = ((long)split * HC + hc) * a.t + lat;
    float* op = a.opart + row * a.d2;
#pragma unroll
    for (int f = 0; f < FT; ++f)
#pragma unroll
      for (int j = 0; j < 16; ++j) op[FW * w + 32 * f + 8 * (j >> 2) + 4 * lg + (j & 3)] = o[f][lt][j];
    if (w == 0 && lg == 0) {
      a.mpart[row] = m_run[lt];
      a.lpart[row] = l_run[lt];
    }
    if constexpr (TOPK > 0) {
#pragma unroll
      for (int q = 0; q < TOPK; ++q) {
        a.cval[row * (8 * TOPK) + (2 * w + lg) * TOPK + q] = tv[lt][q];
        a.cidx[row * (8 * TOPK) + (2 * w + lg) * TOPK + q] = ti[lt][q];
      }
    }
  }
}

}  // namespace still

