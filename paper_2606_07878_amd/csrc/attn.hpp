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
// fp16 cross-attention, workgroup = TT latents x one key range, NW waves.
// Key blocks of KB (256 or 512): wave w owns keys [w*KB/NW, (w+1)*KB/NW) of the block
// in the QK product and output features [w*D2/NW, (w+1)*D2/NW) in the P.X
// product (8 waves keep each wave's accumulators small enough for two waves
// per SIMD).
//   QK:  S^T[key][lat] over the head width.  Q is staged through LDS in
//        chunks of QC (one barrier per chunk) and shared by the waves.  K
//        fragments go from global memory straight into registers (each key
//        row is read once per workgroup) in groups of 32 of the head width,
//        through a ring of QC/32 groups: the group used now is reloaded with
//        the same group of the next chunk, so every K load has a whole chunk
//        of MFMA work to arrive.  Within a group, lane half g holds the
//        contiguous run [16g, 16g + 16), so MFMA step s pairs element e of
//        both operands with width index 16g + 8s + e (any fixed pairing
//        contracts every index once).
//   softmax: per-latent block maxima combined across the waves through LDS;
//        P (fp16) written to LDS as [latent][key].
//   P.X: O^T[feat][lat] += X^T[feat][key] P^T[key][lat]; X^T fragments from
//        global memory (64-byte runs of keys per lane half), P from LDS.
// 1-D grid ordered so that the t tiles of one (KV head, cross head, split)
// are consecutive workgroups of one XCD: they read the same keys through
// that XCD's L2.
// ---------------------------------------------------------------------------
template <int TT, int QC, int D2, int TOPK, int NW, int KB = 256>
__global__ __launch_bounds__(64 * NW) void xattn_f16_kernel(AttnArgs a) {
  constexpr int LT = TT / 32;            // latent tiles
  constexpr int NT = 64 * NW;            // threads
  constexpr int KW = KB / NW;            // keys per wave (QK)
  constexpr int KT = KW / 32;            // key tiles per wave
  constexpr int FW = D2 / NW;            // output features per wave
  constexpr int FT = FW / 32;            // feature tiles per wave
  constexpr int NBK = 2 * NW;            // top-key buckets per latent (wave, lane half)
  constexpr int G = 32;                  // head-width group of one K load (2 MFMA steps)
  constexpr int NG = QC / G;             // groups per Q chunk = depth of the K ring
  constexpr int LQ = QC + 8;             // Q stage row stride (halfs)
  constexpr int LP = KB + 8;             // P row stride (halfs)
  constexpr int QV = TT * QC / 8 / NT;   // Q stage vectors per thread
  static_assert(FT >= 1 && KT >= 1 && QV >= 1 && NG >= 1 && (TT * QC / 8) % NT == 0, "tile sizes");

  __shared__ __attribute__((aligned(16))) f16 Qs[2][TT * LQ];
  __shared__ __attribute__((aligned(16))) f16 Ps[TT * LP];
  __shared__ float red_m[TT][NW], red_l[TT][NW];
  __shared__ float2 rks[KB];   // (1/||k~||, 0) or (0, -inf) past the key range

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int l32 = lane & 31, lg = lane >> 5;

  const int ntt = (a.t + TT - 1) / TT, HC = a.H * a.nc;
  const int total = gridDim.x;
  int L = blockIdx.x;
  if ((total & 7) == 0) L = (L & 7) * (total >> 3) + (L >> 3);
  // order: latent tile fastest, then split, then (KV head, cross head): the
  // workgroups an XCD runs at once share one Q tile set and few key ranges
  const int S = total / (ntt * HC);
  const int tt = L % ntt, rest = L / ntt;
  const int split = rest % S, hc = rest / S;
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
  // Candidate keys for the logit refinement: each lane keeps, per latent
  // tile, a sorted list of its TOPK largest logits (bucket = wave, lane half)
  // in the output arrays cval/cidx (only the lane itself touches its list),
  // and in a register the list's smallest entry.  Keys below the running
  // maximum minus REFINE_MARGIN can never be selected and are skipped, which
  // makes list updates rare.
  float th[LT];
#pragma unroll
  for (int lt = 0; lt < LT; ++lt) {
    th[lt] = -INFINITY;
    const int lat = t0 + 32 * lt + l32;
    if (TOPK > 0 && lat < a.t) {
      const long row = ((long)split * HC + hc) * a.t + lat;
#pragma unroll
      for (int q = 0; q < (TOPK > 0 ? TOPK : 1); ++q) {
        a.cval[row * (NBK * TOPK) + (2 * w + lg) * TOPK + q] = -INFINITY;
        a.cidx[row * (NBK * TOPK) + (2 * w + lg) * TOPK + q] = -1;
      }
    }
  }

  // Loads address uniform bases (q, k, X^T of this head) with 32-bit element
  // offsets (the host bounds them), and are branch-free: rows past the end
  // read the last valid row, whose values are then zeroed (Q) or masked out
  // of the softmax (K), so the number of loads in flight stays static.
  half8 qreg[QV];
  auto load_q = [&](int d0) {
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int v = tid + i * NT, r = v / (QC / 8), kk = (v % (QC / 8)) * 8;
      const unsigned lat = (unsigned)min(t0 + r, a.t - 1);
      qreg[i] = *(const half8*)(qb + (lat * (unsigned)a.ldq + (unsigned)(d0 + kk)));
    }
  };
  auto store_q = [&](int buf) {
#pragma unroll
    for (int i = 0; i < QV; ++i) {
      const int v = tid + i * NT, r = v / (QC / 8), kk = (v % (QC / 8)) * 8;
      *(half8*)&Qs[buf][r * LQ + kk] = (t0 + r < a.t) ? qreg[i] : zero_frag<f16>();
    }
  };
  // K fragments of this wave's keys for one group of 32: [key tile][step]
  unsigned krow[KT];
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) krow[kt] = 0;
  auto set_krows = [&](int n0) {
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) {
      const unsigned n = (unsigned)min(n0 + KW * w + 32 * kt + l32, nend - 1);
      krow[kt] = n * (unsigned)a.ldk + 16u * lg;
    }
  };
  auto load_kg = [&](half8 (&kr)[KT][2], int d0) {
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int s = 0; s < 2; ++s) kr[kt][s] = *(const half8*)(kb + (krow[kt] + (unsigned)(d0 + 8 * s)));
  };
  // X^T fragments for P.X step group s4: [feature tile][step]
  auto load_x = [&](half8 (&xr)[FT][4], int n0, int s4) {
#pragma unroll
    for (int f = 0; f < FT; ++f) {
      const unsigned fr = FW * w + 32 * f + l32;
      const unsigned off = fr * (unsigned)a.ldxt + (unsigned)(n0 + 64 * s4 + 32 * lg);
#pragma unroll
      for (int s = 0; s < 4; ++s) xr[f][s] = *(const half8*)(xtb + (off + 8u * s));   // X^T padded to the block size
    }
  };

  const int nch = a.dc / QC;   // a.dc is a multiple of QC (checked on the host)
  half8 kr[NG][KT][2];
  half8 xA[FT][4], xB[FT][4];
  for (int n0 = nbeg; n0 < nend; n0 += KB) {
    f32x16 s[LT][KT];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt)
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) s[lt][kt] = zero16();
    load_q(0);
    set_krows(n0);
#pragma unroll
    for (int gi = 0; gi < NG; ++gi) load_kg(kr[gi], gi * G);
    store_q(0);
    for (int i = tid; i < KB; i += NT) {
      const int n = n0 + i;
      rks[i] = n < nend ? make_float2(rkb[(long)n * a.nc], 0.f) : make_float2(0.f, -INFINITY);
    }
    __syncthreads();
    for (int c = 0; c < nch; ++c) {
      const int cur = c & 1;
      const bool more = c + 1 < nch;
      if (more) load_q((c + 1) * QC);
      else load_x(xA, n0, 0);
#pragma unroll
      for (int gi = 0; gi < NG; ++gi) {
#pragma unroll
        for (int st = 0; st < 2; ++st) {
#pragma unroll
          for (int lt = 0; lt < LT; ++lt) {
            const half8 bq = *(const half8*)&Qs[cur][(32 * lt + l32) * LQ + gi * G + 16 * lg + 8 * st];
#pragma unroll
            for (int kt = 0; kt < KT; ++kt)
              s[lt][kt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kr[gi][kt][st], bq, s[lt][kt], 0, 0, 0);
          }
        }
        if (more) load_kg(kr[gi], (c + 1) * QC + gi * G);
      }
      if (more) store_q(cur ^ 1);
      __syncthreads();
    }

    // ---- softmax statistics for the block: logit (log2 units) = S * rk + mask
    float mx[LT], lmx[LT];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) mx[lt] = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        // keys KW*w + 32*kt + 8*jq + 4*lg + (0..3): two 16-byte LDS reads
        const float4 r01 = *(const float4*)&rks[KW * w + 32 * kt + 8 * jq + 4 * lg];
        const float4 r23 = *(const float4*)&rks[KW * w + 32 * kt + 8 * jq + 4 * lg + 2];
        const float rk[4] = {r01.x, r01.z, r23.x, r23.z}, mk[4] = {r01.y, r01.w, r23.y, r23.w};
#pragma unroll
        for (int lt = 0; lt < LT; ++lt) {
#pragma unroll
          for (int u = 0; u < 4; ++u) s[lt][kt][4 * jq + u] = fmaf(s[lt][kt][4 * jq + u], rk[u], mk[u]);
          mx[lt] = fmaxf(fmaxf(mx[lt], fmaxf(s[lt][kt][4 * jq], s[lt][kt][4 * jq + 1])),
                         fmaxf(s[lt][kt][4 * jq + 2], s[lt][kt][4 * jq + 3]));
        }
      }
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) {
      lmx[lt] = mx[lt];
      mx[lt] = fmaxf(mx[lt], __shfl_xor(mx[lt], 32));
      if (lg == 0) red_m[32 * lt + l32][w] = mx[lt];
    }
    __syncthreads();
    float alpha[LT];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) {
      const int li = 32 * lt + l32;
      float mb = red_m[li][0];
#pragma unroll
      for (int u = 1; u < NW; ++u) mb = fmaxf(mb, red_m[li][u]);
      const float m_new = fmaxf(m_run[lt], mb);
      const float mref = (m_new == -INFINITY) ? 0.f : m_new;   // all keys masked so far: every p is 0
      alpha[lt] = __builtin_amdgcn_exp2f(m_run[lt] - mref);   // m_run = -inf -> 0 (o, l are 0 then)
      float ps = 0.f;
#pragma unroll
      for (int kt = 0; kt < KT; ++kt)
#pragma unroll
        for (int jq = 0; jq < 4; ++jq) {
          half4 pv;
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float p = __builtin_amdgcn_exp2f(s[lt][kt][4 * jq + u] - mref);
            ps += p;
            pv[u] = (f16)p;
          }
          *(half4*)&Ps[li * LP + KW * w + 32 * kt + 8 * jq + 4 * lg] = pv;
        }
      ps += __shfl_xor(ps, 32);
      if (lg == 0) red_l[li][w] = ps;
      if constexpr (TOPK > 0) {
        const float cut0 = m_new - REFINE_MARGIN;
        if (lmx[lt] > fmaxf(th[lt], cut0) && t0 + li < a.t) {   // rare: update this lane's list
          const long row = ((long)split * HC + hc) * a.t + t0 + li;
          float* cv = a.cval + row * (NBK * TOPK) + (2 * w + lg) * TOPK;
          int* ci = a.cidx + row * (NBK * TOPK) + (2 * w + lg) * TOPK;
          float tv[TOPK > 0 ? TOPK : 1];
          int ti[TOPK > 0 ? TOPK : 1];
#pragma unroll
          for (int q = 0; q < TOPK; ++q) {
            tv[q] = cv[q];
            ti[q] = ci[q];
          }
          for (int kt = 0; kt < KT; ++kt)
            for (int j = 0; j < 16; ++j) {
              float v = s[lt][kt][j];
              if (v > fmaxf(tv[TOPK - 1], cut0)) {
                int id = n0 + KW * w + 32 * kt + 8 * (j >> 2) + 4 * lg + (j & 3);
#pragma unroll
                for (int q = 0; q < TOPK; ++q) {
                  const bool gt = v > tv[q];
                  const float tq = tv[q];
                  const int iq = ti[q];
                  tv[q] = gt ? v : tq;
                  ti[q] = gt ? id : iq;
                  v = gt ? tq : v;
                  id = gt ? iq : id;
                }
              }
            }
#pragma unroll
          for (int q = 0; q < TOPK; ++q) {
            cv[q] = tv[q];
            ci[q] = ti[q];
          }
          th[lt] = tv[TOPK - 1];
        }
      }
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
      float lb = 0.f;
#pragma unroll
      for (int u = 0; u < NW; ++u) lb += red_l[li][u];
      l_run[lt] = l_run[lt] * alpha[lt] + lb;
    }

    // ---- O^T += X^T P^T over the block's KB keys, 64 at a time
    auto xstep = [&](int s4, half8 (&xc)[FT][4], half8 (&xn)[FT][4]) {
      if (s4 + 1 < KB / 64) load_x(xn, n0, s4 + 1);
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
#pragma unroll
    for (int s4 = 0; s4 < KB / 64; s4 += 2) {
      xstep(s4, xA, xB);
      xstep(s4 + 1, xB, xA);
    }
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
  }
}

}  // namespace still

