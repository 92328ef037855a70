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
  const void* k;     // rotated, un-normalised keys (CT): fp32 kernel [H*N][nc*dc] (row stride ldk),
  long ldk;          //   fp16 kernel the fragment-tiled layout (ktile_off) with npad keys per head
  const float* rk;   // [H*N][nc]
  const void* xt;    // X^T (CT), zero beyond N: fp32 kernel [H][2d][ldxt], fp16 kernel tiled (xtile_off)
  long ldxt;
  long npad;         // fp16 kernel: keys per head in the tiled layouts (a multiple of 256)
  long xfeat, xcoff; // fp16 kernel: features per KV head in the tiled values and the first
                     //   feature of head c at c * xcoff (cross-attention: 2d and 0, every head
                     //   reads all of X; self-attention: n_s * d_s and d_s, one value slice per head)
  float* opart;      // [S][H*nc][t][2d]
  float* mpart;      // [S][H*nc][t]
  float* lpart;      // [S][H*nc][t]
  int H, N, t, nc, dc, d2;
  float scale_log2;  // logit scale * log2(e)
  int keys_per_split;
  float* cval;       // TOPK > 0: [S][H*nc][t][ncand] largest logits seen (log2 units) ...
  int* cidx;         // ... and their key indices (-1 = none): the per-list entries (fp32
                     // kernel: 2 TOPK, one list per lane half; fp16 kernel: NBK*TOPK, one
                     // per bucket), then up to ATT_OVF / XATT_OVF overflow entries
  int* ocnt;         // [S][H*nc][t] overflow entries written per row
};

// Overflow capacity per (split, latent row): in-margin keys that a full
// register list rejects or evicts (exact ties of duplicated cache rows, or
// more near-maximal keys per lane than the list holds).  Keys enter while
// they are within the margin of the running maximum, so early blocks can
// fill it with keys that a later, larger maximum leaves outside the margin;
// the capacity is sized for that (a cache of 32-fold duplicated rows writes
// several hundred entries to some rows).
constexpr int XATT_OVF = 1536;   // fp16 kernel
constexpr int ATT_OVF = 1536;    // fp32 kernel

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
  __shared__ int ovn[TT];   // overflow entries of each latent row

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
  if (tid < TT) ovn[tid] = 0;   // read after the first block's barriers
  constexpr int NCAND = 2 * (TOPK > 0 ? TOPK : 1) + ATT_OVF;   // list entries per (split, row)
  const long crow_ = ((long)split * a.H * a.nc + hc) * a.t + my_lat;

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
          // keys within REFINE_MARGIN of the running maximum enter the lane's
          // sorted list; the entry a full list pushes out, or the key itself
          // when it does not enter, goes to the row's overflow list if it is
          // still in the margin (padding rows past t take none)
          const float cut = fmaxf(m_run, mx) - REFINE_MARGIN;
          if (x > cut && my_lat < a.t) {
            auto overflow = [&](float ov, int ok) {
              const int slot = atomicAdd(&ovn[wave * 32 + l32], 1);
              if (slot < ATT_OVF) {
                a.cval[crow_ * NCAND + 2 * TOPK + slot] = ov;
                a.cidx[crow_ * NCAND + 2 * TOPK + slot] = ok;
              }
            };
            if (x > tv[TOPK - 1]) {
              const float ev = tv[TOPK - 1];
              const int ek = ti[TOPK - 1];
              float v = x;
              int id = n0 + kl;
              bool moved = false;   // entries after the insertion point shift (exact ties too)
#pragma unroll
              for (int q = 0; q < TOPK; ++q) {
                const bool gt = moved || v > tv[q];
                const float tvq = tv[q];
                const int tiq = ti[q];
                tv[q] = gt ? v : tvq;
                ti[q] = gt ? id : tiq;
                v = gt ? tvq : v;
                id = gt ? tiq : id;
                moved = gt;
              }
              if (ek >= 0 && ev > cut) overflow(ev, ek);
            } else {
              overflow(x, n0 + kl);
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
        a.cval[row * NCAND + lg * TOPK + q] = tv[q];
        a.cidx[row * NCAND + lg * TOPK + q] = ti[q];
      }
      if (lg == 0) a.ocnt[row] = min(ovn[wave * 32 + l32], ATT_OVF);
    }
  }
}

}  // namespace still

namespace still {

// ---------------------------------------------------------------------------
// fp16 cross-attention.  Workgroup = TT latents x one key range of one
// (KV head, cross head) pair; 4 waves, one per SIMD (512 registers each: the
// logit and output accumulators live in the accumulation registers).  Key
// blocks of KB = 256; wave w owns keys [64 w, 64 w + 64) of a block in the
// QK product (64 keys x TT latents per wave) and output features
// [w D2 / 4, (w + 1) D2 / 4) in the P.X product.
//   QK: S^T[key][lat] over the head width, in chunks of QC = 64 (one barrier
//       per chunk).  Q chunks are copied straight from global memory into a
//       ring of four LDS stages (direct loads, issued three chunks ahead of
//       use), and each step's Q fragments are read one step ahead of the
//       MFMAs that use them.  K fragments come
//       from the tiled layout straight into a ring of registers one chunk
//       deep: the slot used now is reloaded with the same step of the next
//       chunk (of the next block, in a block's last chunk, so those loads
//       have the softmax and P.X of the block to arrive).
//   softmax: logit (log2 units) = S * rk[key] * qs[lat] with qs = rq * scale
//       * log2(e) (the query side of the QK-norm and the logit scale: one
//       factor per lane and latent tile); per-latent block maxima combined
//       over the 4 waves through LDS; P (fp16) to LDS [lat][key].
//   P.X: O^T[feat][lat] += X^T[feat][key] P^T[key][lat]; X^T fragments from
//       the tiled layout through a ring of XR key steps, P from LDS.
// Keys past the range end (only in its last block) are masked by an additive
// -inf: their tiled k slots must hold finite values (the launches zero them,
// zero_ktile_tail_kernel).  The grid is 1-D, ordered so
// that the t tiles of one (pair, split) are consecutive workgroups of one
// XCD and read the same keys through its L2.
// ---------------------------------------------------------------------------
template <int TT, int D2, int TOPK>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1))) void xattn_f16_kernel(AttnArgs a) {
  constexpr int NW = 4, NT = 256, KB = 256, KW = 64, KT = 2;
  constexpr int LT = TT / 32;            // latent tiles
  constexpr int FW = D2 / NW;            // output features per wave
  constexpr int FT = FW / 32;            // feature tiles per wave
  constexpr int QC = 64, NS = QC / 16;   // Q chunk width; k steps per chunk = K ring depth
  constexpr int NQS = 4, QAHEAD = 3;     // Q stages; chunks between a stage's loads and its use
  constexpr int QI = TT / 8 / NW;        // Q stage loads per wave and chunk (8 rows of 128 bytes each)
  constexpr int LP = KB + 8;             // P row stride (halfs)
  constexpr int NBK = 2 * NW;            // candidate buckets per latent (wave, lane half)
  constexpr int XR = 4;                  // X^T ring depth (key steps of 16)
  constexpr int PS = KB / 16;            // key steps per block in P.X
  static_assert(FT >= 1 && QI >= 1 && TT % (8 * NW) == 0, "tile sizes");

  __shared__ __attribute__((aligned(16))) f16 Qs[NQS][TT * QC];   // rows of 8 swizzled 16-byte units
  __shared__ __attribute__((aligned(16))) f16 Ps[TT * LP];
  __shared__ float red_m[TT][NW], red_l[TT][NW];
  __shared__ __attribute__((aligned(16))) float rks[2][KB];   // key norm factors (0 past the range end)
  __shared__ __attribute__((aligned(16))) float kbs[2][KB];   // key mask: 0, or -inf past the range end
  __shared__ float qsl[TT];   // qs of each latent row (read in the softmax, not held in registers)
  __shared__ int ovn[TT];     // overflow entries of each latent row

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index (uniform)
  const int l32 = lane & 31, lg = lane >> 5;

  const int ntt = (a.t + TT - 1) / TT, HC = a.H * a.nc;
  const int total = gridDim.x;
  int L = blockIdx.x;
  if ((total & 7) == 0) L = (L & 7) * (total >> 3) + (L >> 3);
  const int S = total / (ntt * HC);
  const int tt = L % ntt, rest = L / ntt;
  const int split = rest % S, hc = rest / S;
  const int h = hc / a.nc, c = hc - h * a.nc;
  const int t0 = tt * TT;
  const int nbeg = split * a.keys_per_split;
  const int nend = min(a.N, nbeg + a.keys_per_split);

  const f16* qb = (const f16*)a.q + (long)h * a.t * a.ldq + (long)c * a.dc;
  const f16* kb = (const f16*)a.k + (long)hc * a.npad * a.dc;
  const f16* xtb = (const f16*)a.xt + ((long)h * a.xfeat + (long)c * a.xcoff) * a.npad;
  const float* rkb = a.rk + (long)h * a.N * a.nc + c;
  const unsigned ksteps = (unsigned)(a.dc >> 4);   // width steps of one key tile
  const unsigned nsteps = (unsigned)(a.npad >> 4); // key steps of one feature tile

  float m_run[LT], l_run[LT];
#pragma unroll
  for (int lt = 0; lt < LT; ++lt) {
    m_run[lt] = -INFINITY;
    l_run[lt] = 0.f;
  }
  if (tid < TT) {
    const int lat = min(t0 + tid, a.t - 1);   // rows past t: any positive factor
    qsl[tid] = a.rq[((long)h * a.t + lat) * a.nc + c] * a.scale_log2;
    ovn[tid] = 0;
  }
  f32x16 o[FT][LT];
#pragma unroll
  for (int f = 0; f < FT; ++f)
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) o[f][lt] = zero16();
  // Candidate keys for the logit refinement: each lane keeps, per latent
  // tile, a sorted list of its TOPK largest logits (bucket = wave, lane half)
  // in registers, written out once at the end.  Keys below the running
  // maximum minus REFINE_MARGIN can never be selected and are skipped, which
  // makes list updates rare.
  constexpr int TK = TOPK > 0 ? TOPK : 1;
  float tv[LT][TK];
  int ti[LT][TK];
#pragma unroll
  for (int lt = 0; lt < LT; ++lt)
#pragma unroll
    for (int q = 0; q < TK; ++q) {
      tv[lt][q] = -INFINITY;
      ti[lt][q] = -1;
    }

  // Q chunk staging: wave instruction i fills rows [8 b, 8 b + 8) of a stage
  // (b = i NW + w, 1 KB); lane l writes unit l % 8 of row 8 b + l / 8 and so
  // reads the global unit that the swizzle puts there.  Rows past t read the
  // last row: their logits are finite and never reach a stored output.
  // The loads are issued from inline assembly: the compiler, seeing direct
  // loads among the register loads of the K ring, would wait for all of them
  // before each use of a K fragment.  It still counts the K-ring loads, and
  // so over-waits by at most the stage loads issued after them; the waits
  // for the stages are explicit (chunk_barrier).
  unsigned qoff[QI];
#pragma unroll
  for (int i = 0; i < QI; ++i) {
    const int r = 8 * (i * NW + w) + (lane >> 3);
    const unsigned lat = (unsigned)min(t0 + r, a.t - 1);
    qoff[i] = lat * (unsigned)a.ldq + 8u * (unsigned)((lane & 7) ^ lds_swz<8>(r));
  }
  auto dma_q = [&](int stage, int d0) {
#pragma unroll
    for (int i = 0; i < QI; ++i) {
      const unsigned m0v = (unsigned)(size_t)(__attribute__((address_space(3))) f16*)&Qs[stage][(i * NW + w) * 512];
      asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                   :: "v"(qb + (qoff[i] + (unsigned)d0)), "s"(m0v) : "memory", "m0");
    }
  };
  // Q fragment of latent tile lt, 16-column step js, from a stage
  auto q_frag = [&](int stage, int lt, int js) -> half8 {
    const int r = 32 * lt + l32;
    return *(const half8*)&Qs[stage][r * QC + 8 * ((2 * js + lg) ^ lds_swz<8>(r))];
  };
  // Chunks are numbered across blocks (g): chunk g uses stage g % NQS and Q
  // columns [(g % nch) QC, +QC); it issues the loads of chunk g + QAHEAD into
  // the stage that chunk g - 1 released, and its last step reads the first
  // fragments of chunk g + 1.  So at the barrier that ends chunk g the loads
  // of chunk g + 2 must have landed: they were issued at the start of chunk
  // g - 1, followed by the K-ring loads of chunk g - 1 and the stage and
  // K-ring loads of chunk g (more at block boundaries); loads return in
  // order.  The asm statements also keep the compiler from moving memory
  // accesses across the barriers.
  static_assert(NQS == 4 && QAHEAD == 3, "the stage ring and the wait count go together");
  constexpr int QWAIT = NS * KT + QI + NS * KT;
  static_assert(QWAIT <= 63, "vmcnt range");
  auto chunk_barrier = [&]() {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" :: "n"(QWAIT) : "memory");
  };
  // this wave's LDS traffic has completed, then all waves meet (stage loads
  // may still be in flight)
  auto lds_barrier = [&]() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  };
  // K fragment of this wave's key tile kt of the block at n0, width step js
  auto load_k = [&](int n0, int kt, int js) -> half8 {
    const unsigned kti = (unsigned)(n0 + KW * w + 32 * kt) >> 5;
    return *(const half8*)(kb + ((kti * ksteps + (unsigned)js) * 512u + 8u * lane));
  };
  // X^T fragment of this wave's feature tile f, key step ns (absolute)
  auto load_x = [&](int f, int ns) -> half8 {
    const unsigned ft = (unsigned)(FW / 32 * w + f);
    return *(const half8*)(xtb + ((ft * nsteps + (unsigned)ns) * 512u + 8u * lane));
  };
  auto load_rk = [&](int n0) -> float {   // 0 past the range end (branch-free load)
    const int n = n0 + tid;
    const float v = rkb[(long)min(n, nend - 1) * a.nc];
    return n < nend ? v : 0.f;
  };

  const int nch = a.dc / QC;   // a.dc is a multiple of QC (checked on the host), nch >= 2
  half8 kr[NS][KT];
  half8 xr[XR][FT];
  half8 qf[2][LT];
  int g = 0, qn = QAHEAD % nch;   // chunk number; Q chunk of chunk g + QAHEAD
  int rbuf = 0;
  // prologue: Q chunks 0 .. QAHEAD-1, key norms and K ring of the first block
#pragma unroll
  for (int c = 0; c < QAHEAD; ++c) dma_q(c, (c % nch) * QC);
#pragma unroll
  for (int j = 0; j < NS; ++j)
#pragma unroll
    for (int kt = 0; kt < KT; ++kt) kr[j][kt] = load_k(nbeg, kt, j);
  rks[0][tid] = load_rk(nbeg);
  kbs[0][tid] = nbeg + tid < nend ? 0.f : -INFINITY;
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
#pragma unroll
  for (int lt = 0; lt < LT; ++lt) qf[0][lt] = q_frag(0, lt, 0);

  for (int n0 = nbeg; n0 < nend; n0 += KB) {
    const bool next_block = n0 + KB < nend;   // uniform
    f32x16 s[LT][KT];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt)
#pragma unroll
      for (int kt = 0; kt < KT; ++kt) s[lt][kt] = zero16();

    // ---- S^T = K_blk Q^T over the head width.  A chunk runs its MFMAs on the
    // Q chunk in LDS and the K ring while it loads the next stages: Q chunk
    // qn2 (stored at the chunk's end) and, into each ring slot right after its
    // last use, the same step of the next chunk (k steps ks0 + j of the block
    // at kn0).  Each step reads the next step's Q fragments (the next chunk's
    // first ones in the last step) before its own MFMAs; scheduling barriers
    // keep that order and spread the loads over the chunk.
    auto qk_chunk = [&](int kn0, int ks0) {
      dma_q((g + QAHEAD) & (NQS - 1), qn * QC);
      const int sc = g & (NQS - 1), sn = (g + 1) & (NQS - 1);
#pragma unroll
      for (int j = 0; j < NS; ++j) {
#pragma unroll
        for (int lt = 0; lt < LT; ++lt) qf[(j + 1) & 1][lt] = q_frag(j + 1 < NS ? sc : sn, lt, j + 1 < NS ? j + 1 : 0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int lt = 0; lt < LT; ++lt)
#pragma unroll
          for (int kt = 0; kt < KT; ++kt)
            s[lt][kt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(kr[j][kt], qf[j & 1][lt], s[lt][kt], 0, 0, 0);
#pragma unroll
        for (int kt = 0; kt < KT; ++kt) kr[j][kt] = load_k(kn0, kt, ks0 + j);
        __builtin_amdgcn_sched_barrier(0);
      }
      ++g;
      qn = qn + 1 == nch ? 0 : qn + 1;
    };
    for (int ch = 0; ch + 1 < nch; ++ch) {
      qk_chunk(n0, (ch + 1) * NS);
      chunk_barrier();
    }
    {  // last chunk: the K ring moves on to chunk 0 of the next block (of this
       // block again at the very end: loaded, never used), with its key norms
      // (the key norm is selected after the chunk: an earlier use would wait
      // for its load in front of the chunk's stage loads)
      const int nn = n0 + KB + tid;
      const float rk_raw = rkb[(long)min(nn, nend - 1) * a.nc];
      qk_chunk(next_block ? n0 + KB : n0, 0);
      rks[rbuf ^ 1][tid] = nn < nend ? rk_raw : 0.f;
      kbs[rbuf ^ 1][tid] = nn < nend ? 0.f : -INFINITY;
      chunk_barrier();
    }
    // X^T ring for the block's P.X (arrives during the softmax)
#pragma unroll
    for (int i = 0; i < XR; ++i)
#pragma unroll
      for (int f = 0; f < FT; ++f) xr[i][f] = load_x(f, (n0 >> 4) + i);

    // ---- softmax: x = S * rk + kb, written back over S: kb = -inf masks the
    // keys past the range end without a select (their tiled k slots are zero,
    // so S is finite there), and fma with a zero addend is exactly the
    // product; logit (log2 units) = x * qs[lt] (qs > 0, so block maxima of x
    // scale to those of the logits); one pass for the block maxima, one for
    // the probabilities
    const float* rkc = rks[rbuf];
    const float* kbc = kbs[rbuf];
    float mx[LT], lmx[LT], qs[LT];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) qs[lt] = qsl[32 * lt + l32];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) mx[lt] = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < KT; ++kt)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int kl = KW * w + 32 * kt + 8 * jq + 4 * lg;   // keys of j = 4 jq + u: kl + u
        const float4 r4 = *(const float4*)&rkc[kl];
        const float4 b4 = *(const float4*)&kbc[kl];
        const float rk[4] = {r4.x, r4.y, r4.z, r4.w};
        const float kb[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
        for (int lt = 0; lt < LT; ++lt)
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const float x = fmaf(s[lt][kt][4 * jq + u], rk[u], kb[u]);
            s[lt][kt][4 * jq + u] = x;
            mx[lt] = fmaxf(mx[lt], x);
          }
      }
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) {
      lmx[lt] = mx[lt];
      mx[lt] = fmaxf(mx[lt], __shfl_xor(mx[lt], 32));
      if (lg == 0) red_m[32 * lt + l32][w] = mx[lt] * qs[lt];
    }
    lds_barrier();
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
            const float p = __builtin_amdgcn_exp2f(fmaf(s[lt][kt][4 * jq + u], qs[lt], -mref));
            ps += p;
            pv[u] = (f16)p;
          }
          *(half4*)&Ps[li * LP + KW * w + 32 * kt + 8 * jq + 4 * lg] = pv;
        }
      ps += __shfl_xor(ps, 32);
      if (lg == 0) red_l[li][w] = ps;
      if constexpr (TOPK > 0) {
        // Keys whose logit (x * qs) lies within REFINE_MARGIN of the running
        // maximum are candidates.  Usually a lane has none; when it has
        // some, it is nearly always exactly one (its block maximum lmx,
        // handled directly); two or more take the general loop.  A candidate
        // enters the lane's sorted list if it beats the list's last entry;
        // the entry it pushes out, or the candidate itself when it does not
        // enter, goes to the row's overflow list if it is still in the
        // margin, so no in-margin key is lost while the overflow has room.
        // Padding rows past t (zero queries: every key ties at logit 0) are
        // skipped.
        const float cut = m_new - REFINE_MARGIN;
        if (t0 + li < a.t && lmx[lt] * qs[lt] > cut) {
          const long orow = ((long)split * HC + hc) * a.t + (t0 + li);
          auto overflow = [&](float v, int k) {
            const int slot = atomicAdd(&ovn[li], 1);
            if (slot < XATT_OVF) {
              a.cval[orow * (NBK * TOPK + XATT_OVF) + NBK * TOPK + slot] = v;
              a.cidx[orow * (NBK * TOPK + XATT_OVF) + NBK * TOPK + slot] = k;
            }
          };
          auto push = [&](float v, int k) {
            if (!(v > tv[lt][TOPK - 1])) {
              overflow(v, k);
              return;
            }
            const float ev = tv[lt][TOPK - 1];
            const int ek = ti[lt][TOPK - 1];
            // insert before the first smaller entry; every entry after it
            // shifts down one place (also past equal values: exact ties)
            bool moved = false;
#pragma unroll
            for (int q = 0; q < TOPK; ++q) {
              const bool gt = moved || v > tv[lt][q];
              const float tq = tv[lt][q];
              const int iq = ti[lt][q];
              tv[lt][q] = gt ? v : tq;
              ti[lt][q] = gt ? k : iq;
              v = gt ? tq : v;
              k = gt ? iq : k;
              moved = gt;
            }
            if (ek >= 0 && ev > cut) overflow(ev, ek);
          };
          int cnt = 0, id = 0;
#pragma unroll
          for (int kt = 0; kt < KT; ++kt)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
              const float v = s[lt][kt][j];
              cnt += v * qs[lt] > cut ? 1 : 0;
              id = v == lmx[lt] ? n0 + KW * w + 32 * kt + 8 * (j >> 2) + 4 * lg + (j & 3) : id;
            }
          if (cnt == 1) {
            push(lmx[lt] * qs[lt], id);
          } else {
            for (int kt = 0; kt < KT; ++kt)
              for (int j = 0; j < 16; ++j) {
                const float v = s[lt][kt][j] * qs[lt];
                if (v > cut) push(v, n0 + KW * w + 32 * kt + 8 * (j >> 2) + 4 * lg + (j & 3));
              }
          }
        }
      }
      m_run[lt] = m_new;
    }
    lds_barrier();
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) {
      const int li = 32 * lt + l32;
      float lb = 0.f;
#pragma unroll
      for (int u = 0; u < NW; ++u) lb += red_l[li][u];
      l_run[lt] = l_run[lt] * alpha[lt] + lb;
    }
    rbuf ^= 1;
    // rescale O for the latents whose maximum grew (rare after the first
    // blocks), one 32x32 tile at a time
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) {
      if (__any(alpha[lt] != 1.f)) {
#pragma unroll
        for (int f = 0; f < FT; ++f) {
          __builtin_amdgcn_sched_barrier(0);
#pragma unroll
          for (int j = 0; j < 16; ++j) o[f][lt][j] *= alpha[lt];
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }

    // ---- O^T += X^T P^T over the block's KB keys, 16 at a time (the next
    // step's P fragments read before this step's MFMAs)
    half8 pf[2][LT];
#pragma unroll
    for (int lt = 0; lt < LT; ++lt) pf[0][lt] = *(const half8*)&Ps[(32 * lt + l32) * LP + 8 * lg];
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) {
      if (ps + 1 < PS) {
#pragma unroll
        for (int lt = 0; lt < LT; ++lt)
          pf[(ps + 1) & 1][lt] = *(const half8*)&Ps[(32 * lt + l32) * LP + 16 * (ps + 1) + 8 * lg];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int lt = 0; lt < LT; ++lt)
#pragma unroll
        for (int f = 0; f < FT; ++f)
          o[f][lt] = __builtin_amdgcn_mfma_f32_32x32x16_f16(xr[ps % XR][f], pf[ps & 1][lt], o[f][lt], 0, 0, 0);
      if (ps + XR < PS) {
#pragma unroll
        for (int f = 0; f < FT; ++f) xr[ps % XR][f] = load_x(f, (n0 >> 4) + ps + XR);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // stage loads of chunks past the end may still be in flight: they land
  // before the workgroup's LDS is released
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

  // ---- partial (O un-normalised, m, l) of this key range
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
        a.cval[row * (NBK * TOPK + XATT_OVF) + (2 * w + lg) * TOPK + q] = tv[lt][q];
        a.cidx[row * (NBK * TOPK + XATT_OVF) + (2 * w + lg) * TOPK + q] = ti[lt][q];
      }
      if (w == 0 && lg == 0) a.ocnt[row] = min(ovn[32 * lt + l32], XATT_OVF);
    }
  }
}

}  // namespace still
