// gemm.hpp - tiled MFMA GEMM C = A * B^T for the latent-side and projection
// products of the compactor, with the epilogues those products need fused in.
//
//   A [M][K] row-major (K contiguous), B [N][K] row-major (the [out][in] weight
//   layout), both converted to the compute type CT on their way into LDS.
//   256 threads = 4 waves in a 2x2 grid; each wave owns a (BM/2) x (BN/2)
//   block of 32x32 MFMA tiles; two LDS stages, one barrier per k step.  LDS
//   rows are unpadded; the 16-byte units of a row are XOR-swizzled by row so
//   that both the staging stores and the MFMA fragment reads are free of bank
//   conflicts.  The epilogue stages each wave's results through LDS so that
//   global loads and stores are 16-byte vectors along contiguous columns.
//
// Column layout: the tile's BN columns are two halves of BN/2 and every wave
// owns the same sub-range of BN/4 columns in both halves, so paired epilogues
// find both members of a pair in the same lane:
//   PAIR:   pair P -> columns (c*hd + j, c*hd + j + hd/2), c = P / (hd/2),
//           j = P % (hd/2): rotate-half RoPE partners (optional rotation by a
//           cos/sin table, optional bias, optional per-row sum of squares of
//           the un-rotated biased values for the later L2 QK-norm, optional
//           fp32 copy of the result).
//   SWIGLU: pair P -> row P of W_g (half 0) and of W_u (half 1);
//           out[:, P] = SiLU(g) * u.
// Other epilogues: STORE (+bias), GELU (+bias), RESID (C += acc, fp32),
// SCALE (acc * scale * rq[row] * rk[col]).
#pragma once
#include <type_traits>

#include "common.hpp"

namespace still {

enum EpiKind { EPI_STORE = 0, EPI_RESID = 1, EPI_PAIR = 2, EPI_SWIGLU = 3, EPI_SCALE = 4, EPI_GELU = 5 };
enum CTileKind { CTILE_NONE = 0, CTILE_KEYS = 1, CTILE_VALUES = 2 };

struct GemmArgs {
  int M, N, K;   // N = output columns, or column pairs for PAIR / SWIGLU
  int nb2;       // batch index z -> (z / nb2, z % nb2), strides s*1, s*2 (elements)
  const void* A;
  const void* A2;      // optional low part of a split A operand: C = (A + A2) B^T, same layout as A
  long lda, sA1, sA2;
  const void* B;
  const void* B2;      // SWIGLU: W_u
  long ldb, sB1, sB2;
  int bwrap;           // B column k >= bwrap reads column k - bwrap (0 = off)
  // Row grouping: with mgroups > 1 the M rows are mgroups groups of M/mgroups
  // rows spaced mgstride apart, and a tile takes BM/mgroups rows of every
  // group (rows of different groups that share per-row side data, such as a
  // rotation table row, then meet in one tile).
  int mgroups;
  long mgstride;
  void* C;
  long ldc, sC1, sC2;
  const void* bias;    // per output column, NULL = none
  long sBias2;         // bias offset per unit of the inner batch index
  int hd;              // PAIR: head width
  const float2* tab;   // rotation table, row (r % tab_mod), entry [row*hd/2 + j]; NULL = none
  int tab_mod;
  float* part;         // PAIR: sum-of-squares partials [head*nparts + p][ldpart] (ldpart >= rows), NULL = none
  long ldpart;
  float* C2;           // PAIR: optional fp32 copy of the (rotated) outputs, ldc as C
  // PAIR: with qperm, C (not C2) holds each head's widths in the permuted
  // order of the fp16 cross-attention within every step of 16 (position p of
  // a step holds width kperm_width(p)); requires hd % 16 == 0
  int qperm;
  // RESID: optional per-row factor of the product, rowscale[row / rowscale_div]
  // (undoes the fp16 range scale of the value path per KV head)
  const float* rowscale;
  int rowscale_div;
  // Output layout (STORE and PAIR): CTILE_NONE row-major (ldc); CTILE_KEYS the
  // fragment-tiled key layout of the fp16 attention kernel, row r = h *
  // ctile_rows + n, column c * hd + x -> ktile_off(h * ctile_heads + c, n, x,
  // ctile_npad, hd); CTILE_VALUES its tiled value layout, row = feature f,
  // column = key n -> xtile_off(0, f, n, ctile_npad) (per batch: sC1).
  int ctile, ctile_heads;
  long ctile_rows, ctile_npad;
  float scale;         // SCALE: C = acc * scale * rq[r] * rk[col]
  const float* rq;
  long ldrq, sQ1, sQ2;
  const float* rk;
  long ldrk, sK1, sK2;
};

// Element offset of output (row r, column col) in the layout g.ctile names.
// Eight consecutive columns from a multiple of 8 stay contiguous in every
// layout, so the epilogues' 16-byte runs keep their form.
__device__ __forceinline__ long c_off(const GemmArgs& g, long r, long col) {
  if (g.ctile == CTILE_KEYS) {
    const long h = r / g.ctile_rows, n = r - h * g.ctile_rows;
    const long c = col / g.hd, x = col - c * g.hd;
    return ktile_off(h * g.ctile_heads + c, n, x, g.ctile_npad, g.hd);
  }
  if (g.ctile == CTILE_VALUES) return xtile_off(0, r, col, g.ctile_npad, 32);
  return r * g.ldc + col;
}

__device__ __forceinline__ float silu_f(float x) { return x / (1.f + expf(-x)); }
__device__ __forceinline__ float gelu_f(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }

// 16-byte vector of n elements of T
template <class T> struct Vec16 {
  static constexpr int n = 16 / sizeof(T);
};

__device__ __forceinline__ void wave_lds_fence() {
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): this wave's LDS traffic has completed
  __builtin_amdgcn_wave_barrier();
}

// LDS arena: two operand stages, reused after the k loop for the epilogue
// staging (4 waves x 32 rows x (BN/2 + 8) floats).
template <int BM, int BN, int BK, class CT>
constexpr int gemm_lds_bytes(int am = 1) {
  const int ops = 2 * (am * BM + BN) * BK * (int)sizeof(CT);
  const int stg = 4 * 32 * (BN / 2 + 8) * 4;   // epilogue staging
  return ops > stg ? ops : stg;
}

// ST = 0: operands through registers into two LDS stages (any element types,
// converted on the way), loaded two k steps ahead.  ST = 2: fp16 operands
// copied straight from global memory into two LDS stages (global_load_lds,
// 16 bytes a lane), the next k step in flight during the current one's MFMAs;
// needs K % BK == 0 and 16-byte aligned rows and strides (host checks).
template <class CT, class TA, class TB, class TC, class TBias, int EPI, int BM, int BN, int BK, int ST = 0>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
  typedef Mma<CT> MM;
  typedef typename MM::frag frag;
  constexpr int E = MM::E;
  constexpr int LR = BK;                      // LDS row stride (elements), unpadded
  constexpr int TM = BM / 64, TN = BN / 64;    // 32x32 tiles per wave
  constexpr int KV = BK / E;                   // 16-byte vectors per tile row
  constexpr int AV = BM * KV / 256, BV = BN * KV / 256;
  constexpr bool PAIRED = (EPI == EPI_PAIR || EPI == EPI_SWIGLU);
  static_assert(AV >= 1 && BV >= 1 && BM * KV % 256 == 0 && BN * KV % 256 == 0, "tile/threads");
  static_assert(TN % 2 == 0, "BN must allow two column halves per wave");
  // epilogue staging (per wave: 32 rows x TN*32 columns of fp32) must fit the arena
  constexpr int WC = TN * 32;
  constexpr int SLD = WC + 8;                  // staging row stride (floats): rows r and r+4 on disjoint banks
  static_assert(WC == BN / 2, "wave column count");
  // ST = 3: the direct-load path for a split A operand (C = (A + A2) B^T):
  // each stage holds the k step of A, of A2 and of B, and each B fragment
  // read from it serves both products (one pass over K instead of two)
  constexpr int AM = ST == 3 ? 2 : 1;           // A operands per stage
  constexpr int LDSB = gemm_lds_bytes<BM, BN, BK, CT>(AM);
  constexpr int SS = (AM * BM + BN) * LR;       // elements per stage: A rows (A2 rows), then B rows
  static_assert(4 * 32 * SLD * 4 <= LDSB, "staging does not fit");

  __shared__ __attribute__((aligned(16))) unsigned char smem[LDSB];
  __shared__ float sc_f[EPI == EPI_SCALE ? BM + BN : 1];   // SCALE: row factors, then column factors

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, lg = lane >> 5;

  // Tile order.  Workgroup ids are dealt to the 8 XCDs round robin.  A
  // batched product with few tiles per batch (and a multiple of 8 batches)
  // keeps every batch on one XCD, whose L2 then serves all its tiles' operand
  // reuse.  Otherwise XCD x takes the M tiles congruent to x mod 8 and walks
  // them in groups of 8 M tiles x all N tiles, so that the operand tiles its
  // concurrent workgroups touch stay in its L2.
  const int gx = gridDim.x, gy = gridDim.y;
  int lin = blockIdx.x + gx * blockIdx.y;
  int bz = blockIdx.z;
  constexpr int GM = 8;
  int mt0, nt;
  if ((gridDim.z & 7) == 0 && gx * gy <= 64) {
    const int T = gx * gy;
    const int gid = lin + T * blockIdx.z;            // dispatch order
    const int xcd = gid & 7, i = gid >> 3;
    bz = (i / T) * 8 + xcd;
    lin = i - (i / T) * T;
    mt0 = lin / gx;
    nt = lin - mt0 * gx;
  } else if ((gy & 7) == 0) {
    const int xcd = lin & 7, i = lin >> 3, gyx = gy >> 3;
    const int grp = i / (GM * gx), gm0 = grp * GM;
    const int gsz = min(GM, gyx - gm0);
    const int inl = i - grp * GM * gx;
    mt0 = (gm0 + inl % gsz) * 8 + xcd;
    nt = inl / gsz;
  } else {
    const int T = gx * gy;
    if ((T & 7) == 0) lin = (lin & 7) * (T >> 3) + (lin >> 3);
    const int grp = lin / (GM * gx), gm0 = grp * GM;
    const int gsz = min(GM, gy - gm0);
    const int inl = lin - grp * GM * gx;
    mt0 = gm0 + inl % gsz;
    nt = inl / gsz;
  }

  const int b1 = bz / g.nb2, b2 = bz - b1 * g.nb2;
  const int M = g.M;
  {
  const int mt = mt0;
  const TA* A = (const TA*)g.A + b1 * g.sA1 + b2 * g.sA2;
  const TB* B = (const TB*)g.B + b1 * g.sB1 + b2 * g.sB2;
  const TB* B2 = PAIRED && g.B2 ? (const TB*)g.B2 + b1 * g.sB1 + b2 * g.sB2 : nullptr;
  const int N = g.N, K = g.K;
  const int m0 = mt * BM;
  const int hh = g.hd >> 1;
  const int mg = g.mgroups > 1 ? g.mgroups : 1;
  const int RG = BM / mg;                      // rows per group in a tile
  const int Mg = M / mg;                       // rows per group
  // global row of tile-local row lr, or -1 past the end
  auto grow = [&](int lr) -> long {
    if (mg == 1) {
      const int r = m0 + lr;
      return r < M ? r : -1;
    }
    const int grp = lr / RG, rr = mt * RG + (lr - grp * RG);
    return rr < Mg ? (long)grp * g.mgstride + rr : -1;
  };
  // the same row as (group, row within the group); with one group the row
  // itself.  Row indices fit 32 bits (bounded on the host).
  auto grow2 = [&](int lr, int& grp, int& rr) -> bool {
    if (mg == 1) {
      grp = 0;
      rr = m0 + lr;
      return rr < M;
    }
    grp = lr / RG;
    rr = mt * RG + (lr - grp * RG);
    return rr < Mg;
  };

  // LDS element offset of (row, 16-byte unit) in a stage
  auto lds_at = [&](int r, int u) { return r * LR + ((u ^ lds_swz<KV>(r)) * E); };
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
  // B operand row of tile-local row lc (paired kinds: the pair members of
  // the two column halves) and whether it lies inside the product
  auto b_row = [&](int lc, bool& valid) -> const TB* {
    if (PAIRED) {
      const int half = lc / (BN / 2);
      const int P = nt * (BN / 2) + (lc % (BN / 2));
      valid = P < N;
      if (EPI == EPI_PAIR) {
        const int c = P / hh, j = P - c * hh;
        return B + (long)(c * g.hd + j + half * hh) * g.ldb;
      }
      return (half ? B2 : B) + (long)P * g.ldb;
    }
    const int n = nt * BN + lc;
    valid = n < N;
    return B + (long)n * g.ldb;
  };
  // SCALE: the per-row and per-column factors (BM + BN values) are loaded
  // together with the first k step's operands and kept in LDS for the
  // epilogue, so their latency is not exposed after the k loop
  float scf[(BM + BN + 255) / 256];
  auto load_scale = [&]() {
    if constexpr (EPI == EPI_SCALE) {
      const float* rqv = g.rq + b1 * g.sQ1 + b2 * g.sQ2;
      const float* rkv = g.rk + b1 * g.sK1 + b2 * g.sK2;
#pragma unroll
      for (int i = 0; i < (BM + BN + 255) / 256; ++i) {
        const int v = tid + 256 * i;
        float f = 0.f;
        if (v < BM) {
          const long r = grow(v);
          if (r >= 0) f = rqv[r * g.ldrq];
        } else if (v < BM + BN) {
          const int col = nt * BN + (v - BM);
          if (col < N) f = rkv[(long)col * g.ldrk] * g.scale;
        }
        scf[i] = f;
      }
    }
  };
  auto store_scale = [&]() {
    if constexpr (EPI == EPI_SCALE) {
#pragma unroll
      for (int i = 0; i < (BM + BN + 255) / 256; ++i)
        if (tid + 256 * i < BM + BN) sc_f[tid + 256 * i] = scf[i];
    }
  };
  CT* smem_ct = (CT*)smem;
  if constexpr (ST == 0) {
  // global -> register staging, two sets: loads run two k steps ahead
  frag ra[2][AV], rb[2][BV];
  const TB* brow_ptr[BV];
  bool bvalid[BV];
#pragma unroll
  for (int i = 0; i < BV; ++i) {
    brow_ptr[i] = b_row((tid + i * 256) / KV, bvalid[i]);
    if (!bvalid[i]) brow_ptr[i] = B;   // loads always issue (from row 0) and are zeroed
  }

  const TA* Alo = g.A2 ? (const TA*)g.A2 + b1 * g.sA1 + b2 * g.sA2 : nullptr;
  const int nk1 = (K + BK - 1) / BK;
  const int nk = Alo ? 2 * nk1 : nk1;      // split A: second pass over K with the low part
  // per-thread staging slots, fixed for the whole k loop: tile row of each
  // 16-byte vector, its global row offset (-1: past the end) and its k offset
  const int kk = (tid % KV) * E;
  long aoff[AV];
#pragma unroll
  for (int i = 0; i < AV; ++i) {
    const long gr = grow((tid + i * 256) / KV);
    aoff[i] = gr >= 0 ? gr * g.lda : -1;
  }
  // Loads of k step kn into a register set.  Every load instruction issues
  // (out-of-range rows and k read row 0 / column 0) and the zeroing of those
  // happens only when the set is stored to LDS, so the number of loads in
  // flight is static and the wait before a stage store leaves the following
  // step's loads outstanding.  Returns whether this thread's k run is in range.
  auto load_stage = [&](int kn, frag (&xa)[AV], frag (&xb)[BV]) -> bool {
    const bool lo = kn >= nk1;                 // split A: second pass with the low part
    const TA* Ap = lo ? Alo : A;
    const int gk = (lo ? kn - nk1 : kn) * BK + kk;
    const bool kin = gk < K;
    const int gks = kin ? gk : 0;
#pragma unroll
    for (int i = 0; i < AV; ++i) xa[i] = VecLoad<CT, TA>::load(Ap + (aoff[i] >= 0 ? aoff[i] : 0) + gks);
    const int gkb = (g.bwrap && gks >= g.bwrap) ? gks - g.bwrap : gks;
#pragma unroll
    for (int i = 0; i < BV; ++i) xb[i] = VecLoad<CT, TB>::load(brow_ptr[i] + gkb);
    return kin;
  };
  const int su = tid % KV;
  auto store_stage = [&](int buf, const frag (&xa)[AV], const frag (&xb)[BV], bool kin) {
#pragma unroll
    for (int i = 0; i < AV; ++i)
      *(frag*)&smem_ct[buf * SS + lds_at((tid + i * 256) / KV, su)] = (aoff[i] >= 0 && kin) ? xa[i] : zero_frag<CT>();
#pragma unroll
    for (int i = 0; i < BV; ++i)
      *(frag*)&smem_ct[buf * SS + BM * LR + lds_at((tid + i * 256) / KV, su)] = (bvalid[i] && kin) ? xb[i] : zero_frag<CT>();
  };



  // k steps past the end reload the last one (their data is never stored)
  auto issue = [&](int kn, frag (&xa)[AV], frag (&xb)[BV]) -> bool {
    return load_stage(kn < nk ? kn : nk - 1, xa, xb);
  };
  auto compute = [&](int buf) {
    const CT* Ac = smem_ct + buf * SS;
    const CT* Bc = Ac + BM * LR;
#pragma unroll
    for (int ks = 0; ks < BK / (2 * E); ++ks) {
      frag af[TM], bfr[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a)
        af[a] = *(const frag*)&Ac[lds_at(wm * (BM / 2) + a * 32 + l32, ks * 2 + lg)];
#pragma unroll
      for (int b = 0; b < TN; ++b)
        bfr[b] = *(const frag*)&Bc[lds_at(col_base(b) + l32, ks * 2 + lg)];
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) MM::mma(acc[a][b], af[a], bfr[b]);
    }
  };
  // step kt: LDS stage kt & 1 holds k step kt, register set nxt holds k step
  // kt + 1 (in flight); set cur (already in LDS) takes k step kt + 2.
  bool kin0, kin1;
  auto step = [&](int kt, frag (&ca)[AV], frag (&cb)[BV], bool& ckin, frag (&na)[AV], frag (&nb)[BV], bool nkin) {
    ckin = issue(kt + 2, ca, cb);
    __builtin_amdgcn_sched_barrier(0);   // loads go out before this step's MFMA work
    compute(kt & 1);
    if (kt + 1 < nk) store_stage((kt + 1) & 1, na, nb, nkin);
    __syncthreads();
  };
  load_scale();
  kin0 = issue(0, ra[0], rb[0]);
  store_stage(0, ra[0], rb[0], kin0);
  store_scale();
  kin1 = issue(1, ra[1], rb[1]);
  __syncthreads();
  int kt = 0;
  for (; kt + 1 < nk; kt += 2) {   // both steps unconditional: one loop state at the back edge
    step(kt, ra[0], rb[0], kin0, ra[1], rb[1], kin1);
    step(kt + 1, ra[1], rb[1], kin1, ra[0], rb[0], kin0);
  }
  if (kt < nk) step(kt, ra[0], rb[0], kin0, ra[1], rb[1], kin1);
  } else {
  // ---- direct global -> LDS loads into the two stages.  One wave instruction
  // fills one 1 KB block of a stage (RPB tile rows); lane l writes unit l % KV
  // of row l / KV and so reads the global unit that the swizzle puts there.
  // Rows past the end read row 0: they only reach outputs that are not stored.
  static_assert(sizeof(CT) == 2 && sizeof(TA) == 2 && sizeof(TB) == 2, "direct loads copy fp16 operands");
  constexpr int RPB = 512 / BK;                 // tile rows per 1 KB block
  constexpr int NBLK = (AM * BM + BN) / RPB;    // blocks per stage
  constexpr int NI = NBLK / 4;                  // blocks per wave and stage
  static_assert(NBLK % 4 == 0 && BM % RPB == 0 && (ST == 2 || ST == 3), "direct load blocks");
  const int w = __builtin_amdgcn_readfirstlane(wave);
  // split A (C = (A + A2) B^T): a second pass over K reads the low part
  const CT* Alo = g.A2 ? (const CT*)g.A2 + b1 * g.sA1 + b2 * g.sA2 : nullptr;
  const int nk1 = K / BK;
  const int nk = (Alo && AM == 1) ? 2 * nk1 : nk1;
  const CT* src[NI];     // first pass
  const CT* srclo[NI];   // second pass (A rows from A2; B rows unchanged)
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int rho = (i * 4 + w) * RPB + lane / KV;
    const int u = (lane % KV) ^ lds_swz<KV>(rho);   // rho and rho - BM (rho - 2 BM) agree mod 16
    if (rho < AM * BM) {
      const bool second = rho >= BM;                 // AM = 2: rows of A2
      const long gr = grow(second ? rho - BM : rho);
      const long off = (gr >= 0 ? gr * g.lda : 0) + u * E;
      src[i] = (second ? Alo : (const CT*)A) + off;
      srclo[i] = (Alo && AM == 1) ? Alo + off : src[i];
    } else {
      bool valid;
      const TB* bp = b_row(rho - AM * BM, valid);
      src[i] = srclo[i] = (const CT*)(valid ? bp : B) + u * E;
    }
  }
  // k step kn into stage kn % 2
  auto dma = [&](int kn) {
    CT* st = smem_ct + (kn & 1) * SS;
    const bool lo = kn >= nk1;
    const long ks = (long)(lo ? kn - nk1 : kn) * BK;
#pragma unroll
    for (int i = 0; i < NI; ++i)
      __builtin_amdgcn_global_load_lds((const void*)((lo ? srclo[i] : src[i]) + ks),
                                       (__attribute__((address_space(3))) void*)(st + (i * 4 + w) * 512), 16, 0, 0);
  };
  // this wave's loads of all but the newest n k steps have landed and its
  // LDS reads have completed (vmcnt(n * NI), lgkmcnt(0)); the compiler
  // tracks neither across the barrier that follows
  auto wait_steps = [&](auto n) {
    constexpr int c = decltype(n)::value * NI;
    __builtin_amdgcn_s_waitcnt((c & 15) | ((c >> 4) << 14) | 0x70);
  };
  auto compute = [&](const CT* Ac) {
    const CT* Bc = Ac + AM * BM * LR;
    const CT* Lc = Ac + BM * LR;   // AM = 2: the A2 rows
    constexpr int KS = BK / (2 * E);
    frag af[2][TM], al[2][AM == 2 ? TM : 1], bfr[2][TN];
    auto rd = [&](int ks, int p) {
#pragma unroll
      for (int a = 0; a < TM; ++a) af[p][a] = *(const frag*)&Ac[lds_at(wm * (BM / 2) + a * 32 + l32, ks * 2 + lg)];
      if constexpr (AM == 2) {
#pragma unroll
        for (int a = 0; a < TM; ++a) al[p][a] = *(const frag*)&Lc[lds_at(wm * (BM / 2) + a * 32 + l32, ks * 2 + lg)];
      }
#pragma unroll
      for (int b = 0; b < TN; ++b) bfr[p][b] = *(const frag*)&Bc[lds_at(col_base(b) + l32, ks * 2 + lg)];
    };
    rd(0, 0);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + 1 < KS) rd(ks + 1, (ks + 1) & 1);   // next fragments in flight during this step's MFMAs
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) {
          MM::mma(acc[a][b], af[ks & 1][a], bfr[ks & 1][b]);
          if constexpr (AM == 2) MM::mma(acc[a][b], al[ks & 1][a], bfr[ks & 1][b]);
        }
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  dma(0);
  load_scale();
  store_scale();
  wait_steps(std::integral_constant<int, 0>());
  __builtin_amdgcn_s_barrier();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) dma(kt + 1);   // stage (kt + 1) % 2 was released by the last barrier
    __builtin_amdgcn_sched_barrier(0);
    compute(smem_ct + (kt & 1) * SS);
    wait_steps(std::integral_constant<int, 0>());
    __builtin_amdgcn_s_barrier();
  }
  }

  // ------------------------------------------------------------------ epilogue
  // Per 32-row slice a of the wave's block: values -> LDS staging (fp32, the
  // wave's private region) -> contiguous runs of output columns -> 16-byte
  // stores.  Output columns of the wave's run q (q = 0, 1: the two halves):
  //   plain:  nt*BN + q*BN/2 + wn*BN/4 + [0, BN/4)
  //   PAIR:   c*hd + j0 + q*hd/2 + [0, BN/4)  for the wave's pairs P0..P0+BN/4-1
  //   SWIGLU: P0 + [0, BN/4) (one run)
  float* stg = (float*)smem + wave * 32 * SLD;
  TC* C = (TC*)g.C + b1 * g.sC1 + b2 * g.sC2;
  const TBias* bias = g.bias ? (const TBias*)g.bias + b2 * g.sBias2 : nullptr;
  const int P0 = nt * (BN / 2) + wn * (BN / 4);           // first pair of the wave (paired kinds)
  const int pc = PAIRED ? P0 / (hh > 0 ? hh : 1) : 0;     // head of the wave's pairs (PAIR)
  const int pj0 = PAIRED ? P0 - pc * hh : 0;
  constexpr int RUN = BN / 4;
  // PAIR: the bias values of the wave's pairs (the same for every slice),
  // loaded before any store of the epilogue
  float pbv0[PAIRED ? TN / 2 : 1], pbv1[PAIRED ? TN / 2 : 1];
  if constexpr (EPI == EPI_PAIR) {
#pragma unroll
    for (int b = 0; b < TN / 2; ++b) {
      const int x = b * 32 + l32;
      const bool pv = P0 + x < N;
      const int col0 = pc * g.hd + pj0 + x;
      pbv0[b] = (bias && pv) ? to_f32(bias[col0]) : 0.f;
      pbv1[b] = (bias && pv) ? to_f32(bias[col0 + hh]) : 0.f;
    }
  }
  // PAIR: rotation table values of vector-pass step (slice a, step it),
  // double-buffered so that each step's loads are issued before the previous
  // step's stores (a load issued after a store waits for it)
  constexpr int PV_ = 8, NIT_ = (EPI == EPI_PAIR) ? 32 * (RUN / PV_) / 64 : 1;
  f32x4 tcs[2][PV_ / 2];
  auto tab_load = [&](int a, int it, f32x4 (&dst)[PV_ / 2]) {
    if constexpr (EPI == EPI_PAIR) {
      constexpr int NV = RUN / PV_;
      const int e = lane + 64 * it;
      const int rl = e / NV, vx = (e % NV) * PV_;
      int rgrp, rrow;
      const bool rok = grow2(wm * (BM / 2) + a * 32 + rl, rgrp, rrow);
      if (g.tab && rok && N - (P0 + vx) > 0) {
        const long r = (long)rgrp * g.mgstride + rrow;
        const int trow = (mg > 1 && g.mgstride == g.tab_mod) ? rrow : (int)r % g.tab_mod;
        const float2* tp = g.tab + (long)trow * hh + pj0 + vx;
#pragma unroll
        for (int u = 0; u < PV_; u += 2) dst[u / 2] = *(const f32x4*)(tp + u);
      }
    }
  };
  if constexpr (EPI == EPI_PAIR) tab_load(0, 0, tcs[0]);
  // columns of run q, element x: global output column and validity
  auto run_col = [&](int q, int x) -> long {
    if constexpr (EPI == EPI_PAIR) return (long)pc * g.hd + pj0 + q * hh + x;
    else if constexpr (EPI == EPI_SWIGLU) return (long)P0 + x;
    else return (long)nt * BN + q * (BN / 2) + wn * (BN / 4) + x;
  };

#pragma unroll
  for (int a = 0; a < TM; ++a) {
    const int lbase = wm * (BM / 2) + a * 32;    // tile-local first row of the slice
    // ---- 1. values into the staging slice
    if constexpr (EPI == EPI_SCALE) {
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int rl = 8 * (j >> 2) + 4 * lg + (j & 3);
#pragma unroll
        for (int b = 0; b < TN; ++b)
          stg[rl * SLD + b * 32 + l32] = acc[a][b][j] * sc_f[lbase + rl] * sc_f[BM + col_base(b) + l32];
      }
    } else if constexpr (!PAIRED) {
      float rsc[16];
#pragma unroll
      for (int j = 0; j < 16; ++j) rsc[j] = 1.f;
      if (EPI == EPI_RESID && g.rowscale) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const long r = grow(lbase + 8 * (j >> 2) + 4 * lg + (j & 3));
          rsc[j] = r >= 0 ? g.rowscale[r / g.rowscale_div] : 0.f;
        }
      }
#pragma unroll
      for (int b = 0; b < TN; ++b) {
        const int col = nt * BN + col_base(b) + l32;
        const float bv = (bias && col < N) ? to_f32(bias[col]) : 0.f;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int rl = 8 * (j >> 2) + 4 * lg + (j & 3);
          float v = acc[a][b][j] * rsc[j];
          if constexpr (EPI == EPI_GELU) {
            v = gelu_f(v + bv);
          } else if constexpr (EPI != EPI_RESID) {
            v = v + bv;
          }
          stg[rl * SLD + b * 32 + l32] = v;
        }
      }
    } else if constexpr (EPI == EPI_SWIGLU) {
#pragma unroll
      for (int b = 0; b < TN / 2; ++b)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int rl = 8 * (j >> 2) + 4 * lg + (j & 3);
          stg[rl * SLD + b * 32 + l32] = silu_f(acc[a][b][j]) * acc[a][b + TN / 2][j];
        }
    } else {   // PAIR: biased pair members; rotation in the vector pass
#pragma unroll
      for (int b = 0; b < TN / 2; ++b) {
        const float bv0 = pbv0[b], bv1 = pbv1[b];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int rl = 8 * (j >> 2) + 4 * lg + (j & 3);
          stg[rl * SLD + b * 32 + l32] = acc[a][b][j] + bv0;
          stg[rl * SLD + (b + TN / 2) * 32 + l32] = acc[a][b + TN / 2][j] + bv1;
        }
      }
    }
    wave_lds_fence();
    if constexpr (EPI == EPI_PAIR) {
      // ---- 2p. pairs: 8 pairs per lane and step, rows split over NV lanes.
      // Rotation by the table row, 16-byte stores of both members, the
      // row's sum of squares (rotation keeps it), reduced over the NV lanes
      // of a row.
      constexpr int PV = 8, NV = RUN / PV;
      static_assert(NV >= 1 && 64 % NV == 0 && (32 * NV) % 64 == 0, "pair vector pass");
      const bool want_ss = g.part != nullptr;
      const int nparts = (hh / (BN / 2)) * 2;
      const int pidx = (pj0 / (BN / 2)) * 2 + wn;
#pragma unroll
      for (int it = 0; it < 32 * NV / 64; ++it) {
        static_assert(32 * NV / 64 == NIT_, "vector-pass steps");
        const int e = lane + 64 * it;
        // the next step's table values (next slice's first step after the last)
        if (it + 1 < NIT_) tab_load(a, it + 1, tcs[(a * NIT_ + it + 1) & 1]);
        else if (a + 1 < TM) tab_load(a + 1, 0, tcs[(a * NIT_ + it + 1) & 1]);
        const int rl = e / NV, vx = (e % NV) * PV;
        int rgrp, rrow;
        const bool rok = grow2(lbase + rl, rgrp, rrow);
        const long r = rok ? (long)rgrp * g.mgstride + rrow : -1;
        const int nvalid = N - (P0 + vx);
        float sp = 0.f;
        if (rok && nvalid > 0) {
          float v0[PV], v1[PV];
          const float* s0 = stg + rl * SLD + vx;
#pragma unroll
          for (int u = 0; u < PV; u += 4) {
            const f32x4 a0 = *(const f32x4*)(s0 + u);
            const f32x4 a1 = *(const f32x4*)(s0 + RUN + u);
#pragma unroll
            for (int w = 0; w < 4; ++w) {
              v0[u + w] = a0[w];
              v1[u + w] = a1[w];
            }
          }
#pragma unroll
          for (int u = 0; u < PV; ++u) sp += v0[u] * v0[u] + v1[u] * v1[u];
          const int jp = pj0 + vx;
          if (g.tab) {
#pragma unroll
            for (int u = 0; u < PV; u += 2) {
              const f32x4 cs = tcs[(a * NIT_ + it) & 1][u / 2];
              const float y00 = v0[u] * cs[0] - v1[u] * cs[1], y10 = v1[u] * cs[0] + v0[u] * cs[1];
              const float y01 = v0[u + 1] * cs[2] - v1[u + 1] * cs[3], y11 = v1[u + 1] * cs[2] + v0[u + 1] * cs[3];
              v0[u] = y00;
              v1[u] = y10;
              v0[u + 1] = y01;
              v1[u + 1] = y11;
            }
          }
          const long col0 = (long)pc * g.hd + jp;
          {
            TC* d0 = C + c_off(g, r, col0);
            TC* d1 = C + c_off(g, r, col0 + hh);
            constexpr int VE = Vec16<TC>::n;
            const bool vec_ok = nvalid >= PV && (g.ldc % VE) == 0 && (((uintptr_t)C & 15) == 0);
            float s0[PV], s1[PV];   // values in store order
#pragma unroll
            for (int u = 0; u < PV; ++u) {
              s0[u] = v0[u];
              s1[u] = v1[u];
            }
            if (g.qperm) {
              // runs jp and jp ^ 8 (lanes e, e ^ 1 of the same row) swap half
              // runs: the even run stores widths {0-3, 8-11}, the odd one
              // {4-7, 12-15} of their step of 16
              const bool even = ((jp >> 3) & 1) == 0;
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                const float r0 = __shfl_xor(even ? v0[4 + u] : v0[u], 1);
                const float r1 = __shfl_xor(even ? v1[4 + u] : v1[u], 1);
                s0[u] = even ? v0[u] : r0;
                s0[4 + u] = even ? r0 : v0[4 + u];
                s1[u] = even ? v1[u] : r1;
                s1[4 + u] = even ? r1 : v1[4 + u];
              }
            }
            if (vec_ok) {
#pragma unroll
              for (int u = 0; u < PV; u += VE) {
                TC t0[VE], t1[VE];
#pragma unroll
                for (int w = 0; w < VE; ++w) {
                  t0[w] = from_f32<TC>(s0[u + w]);
                  t1[w] = from_f32<TC>(s1[u + w]);
                }
                __builtin_nontemporal_store(*(const u32x4*)t0, (u32x4*)(d0 + u));
                __builtin_nontemporal_store(*(const u32x4*)t1, (u32x4*)(d1 + u));
              }
            } else {
              for (int u = 0; u < PV && u < nvalid; ++u) {
                d0[u] = from_f32<TC>(s0[u]);
                d1[u] = from_f32<TC>(s1[u]);
              }
            }
            if (g.C2) {
              float* e0 = g.C2 + r * g.ldc + col0;
              if (vec_ok && (((uintptr_t)g.C2 & 15) == 0)) {
#pragma unroll
                for (int u = 0; u < PV; u += 4) {
                  __builtin_nontemporal_store(f32x4{v0[u], v0[u + 1], v0[u + 2], v0[u + 3]}, (f32x4*)(e0 + u));
                  __builtin_nontemporal_store(f32x4{v1[u], v1[u + 1], v1[u + 2], v1[u + 3]}, (f32x4*)(e0 + hh + u));
                }
              } else {
                for (int u = 0; u < PV && u < nvalid; ++u) {
                  e0[u] = v0[u];
                  e0[hh + u] = v1[u];
                }
              }
            }
          }
        }
        if (want_ss) {
#pragma unroll
          for (int o = 1; o < NV; o <<= 1) sp += __shfl_xor(sp, o);
          if ((e % NV) == 0 && rok)
            g.part[(long)(pc * nparts + pidx) * g.ldpart + r] = sp;   // partial-major: rows contiguous
        }
      }
    } else {
      // ---- 2. staged slice -> global, 16-byte vectors along each run
      constexpr int NRUN = (EPI == EPI_SWIGLU) ? 1 : 2;
      constexpr int VE = Vec16<TC>::n;
      constexpr int VPR = RUN / VE;                  // vectors per run row
      const bool vec_ok = (g.ldc % VE) == 0 && (((uintptr_t)C & 15) == 0);
      // RESID: C vectors are read in groups of RG before the group's writes
      // (the compiler cannot move a read of C above an earlier store to C, so
      // reading in the store loop costs one memory round trip per vector)
      constexpr int ITN = 32 * NRUN * VPR / 64, RG = 4;
      if constexpr (EPI == EPI_RESID && (32 * NRUN * VPR) % 64 == 0 && ITN % RG == 0) {
#pragma unroll
        for (int g0 = 0; g0 < ITN; g0 += RG) {
          f32x4 cold[RG];
          long off[RG];
          int okv[RG];
#pragma unroll
          for (int u = 0; u < RG; ++u) {
            const int e = lane + 64 * (g0 + u);
            const int rl = e / (NRUN * VPR);
            const int rem = e - rl * NRUN * VPR;
            const int q = rem / VPR, vx = (rem - q * VPR) * VE;
            const long r = grow(lbase + rl);
            const long col = run_col(q, vx);
            off[u] = r < 0 ? -1 : r * g.ldc + col;
            okv[u] = r < 0 ? 0 : ((N - (int)col >= VE && vec_ok) ? 2 : 1);   // 2: vector, 1: scalar tail
            if (okv[u] == 2) cold[u] = *(const f32x4*)(C + off[u]);
          }
#pragma unroll
          for (int u = 0; u < RG; ++u) {
            const int e = lane + 64 * (g0 + u);
            const int rl = e / (NRUN * VPR);
            const int rem = e - rl * NRUN * VPR;
            const int q = rem / VPR, vx = (rem - q * VPR) * VE;
            const float* src = stg + rl * SLD + q * RUN + vx;
            if (okv[u] == 2) {
              f32x4 o = cold[u];
#pragma unroll
              for (int w = 0; w < 4; ++w) o[w] += src[w];
              *(f32x4*)(C + off[u]) = o;
            } else if (okv[u] == 1) {
              const int nvalid = N - (int)run_col(q, vx);
              for (int w = 0; w < VE && w < nvalid; ++w) C[off[u] + w] = from_f32<TC>(to_f32(C[off[u] + w]) + src[w]);
            }
          }
        }
      } else
      for (int e = lane; e < 32 * NRUN * VPR; e += 64) {
        const int rl = e / (NRUN * VPR);
        const int rem = e - rl * NRUN * VPR;
        const int q = rem / VPR, vx = (rem - q * VPR) * VE;
        const long r = grow(lbase + rl);
        if (r < 0) continue;
        const float* src = stg + rl * SLD + q * RUN + vx;
        const long col = run_col(q, vx);
        TC* dst = C + c_off(g, r, col);
        int nvalid;
        if constexpr (PAIRED) {
          nvalid = N - (P0 + vx);
        } else {
          nvalid = N - (int)col;
        }
        if (nvalid >= VE && vec_ok) {
          if constexpr (EPI == EPI_RESID) {
            f32x4 o = *(const f32x4*)dst;
#pragma unroll
            for (int u = 0; u < 4; ++u) o[u] += src[u];
            *(f32x4*)dst = o;
          } else {
            TC tmp[VE];
#pragma unroll
            for (int u = 0; u < VE; ++u) tmp[u] = from_f32<TC>(src[u]);
            __builtin_nontemporal_store(*(const u32x4*)tmp, (u32x4*)dst);
          }
        } else {
          for (int u = 0; u < VE && u < nvalid; ++u) {
            if constexpr (EPI == EPI_RESID) dst[u] = from_f32<TC>(to_f32(dst[u]) + src[u]);
            else dst[u] = from_f32<TC>(src[u]);
          }
        }
      }
    }
    wave_lds_fence();
  }
  }  // tile
}

template <class CT, class TA, class TB, class TC, class TBias, int EPI, int BM, int BN, int BK, int ST = 0>
hipError_t launch_gemm(const GemmArgs& g, int batch, hipStream_t st) {
  constexpr bool PAIRED = (EPI == EPI_PAIR || EPI == EPI_SWIGLU);
  const int ntn = PAIRED ? (g.N + BN / 2 - 1) / (BN / 2) : (g.N + BN - 1) / BN;
  const int mg = g.mgroups > 1 ? g.mgroups : 1;
  const int ntm = mg == 1 ? (g.M + BM - 1) / BM : (g.M / mg + BM / mg - 1) / (BM / mg);
  if (ntn <= 0 || ntm <= 0 || batch <= 0) return hipSuccess;
  dim3 grid(ntn, ntm, batch);
  hipLaunchKernelGGL((gemm_kernel<CT, TA, TB, TC, TBias, EPI, BM, BN, BK, ST>), grid, dim3(256), 0, st, g);
  return hipGetLastError();
}

}  // namespace still
