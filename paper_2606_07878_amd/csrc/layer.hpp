// layer.hpp - the per-layer launch sequence of the compaction: RoPE-fix
// staging, cross-attention (query and key projections, flash attention,
// logit refinement, split merge, value and output projections), latent
// self-attention, FFN and the output heads.
#pragma once
#include "gemm.hpp"
#include "host.hpp"
#include "kproj.hpp"
#include "refine.hpp"
#include "refine64.hpp"

namespace still {

// ---------------------------------------------------------------------------
// Launch helpers
// ---------------------------------------------------------------------------
template <class CT> struct Tile;
template <> struct Tile<f16> { static constexpr int BM = 128, BN = GEMM_BN, BK = 32; };
template <> struct Tile<float> { static constexpr int BM = 128, BN = GEMM_BN, BK = 16; };

// Long reductions take twice the k depth per stage (half the barriers and
// twice the MFMA work between operand loads); short ones keep BK so that more
// workgroups fit a CU.
constexpr int GEMM_LONG_K = 512;

// Direct global -> LDS operand loads (two LDS stages, the next k step's copy
// in flight during the current one's MFMAs; bit-identical results) apply to fp16
// operands with whole k steps, 16-byte aligned rows and batch strides and no
// wrapped operand; paired kinds also need whole runs of 8 pairs.
static bool direct_ok(const GemmArgs& g, int bk, bool paired) {
  auto al = [](const void* p) { return ((uintptr_t)p & 15) == 0; };
  return g.K % bk == 0 && !g.bwrap && g.lda % 8 == 0 && g.ldb % 8 == 0 && g.sA1 % 8 == 0 && g.sA2 % 8 == 0 &&
         g.sB1 % 8 == 0 && g.sB2 % 8 == 0 && (g.mgroups <= 1 || g.mgstride % 8 == 0) && al(g.A) && (!g.A2 || al(g.A2)) &&
         al(g.B) && (!g.B2 || al(g.B2)) && (!paired || g.N % 8 == 0);
}

template <class CT, class TA, class TB, class TC, class TBias, int EPI, int BM, int BN, int BK>
static hipError_t launch_pick(const GemmArgs& g, int batch, hipStream_t st) {
  if constexpr (std::is_same<CT, f16>::value && std::is_same<TA, f16>::value && std::is_same<TB, f16>::value) {
    if (direct_ok(g, BK, EPI == EPI_PAIR || EPI == EPI_SWIGLU)) {
      if constexpr (EPI == EPI_PAIR && BN == 256)
        if (g.A2) return launch_gemm<CT, TA, TB, TC, TBias, EPI, BM, BN, BK, 3>(g, batch, st);
      return launch_gemm<CT, TA, TB, TC, TBias, EPI, BM, BN, BK, 2>(g, batch, st);
    }
  }
  return launch_gemm<CT, TA, TB, TC, TBias, EPI, BM, BN, BK>(g, batch, st);
}

// WIDE: 128 x 256 tiles (BK 32, 2 waves per SIMD) for the latent-side
// products with many output columns and K >= 512 (fp16 mode; paired kinds need
// head widths that are multiples of 256), where they still leave at least two
// workgroups per CU.  The norm partials of a PAIR product then number hd/256*2
// per head instead of hd/128*2, so paired kinds always take them.
template <class CT, class TA, class TB, class TC, class TBias, int EPI, bool WIDE = false>
static hipError_t gemm(const GemmArgs& g, int batch, hipStream_t st, int cls = STILL_K_LATENT) {
  timing::Scope ts(cls, st);
  if constexpr (WIDE && sizeof(CT) == 2) {
    constexpr bool PAIRED = (EPI == EPI_PAIR || EPI == EPI_SWIGLU);
    const long ntn = PAIRED ? (g.N + 127) / 128 : (g.N + 255) / 256;
    const long ntm = g.mgroups > 1 ? (g.M / g.mgroups + 128 / g.mgroups - 1) / (128 / g.mgroups) : (g.M + 127) / 128;
    if (PAIRED || ntn * ntm * batch >= 512) return launch_pick<CT, TA, TB, TC, TBias, EPI, 128, 256, 32>(g, batch, st);
  }
  if constexpr (sizeof(CT) == 2) {
    // fewer 128-row tiles than CUs (the output heads, small t): 64-row tiles
    constexpr bool PAIRED = (EPI == EPI_PAIR || EPI == EPI_SWIGLU);
    const long ntn = PAIRED ? (g.N + 63) / 64 : (g.N + 127) / 128;
    const long ntm = g.mgroups > 1 ? (g.M / g.mgroups + 128 / g.mgroups - 1) / (128 / g.mgroups) : (g.M + 127) / 128;
    if (g.mgroups <= 1 && ntn * ntm * batch < 256) {
      if (g.K >= GEMM_LONG_K)
        return launch_pick<CT, TA, TB, TC, TBias, EPI, 64, Tile<CT>::BN, 2 * Tile<CT>::BK>(g, batch, st);
      return launch_pick<CT, TA, TB, TC, TBias, EPI, 64, Tile<CT>::BN, Tile<CT>::BK>(g, batch, st);
    }
  }
  if (g.K >= GEMM_LONG_K)
    return launch_pick<CT, TA, TB, TC, TBias, EPI, Tile<CT>::BM, Tile<CT>::BN, 2 * Tile<CT>::BK>(g, batch, st);
  return launch_pick<CT, TA, TB, TC, TBias, EPI, Tile<CT>::BM, Tile<CT>::BN, Tile<CT>::BK>(g, batch, st);
}

static GemmArgs gargs(int M, int N, int K, const void* A, long lda, const void* B, long ldb, void* C, long ldc) {
  GemmArgs g;
  memset(&g, 0, sizeof g);
  g.M = M;
  g.N = N;
  g.K = K;
  g.nb2 = 1;
  g.A = A;
  g.lda = lda;
  g.B = B;
  g.ldb = ldb;
  g.C = C;
  g.ldc = ldc;
  return g;
}


template <class CT, int D2, int TOPK = XATT_TOPK>
static hipError_t launch_attn(const AttnArgs& a, int splits, hipStream_t st) {
  dim3 grid((a.t + ATT_TT - 1) / ATT_TT, a.H * a.nc, splits);
  if constexpr (sizeof(CT) == 2) {
    constexpr int TT = D2 <= 256 ? 128 : 64;
    const int ntt = (a.t + TT - 1) / TT;
    static_assert(xatt_waves(D2) == 4, "the fp16 kernel runs 4 waves");
    hipLaunchKernelGGL((xattn_f16_kernel<TT, D2, TOPK>), dim3(ntt * a.H * a.nc * splits), dim3(256), 0, st, a);
  } else {
    hipLaunchKernelGGL((cross_attn_kernel<CT, ATT_TT, (D2 > 256 ? 32 : ATT_NB), 32, D2, ATT_TOPK>), grid, dim3(256),
                       0, st, a);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// One layer: IT = I/O type of K, V, weights and outputs; CT = MFMA operand /
// intermediate storage type.
// ---------------------------------------------------------------------------
template <class IT, class CT>
still_status run_layer(const still_config* cfg, const Dims& m, const Plan& p, char* ws,
                              const still_layer_weights* w, const void* Kp, const void* Vp,
                              const double* positions, bool rerotate, void* Ckp, void* Cvp, hipStream_t st) {
  const long Ht = (long)m.H * m.t;
  const long HN = (long)m.H * m.N;
  CT* X = (CT*)(ws + p.X);
  CT* XT = (CT*)(ws + p.XT);
  float* Z = (float*)(ws + p.Z);
  CT* Y = (CT*)(ws + p.Y);
  CT* q = (CT*)(ws + p.q);
  CT* head = q;
  float* partq = (float*)(ws + p.partq);
  float* rq = (float*)(ws + p.rq);
  CT* O = (CT*)(ws + p.O);
  CT* k = (CT*)(ws + p.k);
  float* partk = (float*)(ws + p.partk);
  float* rk = (float*)(ws + p.rk);
  const float2* tab_ck = m.fp32 ? (const float2*)(ws + p.tab_ck) : nullptr;   // bf16 mode: computed in place
  const double* invf_c = (const double*)(ws + p.invf_c);
  const float2* tab_cq = (const float2*)(ws + p.tab_cq);
  const double* invf_b = (const double*)(ws + p.invf_b);
  const float2* tab_bq = (const float2*)(ws + p.tab_bq);
  const float LOG2E = 1.4426950408889634f;
  // wide GEMM tiles for the paired projections when the head widths allow them
  const bool wide_c = !m.fp32 && m.dc % 256 == 0, wide_s = !m.fp32 && m.ns > 0 && m.ds % 256 == 0;

  // bf16 mode: the layer's weight matrices converted once to the fp16 MFMA
  // operand type (biases and latents stay bf16); every GEMM then reads fp16.
  std::vector<still_block_weights> cblocks(w->blocks, w->blocks + cfg->n_blocks);
  still_layer_weights cw = *w;
  if constexpr (!std::is_same<IT, CT>::value) {
    CT* dst = (CT*)(ws + p.wconv);
    ConvSegs segs;
    memset(&segs, 0, sizeof segs);
    int ns = 0;
    long longest = 0;
    hipError_t err = hipSuccess;
    auto flush = [&]() {
      if (ns == 0 || err != hipSuccess) return;
      TIMED(STILL_K_OTHER);
      hipLaunchKernelGGL((convert_kernel<IT, CT>), dim3(grid1d(longest) > 1024 ? 1024 : grid1d(longest), ns),
                         dim3(256), 0, st, segs);
      err = hipGetLastError();
      memset(&segs, 0, sizeof segs);
      ns = 0;
      longest = 0;
    };
    for_each_matrix(cfg, m, w, cblocks.data(), &cw.w_key, &cw.w_val, [&](const void* src, long n, const void** slot) {
      segs.src[ns] = src;
      segs.dst[ns] = dst;
      segs.n8[ns] = n / 8;
      if (n / 8 > longest) longest = n / 8;
      *slot = dst;
      dst += rup(n, 128);
      if (++ns == CONV_SEGS) flush();
    });
    flush();
    HIP_TRY(err);
    cw.blocks = cblocks.data();
    w = &cw;
  }

  // RoPE-fix staging of X = [R(-p) K ; V] and X^T.  fp16 operands: the first
  // pass also finds each head's max |K|, |V|; heads beyond the fp16 range
  // (scale != 1) are staged again, scaled by an exact power of two.
  {
    const int RW = stage_rows(m);
    const size_t lds = (size_t)RW * (m.d2 + 8) * m.cs;
    const dim3 grid((unsigned)stage_blocks(m), m.H);
    TIMED(STILL_K_STAGE);
    float* part = sizeof(CT) == 2 ? (float*)(ws + p.kvpart) : nullptr;
    float* hscale = sizeof(CT) == 2 ? (float*)(ws + p.hscale) : nullptr;
    hipLaunchKernelGGL((stage_x_kernel<IT, CT>), grid, dim3(256), lds, st, (const IT*)Kp, (const IT*)Vp, positions,
                       invf_b, m.N, m.d, X, XT, m.Npad, RW, part, (const float*)hscale, 0);
    HIP_TRY(hipGetLastError());
    if (hscale) {
      hipLaunchKernelGGL(kv_scale_kernel, dim3(m.H), dim3(256), 0, st, (const float*)part, (int)grid.x, m.H, hscale);
      HIP_TRY(hipGetLastError());
      hipLaunchKernelGGL((stage_x_kernel<IT, CT>), grid, dim3(256), lds, st, (const IT*)Kp, (const IT*)Vp, positions,
                         invf_b, m.N, m.d, X, XT, m.Npad, RW, (float*)nullptr, (const float*)hscale, 1);
      HIP_TRY(hipGetLastError());
    }
  }
  {
    TIMED(STILL_K_OTHER);
    hipLaunchKernelGGL((init_z_kernel<IT>), dim3(grid1d(Ht * m.D / 8)), dim3(256), 0, st, (const IT*)w->latents, Z, Ht * m.D);
  }
  HIP_TRY(hipGetLastError());
  auto rmsnorm = [&]() -> hipError_t {
    TIMED(STILL_K_OTHER);
    hipLaunchKernelGGL((rmsnorm_kernel<CT>), dim3((unsigned)((Ht + 3) / 4)), dim3(256), 0, st, Z, Y, Ht, m.D,
                       cfg->rms_eps);
    return hipGetLastError();
  };
  auto rmsnorm_split = [&](f16* hi, f16* lo) -> hipError_t {
    TIMED(STILL_K_OTHER);
    hipLaunchKernelGGL(rmsnorm_split_kernel, dim3((unsigned)((Ht + 3) / 4)), dim3(256), 0, st, Z, hi, lo, Ht, m.D,
                       cfg->rms_eps);
    return hipGetLastError();
  };
  auto finalize = [&](const float* part, long rows, int nh, int np, float* rn) -> hipError_t {
    TIMED(STILL_K_OTHER);
    hipLaunchKernelGGL(finalize_norm_kernel, dim3(grid1d(rows * nh)), dim3(256), 0, st, part, rows, nh, np,
                       cfg->l2_eps, rn);
    return hipGetLastError();
  };

  for (int b = 0; b < cfg->n_blocks; ++b) {
    const still_block_weights& bw = w->blocks[b];
    // ---------------- cross-attention: Z += CrossAttn(RMSNorm(Z), X)
    if (cfg->cross_every_block || b == 0) {
      if constexpr (sizeof(CT) == 2) {
        if (m.R > 0 && !m.fp32) HIP_TRY(rmsnorm_split((f16*)Y, (f16*)(ws + p.Ylo)));
        else HIP_TRY(rmsnorm());
      } else {
        HIP_TRY(rmsnorm());
      }
      {  // q = RoPE_c(q~) with q~ = Y W_Q^T + b_Q, plus ||q~||^2 partials
        GemmArgs g = gargs((int)Ht, m.Ec / 2, m.D, Y, m.D, bw.ca_wq, m.D, q, m.Ec);
        if (m.R > 0 && !m.fp32) {   // Y split into hi + lo: accurate q~ (fp32 copy for the refinement)
          g.A2 = ws + p.Ylo;
          g.C2 = (float*)(ws + p.qex);
        }
        g.bias = bw.ca_bq;
        g.hd = m.dc;
        g.tab = tab_cq;
        g.tab_mod = m.t;
        g.qperm = m.fp32 ? 0 : 1;   // widths in the order of the tiled keys (kproj.hpp)
        g.part = partq;
        g.ldpart = Ht;
        if (wide_c) HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR, true>(g, 1, st, STILL_K_QPROJ)));
        else HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR>(g, 1, st, STILL_K_QPROJ)));
      }
      if constexpr (sizeof(CT) == 2) {
        // k = RoPE_c(k~), k~ = X W_K^T + b_K, fused kernel writing the tiled key
        // layout; one sum-of-squares partial per (row, cross head)
        TIMED(STILL_K_KPROJ);
        f16* wkt = (f16*)(ws + p.wkt);
        hipLaunchKernelGGL(tile_w_kernel, dim3(grid1d((long)m.Ec * m.d2 / 8)), dim3(256), 0, st,
                           (const f16*)bw.ca_wk, (long)m.Ec, m.d2, wkt);
        HIP_TRY(hipGetLastError());
        KprojArgs ka;
        ka.X = (const f16*)X;
        ka.wkt = wkt;
        ka.bias = bw.ca_bk;
        ka.pos = positions;
        ka.invf = invf_c;
        ka.k = (f16*)k;
        ka.part = partk;
        ka.H = m.H;
        ka.N = (int)m.N;
        ka.nc = m.nc;
        ka.dc = m.dc;
        ka.npad = m.Npad;
        ka.hscale = (const float*)(ws + p.hscale);
        // table stage capacity 16, 64 or 128 key positions (LDS <= 160 KB)
        ka.kpw = 128 / m.H;
        const dim3 grid((unsigned)((m.N + ka.kpw - 1) / ka.kpw));
        if (ka.kpw <= 16) {
          if (m.d2 == 128) hipLaunchKernelGGL((kproj_kernel<128, 16, IT>), grid, dim3(256), 0, st, ka);
          else if (m.d2 == 256) hipLaunchKernelGGL((kproj_kernel<256, 16, IT>), grid, dim3(256), 0, st, ka);
          else hipLaunchKernelGGL((kproj_kernel<512, 16, IT>), grid, dim3(256), 0, st, ka);
        } else if (ka.kpw <= 64 || m.d2 == 512) {
          ka.kpw = std::min(ka.kpw, m.d2 == 512 ? 32 : 64);
          const dim3 g2((unsigned)((m.N + ka.kpw - 1) / ka.kpw));
          if (m.d2 == 128) hipLaunchKernelGGL((kproj_kernel<128, 64, IT>), g2, dim3(256), 0, st, ka);
          else if (m.d2 == 256) hipLaunchKernelGGL((kproj_kernel<256, 64, IT>), g2, dim3(256), 0, st, ka);
          else hipLaunchKernelGGL((kproj_kernel<512, 32, IT>), g2, dim3(256), 0, st, ka);
        } else {
          if (m.d2 == 128) hipLaunchKernelGGL((kproj_kernel<128, 128, IT>), grid, dim3(256), 0, st, ka);
          else hipLaunchKernelGGL((kproj_kernel<256, 128, IT>), grid, dim3(256), 0, st, ka);
        }
        HIP_TRY(hipGetLastError());
        if (m.Npad > m.N) {   // keys past N: finite (zero) slots for the additive mask of the attention
          hipLaunchKernelGGL(zero_ktile_tail_kernel, dim3(grid1d((long)m.H * m.nc * (m.Npad - m.N) * (m.dc / 8))),
                             dim3(256), 0, st, (f16*)k, (long)m.H * m.nc, (int)m.N, (long)m.Npad, m.dc);
          HIP_TRY(hipGetLastError());
        }
        HIP_TRY(finalize(partk, HN, m.nc, 1, rk));
      } else {  // k = RoPE_c(k~) with k~ = X W_K^T + b_K
        GemmArgs g = gargs((int)HN, m.Ec / 2, m.d2, X, m.d2, bw.ca_wk, m.d2, k, m.Ec);
        if (Tile<CT>::BM % m.H == 0) {   // tiles span the same keys of every KV head: shared table rows
          g.mgroups = m.H;
          g.mgstride = m.N;
        }
        g.bias = bw.ca_bk;
        g.hd = m.dc;
        g.tab = tab_ck;
        g.tab_mod = (int)m.N;
        g.part = partk;
        g.ldpart = HN;
        HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR>(g, 1, st, STILL_K_KPROJ)));
        HIP_TRY(finalize(partk, HN, m.nc, m.np_c, rk));
      }
      HIP_TRY(finalize(partq, Ht, m.nc, wide_c ? m.dc / 256 * 2 : m.np_c, rq));
      const float ca_scale = cfg->logit_scale_cross != 0.f ? cfg->logit_scale_cross : (float)m.dc;
      {
        AttnArgs a;
        a.q = q;
        a.ldq = m.Ec;
        a.rq = rq;
        a.k = k;
        a.ldk = m.Ec;
        a.rk = rk;
        a.xt = XT;
        a.ldxt = m.Npad;
        a.npad = m.Npad;
        a.opart = (float*)(ws + p.opart);
        a.mpart = (float*)(ws + p.mpart);
        a.lpart = (float*)(ws + p.lpart);
        a.H = m.H;
        a.N = (int)m.N;
        a.t = m.t;
        a.nc = m.nc;
        a.dc = m.dc;
        a.d2 = m.d2;
        a.scale_log2 = ca_scale * LOG2E;
        a.keys_per_split = (int)m.keys_per_split;
        a.cval = (float*)(ws + p.cval);
        a.cidx = (int*)(ws + p.cidx);
        a.ocnt = (int*)(ws + p.ocnt);
        a.xfeat = m.d2;
        a.xcoff = 0;
        hipError_t e;
        {
        TIMED(STILL_K_CROSS_ATTN);
        if (m.d2 == 128) e = launch_attn<CT, 128>(a, m.splits, st);
        else if (m.d2 == 256) e = launch_attn<CT, 256>(a, m.splits, st);
        else e = launch_attn<CT, 512>(a, m.splits, st);
        }
        HIP_TRY(e);
        RefineArgs ra;
        memset(&ra, 0, sizeof ra);
        if (m.R > 0) {
          const long HCT = Ht * m.nc;
          const int TR = m.t * m.R, NB = m.H * m.nc;
          int* ridx = (int*)(ws + p.ridx);
          int* crow = (int*)(ws + p.crow);
          int* ccount = (int*)(ws + p.ccount);
          {
            TIMED(STILL_K_REFINE);
            hipLaunchKernelGGL((refine_select_kernel<REFINE_R>), dim3((unsigned)((HCT + 3) / 4)), dim3(256), 0,
                               st, a.cval, a.cidx, a.ocnt, a.mpart, m.splits, HCT, m.ncand, m.ncand_fixed, ridx,
                               (float*)(ws + p.rval), (int*)(ws + p.rcnt));
            HIP_TRY(hipGetLastError());
            hipLaunchKernelGGL(refine_compact_kernel, dim3(NB), dim3(256), 0, st, (const int*)(ws + p.rcnt), m.t,
                               m.R, crow, ccount);
            HIP_TRY(hipGetLastError());
            if constexpr (sizeof(CT) == 2) {
              // gather, exact key projection from [K_hi | V | K_lo] and dot
              // product with the fp32 q~ in one kernel
              RefineKArgs rk_;
              rk_.K = Kp;
              rk_.V = Vp;
              rk_.invf_b = invf_b;
              rk_.pos = positions;
              rk_.invf_c = invf_c;
              rk_.wkt = (const f16*)(ws + p.wkt);
              rk_.bias = bw.ca_bk;
              rk_.ridx = ridx;
              rk_.crow = crow;
              rk_.count = ccount;
              rk_.qex = (const float*)(ws + p.qex);
              rk_.rpart = (float2*)(ws + p.rpart);
              rk_.hscale = (const float*)(ws + p.hscale);
              rk_.N = m.N;
              rk_.t = m.t;
              rk_.R = m.R;
              rk_.nc = m.nc;
              rk_.dc = m.dc;
              constexpr int BMR = 64;   // candidate rows per workgroup (LDS: BMR x 3d fp16; 2-3 workgroups per CU)
              rk_.H = m.H;
              rk_.ntile = (m.t * REFINE_GRID_R + BMR - 1) / BMR;
              const dim3 rg((unsigned)(rk_.ntile * NB));
              if (m.d == 64) hipLaunchKernelGGL((refine_kernel<64, BMR, IT, IT>), rg, dim3(256), 0, st, rk_);
              else if (m.d == 128) hipLaunchKernelGGL((refine_kernel<128, BMR, IT, IT>), rg, dim3(256), 0, st, rk_);
              else hipLaunchKernelGGL((refine_kernel<256, BMR, IT, IT>), rg, dim3(256), 0, st, rk_);
              HIP_TRY(hipGetLastError());
            } else {
              // fp32 mode: the refined keys' logits in fp64 (refine64.hpp)
              double* q64 = (double*)(ws + p.q64);
              Q64Args qa;
              qa.Z = Z;
              qa.W = (const float*)bw.ca_wq;
              qa.bias = (const float*)bw.ca_bq;
              qa.Q = q64;
              qa.rows = Ht;
              qa.D = m.D;
              qa.E = m.Ec;
              qa.rms_eps = cfg->rms_eps;
              hipLaunchKernelGGL(q64_gemm_kernel, dim3((unsigned)((m.Ec + 127) / 128), (unsigned)((Ht + 127) / 128)),
                                 dim3(256), 0, st, qa);
              HIP_TRY(hipGetLastError());
              hipLaunchKernelGGL(q64_finalize_kernel, dim3((unsigned)((Ht * m.nc + 3) / 4)), dim3(256), 0, st, q64,
                                 Ht, m.nc, m.dc, m.t, (const double*)(ws + p.pq), (const double*)(ws + p.invf_c),
                                 (double)cfg->l2_eps);
              HIP_TRY(hipGetLastError());
              Refine64Args r6;
              r6.K = (const float*)Kp;
              r6.V = (const float*)Vp;
              r6.pos = positions;
              r6.invf_b = (const double*)(ws + p.invf_b);
              r6.invf_c = (const double*)(ws + p.invf_c);
              r6.W = (const float*)bw.ca_wk;
              r6.bias = (const float*)bw.ca_bk;
              r6.Q = q64;
              r6.ridx = ridx;
              r6.rval = (const float*)(ws + p.rval);
              r6.crow = crow;
              r6.count = ccount;
              r6.rpart = (float2*)(ws + p.rpart);
              r6.N = m.N;
              r6.H = m.H;
              r6.t = m.t;
              r6.R = m.R;
              r6.nc = m.nc;
              r6.dc = m.dc;
              r6.d = m.d;
              r6.scale_log2 = (double)ca_scale * 1.4426950408889634;
              r6.l2_eps = (double)cfg->l2_eps;
              r6.ntile = (m.t * REFINE_GRID_R + 15) / 16;
              const dim3 rg((unsigned)(r6.ntile * NB));
              if (m.d == 64) hipLaunchKernelGGL((refine64_kernel<64>), rg, dim3(256), 0, st, r6);
              else if (m.d == 128) hipLaunchKernelGGL((refine64_kernel<128>), rg, dim3(256), 0, st, r6);
              else hipLaunchKernelGGL((refine64_kernel<256>), rg, dim3(256), 0, st, r6);
              HIP_TRY(hipGetLastError());
            }
          }
          ra.R = m.R;
          ra.NP = sizeof(CT) == 2 ? 1 : 0;
          ra.ridx = ridx;
          ra.rcnt = (const int*)(ws + p.rcnt);
          ra.rval = (const float*)(ws + p.rval);
          ra.rpart = (const float2*)(ws + p.rpart);
          ra.rq = rq;
          ra.X = X;
          ra.N = m.N;
          ra.scale_log2 = a.scale_log2;
          ra.l2_eps = cfg->l2_eps;
        }
        TIMED(STILL_K_OTHER);
        const dim3 mg((unsigned)((Ht * m.nc + 3) / 4));
        if (m.d2 == 128)
          hipLaunchKernelGGL((merge_kernel<CT, 2>), mg, dim3(256), 0, st, a.opart, a.mpart, a.lpart, m.splits, m.H,
                             m.nc, m.t, O, ra);
        else if (m.d2 == 256)
          hipLaunchKernelGGL((merge_kernel<CT, 4>), mg, dim3(256), 0, st, a.opart, a.mpart, a.lpart, m.splits, m.H,
                             m.nc, m.t, O, ra);
        else
          hipLaunchKernelGGL((merge_kernel<CT, 8>), mg, dim3(256), 0, st, a.opart, a.mpart, a.lpart, m.splits, m.H,
                             m.nc, m.t, O, ra);
        HIP_TRY(hipGetLastError());
      }
      {  // head_c = O_c W_V,c^T   (batched over cross heads c)
        GemmArgs g = gargs((int)Ht, m.dc, m.d2, O, (long)m.nc * m.d2, bw.ca_wv, m.d2, head, m.Ec);
        g.nb2 = m.nc;
        g.sA2 = m.d2;
        g.sB2 = (long)m.dc * m.d2;
        g.sC2 = m.dc;
        HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_STORE, true>(g, m.nc, st)));
      }
      {  // Z += Concat(heads) W_O^T (times 2^e_h: the value path carried the fp16 range scale)
        GemmArgs g = gargs((int)Ht, m.D, m.Ec, head, m.Ec, bw.ca_wo, m.Ec, Z, m.D);
        if (!m.fp32) {
          g.rowscale = (const float*)(ws + p.hscale) + m.H;   // 2^e_h
          g.rowscale_div = m.t;
        }
        HIP_TRY((gemm<CT, CT, CT, float, IT, EPI_RESID, true>(g, 1, st)));
      }
    }
    // ---------------- latent self-attention: Z += SelfAttn(RMSNorm(Z))
    // bf16 mode, d_s of 128, 256 or 512: q row-major, k and v written by their
    // projections straight into the fp16 flash kernel's tiled layouts, the
    // flash kernel without logit refinement, then the split merge
    if constexpr (sizeof(CT) == 2) {
      if (m.ns > 0 && m.sa_flash) {
        CT* qs = (CT*)(ws + p.qs);
        CT* ks = (CT*)(ws + p.ks);
        CT* vT = (CT*)(ws + p.vT);
        float* partqs = (float*)(ws + p.partqs);
        float* partks = (float*)(ws + p.partks);
        float* rqs = (float*)(ws + p.rqs);
        float* rks = (float*)(ws + p.rks);
        CT* Osa = (CT*)(ws + p.Osa);
        HIP_TRY(rmsnorm());
        {
          GemmArgs g = gargs((int)Ht, m.Es / 2, m.D, Y, m.D, bw.sa_wq, m.D, qs, m.Es);
          g.bias = bw.sa_bq;
          g.hd = m.ds;
          g.part = partqs;
          g.ldpart = Ht;
          if (wide_s) HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR, true>(g, 1, st)));
          else HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR>(g, 1, st)));
          g.B = bw.sa_wk;
          g.bias = bw.sa_bk;
          g.C = ks;
          g.part = partks;
          g.ctile = CTILE_KEYS;   // [h * n_s + c][key tiles]
          g.ctile_rows = m.t;
          g.ctile_heads = m.ns;
          g.ctile_npad = m.tpadk;
          if (wide_s) HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR, true>(g, 1, st)));
          else HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR>(g, 1, st)));
          if (m.tpadk > m.t) {   // keys past t: finite (zero) slots for the additive mask of the attention
            TIMED(STILL_K_OTHER);
            hipLaunchKernelGGL(zero_ktile_tail_kernel, dim3(grid1d((long)m.H * m.ns * (m.tpadk - m.t) * (m.ds / 8))),
                               dim3(256), 0, st, (f16*)ks, (long)m.H * m.ns, m.t, (long)m.tpadk, m.ds);
            HIP_TRY(hipGetLastError());
          }
        }
        {  // v^T[h] = W_V^sa Y[h]^T, tiled [h][feature tiles][key steps]
          GemmArgs g = gargs(m.Es, m.t, m.D, bw.sa_wv, m.D, Y, m.D, vT, m.tpadk);
          g.sB1 = (long)m.t * m.D;
          g.sC1 = (long)m.Es * m.tpadk;
          g.ctile = CTILE_VALUES;
          g.ctile_npad = m.tpadk;
          HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_STORE, true>(g, m.H, st)));
          if (m.tpadk > m.t) {   // keys past t: zero values (their weights are exactly 0)
            TIMED(STILL_K_OTHER);
            hipLaunchKernelGGL(zero_xtile_tail_kernel, dim3(grid1d((long)m.H * m.Es * (m.tpadk - m.t))), dim3(256), 0,
                               st, (f16*)vT, (long)m.H * m.Es, m.t, m.tpadk);
            HIP_TRY(hipGetLastError());
          }
        }
        HIP_TRY(finalize(partqs, Ht, m.ns, wide_s ? m.ds / 256 * 2 : m.np_s, rqs));
        HIP_TRY(finalize(partks, Ht, m.ns, wide_s ? m.ds / 256 * 2 : m.np_s, rks));
        AttnArgs a;
        memset(&a, 0, sizeof a);
        a.q = qs;
        a.ldq = m.Es;
        a.rq = rqs;
        a.k = ks;
        a.rk = rks;
        a.xt = vT;
        a.npad = m.tpadk;
        a.xfeat = m.Es;
        a.xcoff = m.ds;
        a.opart = (float*)(ws + p.opart_s);
        a.mpart = (float*)(ws + p.mpart_s);
        a.lpart = (float*)(ws + p.lpart_s);
        a.H = m.H;
        a.N = m.t;
        a.t = m.t;
        a.nc = m.ns;
        a.dc = m.ds;
        a.d2 = m.ds;
        a.scale_log2 = (cfg->logit_scale_self != 0.f ? cfg->logit_scale_self : (float)m.ds) * LOG2E;
        a.keys_per_split = (int)m.sa_kps;
        RefineArgs ra;
        memset(&ra, 0, sizeof ra);
        {
          TIMED(STILL_K_LATENT);
          hipError_t e;
          if (m.ds == 128) e = launch_attn<CT, 128, 0>(a, m.sa_splits, st);
          else if (m.ds == 256) e = launch_attn<CT, 256, 0>(a, m.sa_splits, st);
          else e = launch_attn<CT, 512, 0>(a, m.sa_splits, st);
          HIP_TRY(e);
          const dim3 mg((unsigned)((Ht * m.ns + 3) / 4));
          if (m.ds == 128)
            hipLaunchKernelGGL((merge_kernel<CT, 2>), mg, dim3(256), 0, st, a.opart, a.mpart, a.lpart, m.sa_splits,
                               m.H, m.ns, m.t, Osa, ra);
          else if (m.ds == 256)
            hipLaunchKernelGGL((merge_kernel<CT, 4>), mg, dim3(256), 0, st, a.opart, a.mpart, a.lpart, m.sa_splits,
                               m.H, m.ns, m.t, Osa, ra);
          else
            hipLaunchKernelGGL((merge_kernel<CT, 8>), mg, dim3(256), 0, st, a.opart, a.mpart, a.lpart, m.sa_splits,
                               m.H, m.ns, m.t, Osa, ra);
          HIP_TRY(hipGetLastError());
        }
        GemmArgs g = gargs((int)Ht, m.D, m.Es, Osa, m.Es, bw.sa_wo, m.Es, Z, m.D);
        HIP_TRY((gemm<CT, CT, CT, float, IT, EPI_RESID, true>(g, 1, st)));
      }
    }
    if (m.ns > 0 && !m.sa_flash) {
      CT* qs = (CT*)(ws + p.qs);
      CT* ks = (CT*)(ws + p.ks);
      CT* vT = (CT*)(ws + p.vT);
      float* partqs = (float*)(ws + p.partqs);
      float* partks = (float*)(ws + p.partks);
      float* rqs = (float*)(ws + p.rqs);
      float* rks = (float*)(ws + p.rks);
      float* Ssa = (float*)(ws + p.Ssa);
      CT* Psa = (CT*)(ws + p.Psa);
      CT* Osa = (CT*)(ws + p.Osa);
      HIP_TRY(rmsnorm());
      {
        GemmArgs g = gargs((int)Ht, m.Es / 2, m.D, Y, m.D, bw.sa_wq, m.D, qs, m.Es);
        g.bias = bw.sa_bq;
        g.hd = m.ds;
        g.part = partqs;
        g.ldpart = Ht;
        if (wide_s) HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR, true>(g, 1, st)));
        else HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR>(g, 1, st)));
        g.B = bw.sa_wk;
        g.bias = bw.sa_bk;
        g.C = ks;
        g.part = partks;
        if (wide_s) HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR, true>(g, 1, st)));
        else HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_PAIR>(g, 1, st)));
      }
      {  // v^T[h] = W_V^sa Y[h]^T : [Es][tpad] per KV head
        GemmArgs g = gargs(m.Es, m.t, m.D, bw.sa_wv, m.D, Y, m.D, vT, m.tpad);
        g.sB1 = (long)m.t * m.D;
        g.sC1 = (long)m.Es * m.tpad;
        HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_STORE, true>(g, m.H, st)));
        if (m.tpad > m.t) {
          TIMED(STILL_K_OTHER);
          hipLaunchKernelGGL((zero_cols_kernel<CT>), dim3(grid1d((long)m.H * m.Es * (m.tpad - m.t))), dim3(256), 0,
                             st, vT, (long)m.H * m.Es, m.tpad, m.t, m.tpad);
          HIP_TRY(hipGetLastError());
        }
      }
      HIP_TRY(finalize(partqs, Ht, m.ns, wide_s ? m.ds / 256 * 2 : m.np_s, rqs));
      HIP_TRY(finalize(partks, Ht, m.ns, wide_s ? m.ds / 256 * 2 : m.np_s, rks));
      {  // S = s * q k^T with the QK-norm factors, per (h, c)
        GemmArgs g = gargs(m.t, m.t, m.ds, qs, m.Es, ks, m.Es, Ssa, m.tpad);
        g.nb2 = m.ns;
        g.sA1 = (long)m.t * m.Es;
        g.sA2 = m.ds;
        g.sB1 = (long)m.t * m.Es;
        g.sB2 = m.ds;
        g.sC1 = (long)m.ns * m.t * m.tpad;
        g.sC2 = (long)m.t * m.tpad;
        g.scale = cfg->logit_scale_self != 0.f ? cfg->logit_scale_self : (float)m.ds;
        g.rq = rqs;
        g.ldrq = m.ns;
        g.sQ1 = (long)m.t * m.ns;
        g.sQ2 = 1;
        g.rk = rks;
        g.ldrk = m.ns;
        g.sK1 = (long)m.t * m.ns;
        g.sK2 = 1;
        HIP_TRY((gemm<CT, CT, CT, float, IT, EPI_SCALE, true>(g, m.H * m.ns, st)));
      }
      {
      TIMED(STILL_K_OTHER);
      SoftmaxRefine sr;
      memset(&sr, 0, sizeof sr);
      if (m.fp32) {   // fp32 mode: q, k already fp32 -> recompute each row's top logits
        sr.q = (const float*)qs;
        sr.k = (const float*)ks;
        sr.rq = rqs;
        sr.rk = rks;
        sr.Es = m.Es;
        sr.ds = m.ds;
        sr.ns = m.ns;
        sr.t = m.t;
        sr.scale = cfg->logit_scale_self != 0.f ? cfg->logit_scale_self : (float)m.ds;
      }
      hipLaunchKernelGGL((softmax_rows_kernel<CT>), dim3((unsigned)(((long)m.H * m.ns * m.t + 3) / 4)), dim3(256), 0,
                         st, Ssa, Psa, (long)m.H * m.ns * m.t, m.t, m.tpad, sr);
      }
      HIP_TRY(hipGetLastError());
      {  // O = P v per (h, c)
        GemmArgs g = gargs(m.t, m.ds, m.tpad, Psa, m.tpad, vT, m.tpad, Osa, m.Es);
        g.nb2 = m.ns;
        g.sA1 = (long)m.ns * m.t * m.tpad;
        g.sA2 = (long)m.t * m.tpad;
        g.sB1 = (long)m.Es * m.tpad;
        g.sB2 = (long)m.ds * m.tpad;
        g.sC1 = (long)m.t * m.Es;
        g.sC2 = m.ds;
        HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_STORE, true>(g, m.H * m.ns, st)));
      }
      {
        GemmArgs g = gargs((int)Ht, m.D, m.Es, Osa, m.Es, bw.sa_wo, m.Es, Z, m.D);
        HIP_TRY((gemm<CT, CT, CT, float, IT, EPI_RESID, true>(g, 1, st)));
      }
    }
    // ---------------- FFN: Z += FFN(RMSNorm(Z))
    if (cfg->ffn_kind != STILL_FFN_NONE) {
      CT* hid = (CT*)(ws + p.hid);
      HIP_TRY(rmsnorm());
      if (cfg->ffn_kind == STILL_FFN_SWIGLU) {
        GemmArgs g = gargs((int)Ht, m.F, m.D, Y, m.D, bw.ffn_wg, m.D, hid, m.F);
        g.B2 = bw.ffn_wu;
        HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_SWIGLU, true>(g, 1, st)));
      } else {
        GemmArgs g = gargs((int)Ht, m.F, m.D, Y, m.D, bw.ffn_wu, m.D, hid, m.F);
        HIP_TRY((gemm<CT, CT, CT, CT, IT, EPI_GELU, true>(g, 1, st)));
      }
      GemmArgs g = gargs((int)Ht, m.D, m.F, hid, m.F, bw.ffn_wd, m.F, Z, m.D);
      HIP_TRY((gemm<CT, CT, CT, float, IT, EPI_RESID, true>(g, 1, st)));
    }
  }
  // ---------------- output heads: C_k = Z_out W_key^T (re-rotated), C_v = Z_out W_val^T
  {
    GemmArgs gk = gargs((int)Ht, m.d / 2, m.D, Z, m.D, w->w_key, m.D, Ckp, m.d);
    gk.hd = m.d;
    gk.tab = rerotate ? tab_bq : nullptr;
    gk.tab_mod = m.t;
    GemmArgs gv = gargs((int)Ht, m.d, m.D, Z, m.D, w->w_val, m.D, Cvp, m.d);
    if (cfg->final_norm) {
      HIP_TRY(rmsnorm());
      gk.A = Y;
      gv.A = Y;
      HIP_TRY((gemm<CT, CT, CT, IT, IT, EPI_PAIR>(gk, 1, st)));
      HIP_TRY((gemm<CT, CT, CT, IT, IT, EPI_STORE>(gv, 1, st)));
    } else {
      HIP_TRY((gemm<CT, float, CT, IT, IT, EPI_PAIR>(gk, 1, st)));
      HIP_TRY((gemm<CT, float, CT, IT, IT, EPI_STORE>(gv, 1, st)));
    }
  }
  return STILL_OK;
}

}  // namespace still
